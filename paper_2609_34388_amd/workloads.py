"""Seeded synthetic inputs for the fused draft-verify step.

The paper measures on a real diffusion/AR backbone over eight public benchmarks
(Sec. 6.1).  Neither the weights nor the datasets are used here: these
generators stand in for them with random tensors whose shapes follow the
paper's serving regimes -- one request with B = 16 at concurrency 1 (Sec. 6.1,
Table 1), per-request block sizes from {8, 16, 32} and smaller at higher
concurrency (Sec. 5.2, Eq. 3), concurrency up to 128 (Sec. 6.1) -- in an
8B-style grouped-query shape (32 query heads, 8 KV heads, head dim 128,
vocabulary 128256).

This module only draws random numbers and lays them out in the layouts the
library reads.  It computes nothing that the attention, the acceptance rule or
the confidence statistics compute, so both the CPU oracle and the GPU path can
consume its output without sharing any of the method's arithmetic.

Layouts produced (all contiguous):
  q             [sum_r n_r, Hq, D]        bf16, rows of request r at q_indptr[r]
  k_cache       [num_pages, Hkv, 16, D]   bf16, token-major pages
  v_cache       [num_pages, Hkv, D, 16]   bf16, dim-major pages
  verify_logits [sum_r rows_r, vocab]     bf16, rows of request r at row_indptr[r]
  draft_tokens  [sum_r rows_r]            int32, token judged by each verify row
  draft_logits  [sum_r B_r, vocab]        bf16
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Tuple

import numpy as np
import torch

PAGE_SIZE = 16
_SEED_TAG = 0x52476964  # fixed tag so every workload has its own seed family


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    """Distribution of one synthetic workload.

    ``ctx``, ``verify``, ``draft`` and ``sigma`` are tuples
    ``("fixed", x)``, ``("uniform", lo, hi)`` (integers inclusive for lengths,
    real for sigma) or ``("choice", values, probs_or_None)``.
    """

    name: str
    index: int
    num_requests: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    vocab: int
    ctx: tuple
    verify: tuple
    draft: tuple
    sigma: tuple
    qkv_std: float
    draft_std: float = 2.0


_8B = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, vocab=128256,
           qkv_std=1.0 / math.sqrt(128.0))

SPECS: Dict[str, WorkloadSpec] = {
    # Tiny case the oracle finishes in well under a second.
    "tiny": WorkloadSpec("tiny", 0, 1, 2, 1, 64, 1024, ("fixed", 128),
                         ("fixed", 4), ("fixed", 8), ("fixed", 1.0), 1.0),
    # Concurrency 1, B = 16 after a B = 16 block (the low-concurrency regime).
    "low": WorkloadSpec("low", 1, 1, ctx=("fixed", 4096), verify=("fixed", 16),
                        draft=("fixed", 16), sigma=("fixed", 0.5), **_8B),
    "low_sigma2": WorkloadSpec("low_sigma2", 1, 1, ctx=("fixed", 4096),
                               verify=("fixed", 16), draft=("fixed", 16),
                               sigma=("fixed", 2.0), **_8B),
    # 16 requests, per-request block sizes.
    "mid": WorkloadSpec("mid", 2, 16, ctx=("uniform", 1024, 8192),
                        verify=("choice", (4, 8, 16, 32), None),
                        draft=("choice", (4, 8, 16, 32), None),
                        sigma=("choice", (0.5, 2.0), None), **_8B),
    # 128 requests, small blocks dominate.
    "high": WorkloadSpec("high", 3, 128, ctx=("uniform", 512, 4096),
                         verify=("choice", (2, 4, 8, 16), (0.4, 0.3, 0.2, 0.1)),
                         draft=("choice", (2, 4, 8, 16), (0.4, 0.3, 0.2, 0.1)),
                         sigma=("uniform", 0.5, 3.0), **_8B),
    # 64 requests with 16k-32k contexts.
    "long": WorkloadSpec("long", 4, 64, ctx=("uniform", 16384, 32768),
                         verify=("choice", (4, 8, 16, 32), None),
                         draft=("choice", (4, 8, 16, 32), None),
                         sigma=("fixed", 1.0), **_8B),
}
CONFIG_ORDER = ("tiny", "low", "mid", "high", "long")


@dataclasses.dataclass
class Layout:
    """One seeded draw of a workload's ragged structure (host arrays)."""

    spec: WorkloadSpec
    seed: int
    ctx_len: np.ndarray        # [R] int32, keys already cached before the new rows
    n_verify: np.ndarray       # [R] int32, verify query rows
    n_draft: np.ndarray        # [R] int32, next-draft query rows
    sigma: np.ndarray          # [R] float64, verify-noise std
    bonus: np.ndarray          # [R] int32, 1 if a bonus verify-logit row is appended
    q_indptr: np.ndarray       # [R+1] int32
    page_indptr: np.ndarray    # [R+1] int32
    page_indices: np.ndarray   # [sum pages] int32
    num_pages: int             # pool size (>= pages referenced)
    row_indptr: np.ndarray     # [R+1] int32, verify-logit rows per request
    draft_row_indptr: np.ndarray  # [R+1] int32, draft-logit rows per request

    @property
    def num_requests(self) -> int:
        return int(self.ctx_len.shape[0])

    @property
    def q_len(self) -> np.ndarray:
        return (self.n_verify + self.n_draft).astype(np.int32)

    @property
    def kv_len(self) -> np.ndarray:
        return (self.ctx_len + self.q_len).astype(np.int32)

    @property
    def total_q(self) -> int:
        return int(self.q_indptr[-1])

    @property
    def total_verify_rows(self) -> int:
        return int(self.row_indptr[-1])

    @property
    def total_draft_rows(self) -> int:
        return int(self.draft_row_indptr[-1])


def _draw(rng: np.random.Generator, dist: tuple, n: int, integer: bool) -> np.ndarray:
    kind = dist[0]
    if kind == "fixed":
        out = np.full(n, dist[1])
    elif kind == "uniform":
        if integer:
            out = rng.integers(dist[1], dist[2] + 1, size=n)
        else:
            out = rng.uniform(dist[1], dist[2], size=n)
    elif kind == "choice":
        out = rng.choice(np.asarray(dist[1]), size=n, p=dist[2])
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return out.astype(np.int32 if integer else np.float64)


def _prefix(x: np.ndarray) -> np.ndarray:
    out = np.zeros(x.shape[0] + 1, dtype=np.int64)
    np.cumsum(x, out=out[1:])
    if out[-1] > np.iinfo(np.int32).max:
        raise ValueError("prefix exceeds int32")
    return out.astype(np.int32)


def _seed_sequence(spec: WorkloadSpec, seed: int) -> np.random.SeedSequence:
    return np.random.SeedSequence([_SEED_TAG, spec.index, seed])


def make_layout(spec, seed: int = 0, *, num_requests: Optional[int] = None,
                ctx: Optional[tuple] = None, verify: Optional[tuple] = None,
                draft: Optional[tuple] = None, sigma: Optional[tuple] = None,
                spare_pages: int = 8, shuffle_pages: bool = True,
                bonus_rows: bool = False) -> Layout:
    """Draw the ragged structure of a workload.

    Overrides replace the spec's distributions (used by tests for scaled-down
    or degenerate cases).  Pages are taken from a pool with ``spare_pages``
    unreferenced pages and, by default, assigned in a random order.
    """
    if isinstance(spec, str):
        spec = SPECS[spec]
    changes = {k: v for k, v in dict(num_requests=num_requests, ctx=ctx, verify=verify,
                                     draft=draft, sigma=sigma).items() if v is not None}
    if changes:
        spec = dataclasses.replace(spec, **changes)
    rng = np.random.default_rng(_seed_sequence(spec, seed).spawn(1)[0])
    R = spec.num_requests
    ctx_len = _draw(rng, spec.ctx, R, True)
    n_verify = _draw(rng, spec.verify, R, True)
    n_draft = _draw(rng, spec.draft, R, True)
    sig = _draw(rng, spec.sigma, R, False)
    bonus = np.full(R, 1 if bonus_rows else 0, dtype=np.int32)
    q_len = n_verify + n_draft
    kv_len = ctx_len + q_len
    pages_per = (kv_len + PAGE_SIZE - 1) // PAGE_SIZE
    used = int(pages_per.sum())
    num_pages = used + spare_pages
    order = rng.permutation(num_pages) if shuffle_pages else np.arange(num_pages)
    page_indices = order[:used].astype(np.int32)
    return Layout(spec=spec, seed=seed, ctx_len=ctx_len, n_verify=n_verify,
                  n_draft=n_draft, sigma=sig, bonus=bonus,
                  q_indptr=_prefix(q_len), page_indptr=_prefix(pages_per),
                  page_indices=page_indices, num_pages=num_pages,
                  row_indptr=_prefix(n_verify + bonus),
                  draft_row_indptr=_prefix(n_draft))



def overlap_branches(layout: Layout):
    """Branches of an overlap round for each request of ``layout``, in the
    largest form Sec. 5.1 prepares: correction branches at two distinct
    seeded positions of the V-token block under verification (one when
    V = 1, none when V = 0), each a committed replacement token followed by a
    B-token draft block -- (prefix = position, lead = 1, rows = 1 + B) --
    then a continuation branch that keeps the whole block and drafts B rows
    -- (V, 0, B).  B is the request's draft block size in ``layout``.
    Returns one list of (prefix, lead, rows) per request."""
    rng = np.random.default_rng(_seed_sequence(layout.spec, layout.seed).spawn(8)[6])
    out = []
    for r in range(layout.num_requests):
        V, B = int(layout.n_verify[r]), int(layout.n_draft[r])
        pos = sorted(int(p) for p in rng.choice(V, size=min(2, V), replace=False)) if V else []
        br = [(p, 1, 1 + B) for p in pos]
        if B:
            br.append((V, 0, B))
        out.append(br)
    return out



def quadratic_branches(layout: Layout):
    """The quadratic speculative layout the paper contrasts RecGuide with
    (Sec. 6.2): for each request, one B-row draft block per hypothetical
    accepted length a = 0 .. V of the block under verification, each keeping
    the first a verify rows and supplying no correction token --
    (prefix = a, lead = 0, rows = B) for every a; (V + 1) B rows in all."""
    out = []
    for r in range(layout.num_requests):
        V, B = int(layout.n_verify[r]), int(layout.n_draft[r])
        out.append([(a, 0, B) for a in range(V + 1)] if B else [])
    return out

def _paged(layout: Layout, ctx_len, n_verify, n_draft, page_indptr, page_indices, num_pages) -> Layout:
    z = np.zeros(len(ctx_len), dtype=np.int32)
    ctx_len, n_verify, n_draft = (np.asarray(a, dtype=np.int32) for a in (ctx_len, n_verify, n_draft))
    return Layout(spec=layout.spec, seed=layout.seed, ctx_len=ctx_len, n_verify=n_verify, n_draft=n_draft,
                  sigma=np.ones(len(ctx_len)), bonus=z, q_indptr=_prefix(n_verify + n_draft),
                  page_indptr=np.asarray(page_indptr, dtype=np.int32),
                  page_indices=np.asarray(page_indices, dtype=np.int32), num_pages=int(num_pages),
                  row_indptr=_prefix(n_verify), draft_row_indptr=_prefix(n_draft))


def make_overlap_layout(layout: Layout, branches, spare_pages: int = 8) -> Layout:
    """``layout`` with each request's rows after its verify rows replaced by
    its branches' rows (their keys follow the verify rows in the request's
    pages, in branch order); pages freshly permuted."""
    rng = np.random.default_rng(_seed_sequence(layout.spec, layout.seed).spawn(8)[7])
    n_draft = np.array([sum(b[2] for b in br) for br in branches], dtype=np.int32)
    kv = layout.ctx_len + layout.n_verify + n_draft
    pages = (kv + PAGE_SIZE - 1) // PAGE_SIZE
    used = int(pages.sum())
    order = rng.permutation(used + spare_pages)
    return _paged(layout, layout.ctx_len, layout.n_verify, n_draft, _prefix(pages), order[:used],
                  used + spare_pages)



def with_blocks(layout: Layout, n_verify, n_draft, spare_pages: int = 8) -> Layout:
    """``layout``'s requests (same contexts) with new verify / draft row counts
    and a freshly permuted page table."""
    rng = np.random.default_rng(_seed_sequence(layout.spec, layout.seed).spawn(8)[7])
    nv = np.asarray(n_verify, dtype=np.int32)
    nd = np.asarray(n_draft, dtype=np.int32)
    kv = layout.ctx_len + nv + nd
    pages = (kv + PAGE_SIZE - 1) // PAGE_SIZE
    used = int(pages.sum())
    order = rng.permutation(used + spare_pages)
    return _paged(layout, layout.ctx_len, nv, nd, _prefix(pages), order[:used], used + spare_pages)


def subset(layout: Layout, requests) -> Layout:
    """The listed requests of ``layout`` as a batch of their own (same
    pages, same order of the page pool)."""
    req = np.asarray(requests, dtype=np.int64)
    counts = (layout.page_indptr[req + 1] - layout.page_indptr[req]).astype(np.int64)
    idx = np.concatenate([layout.page_indices[layout.page_indptr[r]:layout.page_indptr[r + 1]] for r in req]) \
        if len(req) else np.zeros(0, np.int32)
    return _paged(layout, layout.ctx_len[req], layout.n_verify[req], layout.n_draft[req], _prefix(counts), idx,
                  layout.num_pages)

def make_separate_layout(overlap: Layout, branches) -> Tuple[Layout, list]:
    """The same rows served without a shared prefix: every request of
    ``overlap`` becomes one request of its verify rows plus one request per
    branch, whose context is the branch's kept prefix (its full pages alias
    the shared request's pages, as prefix caching would) followed by the
    branch's own rows on fresh pages.  Returns the layout and, per new
    request, (original request, branch index or -1)."""
    ctx, nv, nd, counts, idx, origin = [], [], [], [], [], []
    fresh = overlap.num_pages
    for r, br in enumerate(branches):
        L, V = int(overlap.ctx_len[r]), int(overlap.n_verify[r])
        own = overlap.page_indices[int(overlap.page_indptr[r]):int(overlap.page_indptr[r + 1])]
        if V:
            n_pages = (L + V + PAGE_SIZE - 1) // PAGE_SIZE
            ctx.append(L); nv.append(V); nd.append(0); counts.append(n_pages)
            idx.extend(own[:n_pages]); origin.append((r, -1))
        for b, (prefix, lead, rows) in enumerate(br):
            kept = L + prefix
            full = kept // PAGE_SIZE
            total = (kept + rows + PAGE_SIZE - 1) // PAGE_SIZE
            ctx.append(kept); nv.append(lead); nd.append(rows - lead); counts.append(total)
            idx.extend(own[:full])
            idx.extend(range(fresh, fresh + total - full))
            fresh += total - full
            origin.append((r, b))
    return _paged(overlap, ctx, nv, nd, _prefix(np.asarray(counts, dtype=np.int64)), idx, fresh), origin


def make_separate_kv(overlap: Layout, branches, separate: Layout, origin, k_cache: torch.Tensor,
                     v_cache: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """K/V pools for ``make_separate_layout``'s layout holding the same keys:
    the shared pages as they are, and on each branch request's fresh pages
    the rest of its kept prefix and its own rows, copied from ``overlap``'s
    pools (a data copy only)."""
    dst_p, dst_s, src_p, src_s = [], [], [], []
    offsets = []
    for br in branches:
        off, acc = [], 0
        for b in br:
            off.append(acc)
            acc += b[2]
        offsets.append(off)
    for i, (r, b) in enumerate(origin):
        if b < 0:
            continue
        L, V = int(overlap.ctx_len[r]), int(overlap.n_verify[r])
        prefix, _, rows = branches[r][b]
        kept = L + prefix
        first = (kept // PAGE_SIZE) * PAGE_SIZE
        j = np.arange(first, kept + rows)
        src = np.where(j < kept, j, L + V + offsets[r][b] + (j - kept))
        own = overlap.page_indices[int(overlap.page_indptr[r]):]
        sp = separate.page_indices[int(separate.page_indptr[i]):]
        dst_p.append(sp[j // PAGE_SIZE]); dst_s.append(j % PAGE_SIZE)
        src_p.append(own[src // PAGE_SIZE]); src_s.append(src % PAGE_SIZE)
    k = torch.zeros((separate.num_pages,) + tuple(k_cache.shape[1:]), dtype=k_cache.dtype, device=k_cache.device)
    v = torch.zeros((separate.num_pages,) + tuple(v_cache.shape[1:]), dtype=v_cache.dtype, device=v_cache.device)
    k[:k_cache.shape[0]] = k_cache
    v[:v_cache.shape[0]] = v_cache
    if dst_p:
        t = lambda a: torch.as_tensor(np.concatenate(a).astype(np.int64), device=k_cache.device)
        dp, ds, sp_, ss = t(dst_p), t(dst_s), t(src_p), t(src_s)
        k[dp, :, ds, :] = k_cache[sp_, :, ss, :]
        v[dp, :, :, ds] = v_cache[sp_, :, :, ss]
    return k, v


BLOCK_CANDIDATES = (8, 16, 32)


def make_block_policy_inputs(seed: int = 0, num_requests: int = 128, num_s_bins: int = 8,
                             candidates=BLOCK_CANDIDATES) -> Dict[str, np.ndarray]:
    """A synthetic block-size policy and one round of request states.

    The paper calibrates its value table from model rollouts; this stand-in
    is a smooth table of the same shape: an expected acceptance potential
    A = 2 + 30 exp(2 s) (1.5 after a full acceptance) (B_prev / 16)^0.25 at
    each s-bin centre, and V_B = A (1 - exp(-B / A)) -- more progress for
    larger blocks, saturating at A -- plus N(0, 0.05) noise.  s-bin edges
    are evenly spaced on [-4, 0].  Request states: entropies U[0, 3],
    previous block sizes drawn from the candidates, accepted lengths
    U{0 .. B_prev}.  Costs are left to the caller (they are measured)."""
    rng = np.random.default_rng(np.random.SeedSequence([_SEED_TAG, 99, seed]))
    cand = np.asarray(candidates, dtype=np.int32)
    nb, ns = len(cand), int(num_s_bins)
    edges = np.linspace(-4.0, 0.0, ns + 1)[1:-1].astype(np.float32) if ns > 1 else np.zeros(0, np.float32)
    lo = np.concatenate([[-5.0], edges])
    hi = np.concatenate([edges, [0.5]])
    centre = 0.5 * (lo + hi)
    value = np.zeros((nb, ns, nb, 2), dtype=np.float32)
    for k in range(ns):
        for j in range(nb):
            for f in range(2):
                A = 2.0 + 30.0 * np.exp(2.0 * centre[k]) * (1.5 if f else 1.0) * (cand[j] / 16.0) ** 0.25
                value[:, k, j, f] = A * (1.0 - np.exp(-cand / A))
    value += rng.normal(0.0, 0.05, size=value.shape).astype(np.float32)
    R = int(num_requests)
    prev = rng.choice(cand, size=R).astype(np.int32)
    accept = np.array([rng.integers(0, p + 1) for p in prev], dtype=np.int32)
    return dict(candidates=cand, s_edges=edges, value=value.astype(np.float32),
                accept_len=accept, accept_entropy=rng.uniform(0, 3, R).astype(np.float32),
                entropy_hist=rng.uniform(0, 3, R).astype(np.float32), prev_block=prev)

def _gen(layout: Layout, device, stream: int) -> torch.Generator:
    ss = _seed_sequence(layout.spec, layout.seed).spawn(8)[stream]
    g = torch.Generator(device=device)
    g.manual_seed(int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    return g


def _randn(shape, std, gen, device, chunk_elems=1 << 26) -> torch.Tensor:
    """fp32 N(0, std) draws rounded once (round-to-nearest-even) to bf16."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    for s in range(0, flat.numel(), chunk_elems):
        e = min(flat.numel(), s + chunk_elems)
        flat[s:e] = (torch.randn(e - s, generator=gen, device=device,
                                 dtype=torch.float32) * std).to(torch.bfloat16)
    return out


def _unused_slots(layout: Layout):
    """(page, first_unused_slot) for every referenced page with unused slots,
    plus the list of pool pages no request references."""
    partial = []
    for r in range(layout.num_requests):
        T = int(layout.kv_len[r])
        if T % PAGE_SIZE:
            last = int(layout.page_indices[layout.page_indptr[r + 1] - 1])
            partial.append((last, T % PAGE_SIZE))
    used = np.zeros(layout.num_pages, dtype=bool)
    used[layout.page_indices] = True
    return partial, np.nonzero(~used)[0]


def make_attention_inputs(layout: Layout, device="cpu", *, poison: Optional[float] = None,
                          qk_std: Optional[float] = None) -> Dict[str, torch.Tensor]:
    """q, k_cache, v_cache for ``layout``.

    ``poison`` (e.g. NaN or 1e4) fills every cache slot no request may read:
    the unused tail slots of each request's last page and every unreferenced
    pool page.  ``qk_std`` overrides the q/k standard deviation (sharp-softmax
    variant); v keeps the spec's.
    """
    s = layout.spec
    std = s.qkv_std
    qk = std if qk_std is None else qk_std
    q = _randn((layout.total_q, s.num_q_heads, s.head_dim), qk, _gen(layout, device, 1), device)
    k = _randn((layout.num_pages, s.num_kv_heads, PAGE_SIZE, s.head_dim), qk,
               _gen(layout, device, 2), device)
    v = _randn((layout.num_pages, s.num_kv_heads, s.head_dim, PAGE_SIZE), std,
               _gen(layout, device, 3), device)
    if poison is not None:
        partial, unused = _unused_slots(layout)
        for page, first in partial:
            k[page, :, first:, :] = poison
            v[page, :, :, first:] = poison
        if len(unused):
            idx = torch.as_tensor(unused, device=device, dtype=torch.long)
            k[idx] = poison
            v[idx] = poison
    return dict(q=q, k_cache=k, v_cache=v)


def make_logit_inputs(layout: Layout, device="cpu", *, sigma: Optional[float] = None,
                      spike: Optional[float] = None, ties: bool = False) -> Dict[str, torch.Tensor]:
    """Verify logits, draft tokens and next-draft logits for ``layout``.

    Recipe: the previous block's draft logits are N(0, draft_std); the token
    each verify row judges is the first maximum of that row; the verify logits
    are those draft logits plus N(0, sigma_r) noise, so sigma sets how often
    the verifier agrees.  The next block's draft logits are an independent
    N(0, draft_std) draw.  ``spike`` adds a constant at one random position
    per row of both logit sets (peaked rows); ``ties`` copies each row's
    largest entry to a second position so the top value occurs twice.
    Appended bonus rows (``layout.bonus``) judge token -1.
    """
    s = layout.spec
    V = s.vocab
    rows = layout.total_verify_rows
    gen = _gen(layout, device, 4)
    prev = torch.randn((rows, V), generator=gen, device=device, dtype=torch.float32) * s.draft_std
    if spike is not None and rows:
        pos = torch.randint(0, V, (rows,), generator=gen, device=device)
        prev[torch.arange(rows, device=device), pos] += spike
    tokens = torch.argmax(prev.to(torch.bfloat16).float(), dim=1).to(torch.int32)
    sig = np.repeat(layout.sigma if sigma is None else np.full(layout.num_requests, sigma),
                    np.diff(layout.row_indptr))
    sig_t = torch.as_tensor(sig, device=device, dtype=torch.float32)[:, None]
    noise = torch.randn((rows, V), generator=gen, device=device, dtype=torch.float32)
    verify = (prev + noise * sig_t).to(torch.bfloat16)
    del prev, noise
    for r in range(layout.num_requests):
        if layout.bonus[r]:
            tokens[int(layout.row_indptr[r + 1]) - 1] = -1
    drows = layout.total_draft_rows
    g2 = _gen(layout, device, 5)
    draft = torch.randn((drows, V), generator=g2, device=device, dtype=torch.float32) * s.draft_std
    if spike is not None and drows:
        pos = torch.randint(0, V, (drows,), generator=g2, device=device)
        draft[torch.arange(drows, device=device), pos] += spike
    draft = draft.to(torch.bfloat16)
    if ties:
        for t in (verify, draft):
            if t.shape[0]:
                top = torch.argmax(t.float(), dim=1)
                other = (top + 1 + torch.randint(0, V - 1, top.shape, generator=g2,
                                                 device=device)) % V
                t[torch.arange(t.shape[0], device=device), other] = \
                    t[torch.arange(t.shape[0], device=device), top]
    return dict(verify_logits=verify, draft_tokens=tokens.contiguous(), draft_logits=draft)


def make_mask_probe(layout: Layout, device="cpu", *, score_gap: float = 45.0,
                    poison: Optional[float] = None) -> Dict[str, torch.Tensor]:
    """Attention inputs whose softmax weights are known in closed form.

    Every cached context key has a zero first component; every key of the
    request's new rows (verify and draft rows) is ``c * e_0``; every query is
    ``s * e_0``.  With ``sm_scale * s * c = score_gap`` the new-row keys a
    query may see outweigh the context keys by about exp(score_gap), and all
    of them score the same, so a query's output is the plain mean of the
    values of the new-row keys it may see.  Values stay random; ``poison``
    as in ``make_attention_inputs`` (slots no request may read keep it in
    every component but the first key component).
    """
    s = layout.spec
    base = make_attention_inputs(layout, device, poison=poison)
    q, k, v = base["q"], base["k_cache"], base["v_cache"]
    D = s.head_dim
    scale = 1.0 / math.sqrt(D)
    # s = c = power of two, so both are exact in bf16.
    mag = 2.0 ** math.ceil(0.5 * math.log2(score_gap / scale))
    q.zero_()
    q[:, :, 0] = mag
    k[:, :, :, 0] = 0.0
    pages, slots = new_row_slots(layout)
    if len(pages):
        pt = torch.as_tensor(pages, device=k.device)
        st = torch.as_tensor(slots, device=k.device)
        k[pt, :, st, :] = 0.0
        k[pt, :, st, 0] = mag
    return dict(q=q, k_cache=k, v_cache=v, probe_magnitude=torch.tensor(mag))


def new_row_slots(layout: Layout) -> Tuple[np.ndarray, np.ndarray]:
    """(page, slot) of every new-row key (positions L .. T-1 of each
    request), requests in order, positions ascending."""
    pages, slots = [], []
    for r in range(layout.num_requests):
        L, T = int(layout.ctx_len[r]), int(layout.kv_len[r])
        j = np.arange(L, T)
        pages.append(layout.page_indices[int(layout.page_indptr[r]) + j // PAGE_SIZE].astype(np.int64))
        slots.append(j % PAGE_SIZE)
    if not pages:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(pages), np.concatenate(slots).astype(np.int64)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """The raw bf16 bit patterns of a tensor as a host uint16 array."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
