"""fp64 / integer CPU oracle for the predictive draft-verify overlap.

TEST INFRASTRUCTURE ONLY, like the rest of this package: nothing in the
library imports or calls it.

Sec. 5.1 prepares, next to a round's verification, drafts for the next round
under hypothetical outcomes of that verification: a correction branch for
each of the earliest two positions whose draft margin M_i = P_1st - P_2nd
(Sec. 4.1) is below delta -- the draft token there replaced by its second
candidate -- and, when at most two positions are risky, a continuation
branch that assumes the whole block is accepted.  Sec. 5.3 serves all
branches in one pass that reads the canonical prefix's KV once and processes
only valid query tokens.  A branch is reused only if the verifier rejects
exactly at its position with the same replacement token (correction) or
accepts the whole block and the branch's first token equals the verifier's
bonus token (continuation).

Functions and the passage each follows:

* ``branch_step_mask`` / ``oracle_branch_attention`` -- the attention of one
  step whose query rows are the verify rows and the rows of every branch.
  A branch's own sequence is the canonical prefix it keeps (the context and
  its first ``prefix`` verify rows) followed by its rows; on that sequence
  Eq. 1's diffusion mask applies, with the branch's ``lead`` committed rows
  (a correction token) in the prefix set and its remaining rows in the draft
  set.  Verify rows keep the autoregressive pattern over context + verify
  rows.  Branch rows never see other branches' rows nor the verify rows past
  their prefix.
* ``oracle_plan_branches`` -- risky positions and the branches of Sec. 5.1.
* ``oracle_match_branches`` -- the reuse rule of Sec. 5.1.

Readings (the paper is silent on them): the key order of a request is
context, verify rows, then each branch's rows in branch order (the order the
caller writes their K/V into the request's pages); a request listed with no
branches treats its rows after the verify rows as one continuation block
(prefix = all verify rows, no committed lead rows), which is the fused step
of ``oracle_attention``; ``M_i < delta`` is strict; the continuation branch
is prepared when the block has at most two risky positions in total;
corrections come first (by position), the continuation last.

Pinned by tests/test_oracle_branches.py.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .recguide_oracle import (bf16_bits_to_f64, diffusion_mask, fused_step_mask,
                              gather_request_kv, softmax_attention)

Branch = Tuple[int, int, int]  # (prefix verify rows kept, committed lead rows, rows)


def request_branches(n_rows: int, n_verify: int, branches: Sequence[Branch]) -> List[Branch]:
    """The branches of one request, the default continuation block included.

    With no branches listed, the rows after the verify rows (if any) form one
    continuation block: prefix = n_verify, lead = 0.
    """
    if len(branches) == 0:
        rest = n_rows - n_verify
        return [(n_verify, 0, rest)] if rest > 0 else []
    return [tuple(int(v) for v in b) for b in branches]


def branch_step_mask(ctx_len: int, n_verify: int, branches: Sequence[Branch]) -> np.ndarray:
    """Additive mask [rows, keys] of one request with overlap branches.

    Keys: ctx_len context tokens, n_verify verify rows, then each branch's
    rows.  Rows: the verify rows, then each branch's rows.
    """
    L, V = int(ctx_len), int(n_verify)
    total = V + sum(b[2] for b in branches)
    T = L + total
    mask = np.full((total, T), -np.inf)
    # verify rows: Eq. 1 with the whole context + verify rows as the prefix
    # and no draft set, i.e. the autoregressive pattern
    if V:
        mask[:V, :L + V] = fused_step_mask(L, V, 0)
    row, key = V, L + V
    for prefix, lead, rows in branches:
        # Eq. 1 on the branch's own sequence: prefix set = context, the kept
        # verify rows and the committed lead rows; draft set = the rest.
        P = L + prefix + lead
        own = diffusion_mask(P, rows - lead, np.arange(L + prefix + 1, L + prefix + rows + 1))
        mask[row:row + rows, :L + prefix] = own[:, :L + prefix]
        mask[row:row + rows, key:key + rows] = own[:, L + prefix:]
        row += rows
        key += rows
    return mask


def oracle_branch_attention(q_bits: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray,
                            q_indptr: np.ndarray, n_verify: np.ndarray, ctx_len: np.ndarray,
                            page_indptr: np.ndarray, page_indices: np.ndarray,
                            branches: Sequence[Sequence[Branch]],
                            sm_scale: Optional[float] = None,
                            requests=None, heads=None) -> Dict[str, np.ndarray]:
    """Attention of a step with overlap branches, fp64 (layouts as in
    ``oracle_attention``; ``branches[r]`` lists request r's branches)."""
    total, Hq, D = q_bits.shape
    Hkv = k_bits.shape[1]
    g = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if sm_scale is None or sm_scale <= 0 else float(sm_scale)
    out = np.full((total, Hq, D), np.nan)
    lse = np.full((total, Hq), np.nan)
    for r in (range(len(ctx_len)) if requests is None else requests):
        q0, q1 = int(q_indptr[r]), int(q_indptr[r + 1])
        n = q1 - q0
        if n == 0:
            continue
        L, V = int(ctx_len[r]), int(n_verify[r])
        br = request_branches(n, V, branches[r])
        mask = branch_step_mask(L, V, br)
        assert mask.shape == (n, L + n)
        for h in (range(Hq) if heads is None else heads):
            K, Vv = gather_request_kv(k_bits, v_bits, page_indices, int(page_indptr[r]), L + n, h // g)
            o, l, _ = softmax_attention(bf16_bits_to_f64(q_bits[q0:q1, h, :]), K, Vv, mask, scale)
            out[q0:q1, h, :] = o
            lse[q0:q1, h] = l
    return dict(out=out, lse=lse)


def oracle_plan_branches(margin: np.ndarray, top2: np.ndarray, row_indptr: np.ndarray,
                         delta: float, max_risky: int = 2) -> Dict[str, np.ndarray]:
    """Branches of Sec. 5.1 for each request's draft block.

    margin, top2: per draft row (the block being verified, rows
    row_indptr[r] .. row_indptr[r+1]-1 at positions 0, 1, ...), as draft
    confidence produced them.  Positions with margin < delta are risky; the
    earliest ``max_risky`` each give a correction branch (position, top2
    token there); a continuation branch is prepared when the block has at
    most ``max_risky`` risky positions.
    """
    margin = np.asarray(margin)
    R = len(row_indptr) - 1
    pos = np.full((R, max_risky), -1, dtype=np.int64)
    tok = np.full((R, max_risky), -1, dtype=np.int64)
    n_corr = np.zeros(R, dtype=np.int64)
    n_risky = np.zeros(R, dtype=np.int64)
    cont = np.zeros(R, dtype=np.int64)
    for r in range(R):
        k0, k1 = int(row_indptr[r]), int(row_indptr[r + 1])
        risky = [i for i in range(k1 - k0) if margin[k0 + i] < delta]
        n_risky[r] = len(risky)
        for c, i in enumerate(risky[:max_risky]):
            pos[r, c] = i
            tok[r, c] = int(top2[k0 + i])
        n_corr[r] = min(len(risky), max_risky)
        cont[r] = 1 if len(risky) <= max_risky else 0
    return dict(n_corr=n_corr, corr_pos=pos, corr_tok=tok, n_risky=n_risky, continuation=cont)


def oracle_match_branches(accept_len: np.ndarray, next_token: np.ndarray, block_len: np.ndarray,
                          n_corr: np.ndarray, corr_pos: np.ndarray, corr_tok: np.ndarray,
                          continuation: np.ndarray, cont_first: np.ndarray) -> np.ndarray:
    """Which prepared branch the verification outcome confirms (Sec. 5.1).

    A correction branch at position i is reused iff the verifier accepted
    exactly i tokens and its token there (next_token) is the branch's
    replacement; the continuation branch iff all block_len tokens were
    accepted and the verifier's bonus token (next_token) equals the
    branch's first token.  Returns, per request, the branch's index in the
    request's branch order (corrections by position, then the continuation)
    or -1.
    """
    R = len(accept_len)
    out = np.full(R, -1, dtype=np.int64)
    for r in range(R):
        a, nt = int(accept_len[r]), int(next_token[r])
        for c in range(int(n_corr[r])):
            if a == int(corr_pos[r, c]) and nt == int(corr_tok[r, c]):
                out[r] = c
        if continuation[r] and a == int(block_len[r]) and nt == int(cont_first[r]):
            out[r] = int(n_corr[r])
    return out
