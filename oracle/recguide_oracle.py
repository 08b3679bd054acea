"""Plain fp64 CPU oracle for the fused draft-verify step of RecGuide.

TEST INFRASTRUCTURE ONLY.  Nothing in the library calls, imports or links this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg
do.  It is deliberately slow and literal: explicit dense masks, whole-row
softmaxes, no blocking, no fusion, no reordering beyond the definitions below.

What it computes, and the passage each function follows:

* ``diffusion_mask`` / ``ar_mask`` -- the two attention masks of Eq. 1
  (Sec. 3.1), written out over 1-indexed positions.
* ``oracle_attention`` -- one fused draft-verify forward step's attention: the
  previous block's verify rows and the next draft block are query rows of the
  same request.  With the prefix set to context + verify rows and the draft
  set to the next block, Eq. 1's diffusion mask gives verify rows the causal
  (autoregressive) pattern and draft rows the whole prefix plus the whole
  block.  Softmax attention with that mask, grouped-query heads mapped
  contiguously (query head h uses KV head h // (Hq / Hkv)).
* ``oracle_accept`` -- greedy verification (Sec. 3.1, Sec. 6.1 uses greedy
  decoding): accept draft tokens up to the first position where the
  verifier's most likely token differs; the verifier's token there (or on a
  bonus row) is the next token; and the mean verifier entropy over the rows up
  to and including the first mismatch (the e_t of Sec. 5.2).
* ``oracle_confidence`` -- draft confidence C_i = P_1st(i) and top-2 margin
  M_i = P_1st(i) - P_2nd(i) (Sec. 4.1), plus the draft row's entropy.

Inputs are the raw bf16 bit patterns the GPU reads, decoded exactly to fp64.
Readings where the paper is silent (tie-breaking, log base, which rows enter
e_t, row alignment of tokens and verify logits) are listed with each function.

Pinned by tests/test_oracle_*.py against closed forms, brute force, library
routines and hand-written fixtures; no function here is "parity unpinned".
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np

PAGE_SIZE = 16


# --------------------------------------------------------------------------
# bf16 decoding
# --------------------------------------------------------------------------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of each bf16 bit pattern (uint16) as float64.

    A bf16 number is the upper half of an IEEE binary32, so shifting the bits
    into the high half of a 32-bit word and reading it as binary32 gives the
    value exactly; widening binary32 to binary64 is exact as well.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Eq. 1: attention masks
# --------------------------------------------------------------------------
def diffusion_mask(P: int, B: int, query_positions=None) -> np.ndarray:
    """Eq. 1 (left): additive mask over 1-indexed positions 1..P+B.

    Prefix positions {1..P} attend causally to the prefix; draft positions
    {P+1..P+B} attend to every prefix and draft position; everything else is
    -inf.  Rows are the query positions (all of 1..P+B unless
    ``query_positions`` lists a subset), columns the key positions 1..P+B.
    """
    N = P + B
    i = np.arange(1, N + 1) if query_positions is None else np.asarray(query_positions)
    i = i[:, None]
    j = np.arange(1, N + 1)[None, :]
    i_in_P, j_in_P = i <= P, j <= P
    i_in_D = (i > P) & (i <= N)
    j_in_PD = j <= N
    case1 = i_in_P & j_in_P & (j <= i)
    case2 = i_in_D & j_in_PD
    return np.where(case1 | case2, 0.0, -np.inf)


def ar_mask(N: int) -> np.ndarray:
    """Eq. 1 (right): additive mask over positions 1..N, 0 iff j <= i."""
    i = np.arange(1, N + 1)[:, None]
    j = np.arange(1, N + 1)[None, :]
    return np.where(j <= i, 0.0, -np.inf)


def fused_step_mask(ctx_len: int, n_verify: int, n_draft: int) -> np.ndarray:
    """Additive mask of one request's query rows in the fused step.

    The cached context (ctx_len tokens) and the previous block's verify rows
    form the prefix of Eq. 1 (P = ctx_len + n_verify); the next draft block
    is the draft set (B = n_draft).  Only the new tokens (positions
    ctx_len+1 .. P+B) are queries; all P + B positions are keys.
    """
    P = ctx_len + n_verify
    return diffusion_mask(P, n_draft, np.arange(ctx_len + 1, P + n_draft + 1))


# --------------------------------------------------------------------------
# Attention
# --------------------------------------------------------------------------
def gather_request_kv(k_bits: np.ndarray, v_bits: np.ndarray, page_indices: np.ndarray,
                      page_start: int, kv_len: int, kv_head: int) -> Tuple[np.ndarray, np.ndarray]:
    """Keys and values of one request and KV head, in token order.

    Cache layouts: k [pages, Hkv, 16, D] (token-major pages) and
    v [pages, Hkv, D, 16] (dimension-major pages).  Token j of the request
    lives in slot j % 16 of page page_indices[page_start + j // 16].
    """
    j = np.arange(kv_len)
    pages = np.asarray(page_indices)[page_start + j // PAGE_SIZE].astype(np.int64)
    slots = j % PAGE_SIZE
    K = bf16_bits_to_f64(k_bits[pages, kv_head, slots, :])
    V = bf16_bits_to_f64(v_bits[pages, kv_head, :, slots])
    return K, V


def softmax_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, mask: np.ndarray,
                      scale: float) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """softmax(scale * q K^T + mask) V for one head.

    Returns (out [n, D], lse [n] natural log, probabilities [n, T]).
    """
    s = scale * (q @ K.T) + mask
    mx = s.max(axis=1, keepdims=True)
    e = np.exp(s - mx)
    z = e.sum(axis=1, keepdims=True)
    p = e / z
    return p @ V, (mx + np.log(z))[:, 0], p


def oracle_attention(q_bits: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray,
                     q_indptr: np.ndarray, n_verify: np.ndarray, ctx_len: np.ndarray,
                     page_indptr: np.ndarray, page_indices: np.ndarray,
                     sm_scale: Optional[float] = None,
                     requests=None, heads=None) -> Dict[str, np.ndarray]:
    """Fused draft-verify attention over a paged cache, fp64.

    q [sum n, Hq, D] bf16 bits; request r owns query rows
    q_indptr[r]..q_indptr[r+1]; the first n_verify[r] are verify rows, the
    rest the next draft block.  The request's keys are its ctx_len[r] cached
    tokens followed by its n_r new tokens (already in the pages).

    Readings: softmax scale 1/sqrt(D) unless given; query head h reads KV
    head h // (Hq / Hkv).  ``requests`` / ``heads`` restrict the work to a
    subset (other outputs stay NaN) for sampled checks on large inputs.

    Returns out [sum n, Hq, D] and lse [sum n, Hq] (natural log), fp64.
    """
    total, Hq, D = q_bits.shape
    Hkv = k_bits.shape[1]
    g = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if sm_scale is None or sm_scale <= 0 else float(sm_scale)
    out = np.full((total, Hq, D), np.nan)
    lse = np.full((total, Hq), np.nan)
    R = len(ctx_len)
    for r in (range(R) if requests is None else requests):
        q0, q1 = int(q_indptr[r]), int(q_indptr[r + 1])
        n = q1 - q0
        if n == 0:
            continue
        L = int(ctx_len[r])
        T = L + n
        mask = fused_step_mask(L, int(n_verify[r]), n - int(n_verify[r]))
        for h in (range(Hq) if heads is None else heads):
            K, V = gather_request_kv(k_bits, v_bits, page_indices, int(page_indptr[r]), T, h // g)
            qh = bf16_bits_to_f64(q_bits[q0:q1, h, :])
            o, l, _ = softmax_attention(qh, K, V, mask, scale)
            out[q0:q1, h, :] = o
            lse[q0:q1, h] = l
    return dict(out=out, lse=lse)


# --------------------------------------------------------------------------
# Row statistics shared by verification and drafting
# --------------------------------------------------------------------------
def first_argmax(x: np.ndarray) -> int:
    """Lowest index holding the row maximum (ties broken to the lowest index)."""
    return int(np.argmax(x))


def softmax_row(x: np.ndarray) -> np.ndarray:
    e = np.exp(x - x.max())
    return e / e.sum()


def entropy_row(x: np.ndarray) -> float:
    """Shannon entropy (natural log) of softmax(x), with 0 * log 0 = 0.

    Evaluated as -sum p_v ln p_v with the log-probabilities taken from the
    log-softmax identity ln p_v = (x_v - m) - ln Z, Z = sum_u exp(x_u - m),
    m = max x.  Since the maximal entry contributes exactly 1 to Z, ln Z is
    log1p of the sum over the other entries; this keeps fp64's relative
    accuracy on sharply peaked rows, where forming p_top = 1 - tiny first
    would lose it.
    """
    top = first_argmax(x)
    d = x - x[top]
    rest = np.exp(np.delete(d, top)).sum()
    log_z = np.log1p(rest)
    logp = d - log_z
    p = np.exp(logp)
    nz = p > 0
    return float(-(p[nz] * logp[nz]).sum())


# --------------------------------------------------------------------------
# Verification and acceptance
# --------------------------------------------------------------------------
def oracle_accept(verify_bits: np.ndarray, row_indptr: np.ndarray,
                  draft_tokens: np.ndarray) -> Dict[str, np.ndarray]:
    """Greedy verification of each request's draft tokens.

    verify_bits [rows, vocab] bf16 bits; request r owns rows
    row_indptr[r]..row_indptr[r+1].  Verify row k judges draft_tokens[k]
    (row-aligned); a negative token marks a bonus row that never matches.

    Per row: argmax (lowest index on ties) and entropy of softmax.
    Per request with V rows:
      accept_len = first k < V whose argmax differs from its token, else V;
      next_token = argmax of that row, or -1 if every row matched;
      accept_entropy = mean row entropy over rows 0..min(accept_len, V-1)
        (reading of "excluding those after the first mismatch": the
        mismatching row itself is causally valid and is kept);
      a request with no rows gets (0, -1, 0.0).
    """
    rows = verify_bits.shape[0]
    x = bf16_bits_to_f64(verify_bits)
    am = np.array([first_argmax(x[k]) for k in range(rows)], dtype=np.int64)
    ent = np.array([entropy_row(x[k]) for k in range(rows)], dtype=np.float64)
    R = len(row_indptr) - 1
    acc = np.zeros(R, dtype=np.int64)
    nxt = np.full(R, -1, dtype=np.int64)
    e_t = np.zeros(R, dtype=np.float64)
    for r in range(R):
        k0, k1 = int(row_indptr[r]), int(row_indptr[r + 1])
        V = k1 - k0
        if V == 0:
            continue
        a = V
        for i in range(V):
            tok = int(draft_tokens[k0 + i])
            if tok < 0 or am[k0 + i] != tok:
                a = i
                break
        acc[r] = a
        nxt[r] = am[k0 + a] if a < V else -1
        last = min(a, V - 1)
        e_t[r] = ent[k0:k0 + last + 1].mean()
    return dict(row_argmax=am, row_entropy=ent, accept_len=acc, next_token=nxt,
                accept_entropy=e_t)


# --------------------------------------------------------------------------
# Draft confidence
# --------------------------------------------------------------------------
def oracle_confidence(draft_bits: np.ndarray) -> Dict[str, np.ndarray]:
    """Per draft row: C = P_1st, M = P_1st - P_2nd (Sec. 4.1) and entropy.

    top1 = lowest index of the maximum; top2 = lowest index of the maximum
    over the remaining entries (so with a tie at the top, top2 is the second
    tied index and P_2nd = P_1st).  Probabilities are softmax at temperature 1.
    """
    rows = draft_bits.shape[0]
    x = bf16_bits_to_f64(draft_bits)
    t1 = np.zeros(rows, dtype=np.int64)
    t2 = np.zeros(rows, dtype=np.int64)
    p1 = np.zeros(rows)
    p2 = np.zeros(rows)
    ent = np.zeros(rows)
    for k in range(rows):
        row = x[k]
        a = first_argmax(row)
        rest = row.copy()
        rest[a] = -np.inf
        b = first_argmax(rest)
        p = softmax_row(row)
        t1[k], t2[k] = a, b
        p1[k], p2[k] = p[a], p[b]
        ent[k] = entropy_row(row)
    return dict(top1=t1, top2=t2, p1=p1, p2=p2, margin=p1 - p2, entropy=ent)
