"""CPU oracle for verification-guided block sizing and block-size bucketing.

TEST INFRASTRUCTURE ONLY, like the rest of this package: nothing in the
library imports or calls it.

Sec. 5.2 picks each request's next draft block size from the history of its
verification rounds.  The state (Eq. 2) is

    s_t = -(e_{t-1} + e_{t-2}) / 2,        z_t = (B_{t-1}, F_{t-1}),

with e the mean verifier entropy of a round over its causally valid rows up to
the first mismatch (``oracle_accept``'s e_t), B_{t-1} the size of the block
just verified and F_{t-1} whether it was accepted in full.  The decision
(Eq. 3) is the candidate B maximising V_B(s_t, z_t) - rho_C * T_C(B): a table
of expected accepted progress (calibrated offline) minus the weighted profiled
cost of a block of size B at the current load.  Sec. 5.3 then groups the
requests by planned block size (block-size bucketed serving).

Functions and the passage each follows:

* ``oracle_block_state``  -- Eq. 2 for one request.
* ``oracle_utilities``    -- the objective of Eq. 3 for every candidate.
* ``oracle_route``        -- Eq. 3 for one request, by table lookup.
* ``oracle_bucket``       -- the grouping of Sec. 5.3.
* ``oracle_plan_block_sizes`` -- one round of the three for a batch, with the
  entropy history shifted by one round.

Precision: s_t and every utility are computed in float64 from the exact
values of the inputs (the entropies, table entries, costs and rho arrive as
float32 numbers; each is widened exactly).  With no more than one rounding
per operation in float64 these are the real-number definitions of Eq. 2-3 to
within 2^-52 relative, so the decisions here are the definition's decisions
except where two utilities (or s and a bin edge) are closer than that.  A
GPU path that evaluates the same formulas in float32 may take the other side
of a closer call than its own rounding bound; the parity tests accept either
candidate exactly there (see ``oracle_utilities``).

Readings (the paper is silent on them):

- the table's s axis is cut into bins by ascending edges: bin k holds
  edges[k-1] <= s < edges[k] (bin 0 everything below edges[0], the last bin
  everything at or above the last edge);
- z's block size is looked up among the candidates: the largest candidate not
  above B_{t-1}, or the smallest candidate when B_{t-1} is below all of them;
  F_{t-1} = 1 iff the accepted length reached B_{t-1};
- ties in Eq. 3 go to the smaller block (a larger block has to pay for itself,
  Sec. 5.2), i.e. the first maximum over ascending candidates;
- bucketing is a stable sort of the request indices by planned block size
  (ascending), with the start of each candidate's bucket;
- the history update replaces e_{t-2} by e_{t-1} for the next round; the
  caller seeds the history of a new request (e.g. with its first round's
  entropy).

Pinned by tests/test_oracle_blocksize.py.
"""
from __future__ import annotations

from typing import Dict, Sequence, Tuple

import numpy as np


def oracle_block_state(e_prev1: float, e_prev2: float, prev_block: int, accept_len: int,
                       candidates: Sequence[int]) -> Tuple[float, int, int]:
    """(s_t, index of B_{t-1} among the candidates, F_{t-1}) of Eq. 2, s_t in
    float64."""
    s = -(float(e_prev1) + float(e_prev2)) / 2.0
    zb = 0
    for i, c in enumerate(candidates):
        if int(c) <= int(prev_block):
            zb = i
    full = 1 if int(accept_len) >= int(prev_block) else 0
    return s, zb, full


def s_bin(s: float, edges: Sequence[float]) -> int:
    """Bin of s: the number of edges at or below it."""
    k = 0
    for e in edges:
        if float(e) <= float(s):
            k += 1
    return k


def oracle_utilities(s: float, zb: int, full: int, candidates: Sequence[int], edges: Sequence[float],
                     value: np.ndarray, cost: Sequence[float], rho: float) -> Tuple[int, np.ndarray]:
    """The bin of s and V_B(s, z) - rho * T_C(B) of Eq. 3 for every candidate
    B, in float64: utility[b] = value[b, bin(s), zb, full] - rho * cost[b]."""
    k = s_bin(s, edges)
    u = np.array([float(value[b, k, zb, full]) - float(rho) * float(cost[b]) for b in range(len(candidates))],
                 dtype=np.float64)
    return k, u


def oracle_route(s: float, zb: int, full: int, candidates: Sequence[int], edges: Sequence[float],
                 value: np.ndarray, cost: Sequence[float], rho: float) -> int:
    """B_t of Eq. 3: the first candidate (the smallest block) maximising the
    utility of ``oracle_utilities``."""
    _, u = oracle_utilities(s, zb, full, candidates, edges, value, cost, rho)
    best = 0
    for b in range(1, len(candidates)):
        if u[b] > u[best]:
            best = b
    return int(candidates[best])


def oracle_bucket(next_block: Sequence[int], candidates: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Requests grouped by planned block size (ascending, stable): the order
    and the start of each candidate's bucket (len(candidates) + 1 entries)."""
    R = len(next_block)
    order = []
    offsets = [0]
    for c in candidates:
        for r in range(R):
            if int(next_block[r]) == int(c):
                order.append(r)
        offsets.append(len(order))
    return np.array(order, dtype=np.int64), np.array(offsets, dtype=np.int64)


def oracle_plan_block_sizes(accept_len: np.ndarray, accept_entropy: np.ndarray, prev_block: np.ndarray,
                            entropy_hist: np.ndarray, candidates: Sequence[int], edges: Sequence[float],
                            value: np.ndarray, cost: Sequence[float], rho: float) -> Dict[str, np.ndarray]:
    """One round for a batch.  accept_entropy[r] is e_{t-1} (the round just
    verified), entropy_hist[r] is e_{t-2}; returns next_block (B_t), the new
    history (e_{t-1}, the same numbers), the bucketing of next_block, and per
    request the state s_t and bin used (``s``, ``bin``) and the utilities of
    every candidate (``utility`` [R, NB]), all float64."""
    R = len(accept_len)
    nb = np.zeros(R, dtype=np.int64)
    s_all = np.zeros(R, dtype=np.float64)
    bins = np.zeros(R, dtype=np.int64)
    util = np.zeros((R, len(candidates)), dtype=np.float64)
    for r in range(R):
        s, zb, full = oracle_block_state(accept_entropy[r], entropy_hist[r], prev_block[r], accept_len[r],
                                         candidates)
        nb[r] = oracle_route(s, zb, full, candidates, edges, value, cost, rho)
        bins[r], util[r] = oracle_utilities(s, zb, full, candidates, edges, value, cost, rho)
        s_all[r] = s
    order, offsets = oracle_bucket(nb, candidates)
    return dict(next_block=nb, entropy_hist=np.asarray(accept_entropy, dtype=np.float32).copy(),
                order=order, bucket_offsets=offsets, s=s_all, bin=bins, utility=util)
