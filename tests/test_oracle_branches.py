"""Pins for the oracle of the predictive draft-verify overlap (CPU only).

The branch attention is checked against a hand-written mask fixture, against
the already pinned single-branch step (a request with no listed branches, or
one continuation branch, is exactly the fused step), against the plain step
recomputed on each branch's own gathered sequence (an independent data path:
the branch's keys re-laid into a fresh page pool), and against isolation
invariants.  Branch planning and reuse matching are checked on hand-made
cases that cover each rule of Sec. 5.1.
"""
import os

import numpy as np
import pytest

from oracle import (branch_step_mask, fused_step_mask, oracle_attention, oracle_branch_attention,
                    oracle_match_branches, oracle_plan_branches, request_branches)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
PS = 16


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest even) and return the bit patterns."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _fixture(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#") and not line[0].isalpha():
                rows.append([int(t) for t in line.split()])
    return np.array(rows)


def test_mask_matches_hand_written_fixture():
    m = branch_step_mask(2, 2, [(1, 1, 2), (2, 0, 2)])
    want = _fixture("branch_mask_L2_V2.txt")
    np.testing.assert_array_equal(np.isfinite(m).astype(int), want)
    assert set(np.unique(m[np.isfinite(m)])) == {0.0}


@pytest.mark.parametrize("L,V,B", [(0, 0, 3), (5, 3, 0), (37, 4, 9), (16, 16, 16), (1, 7, 1)])
def test_default_and_single_continuation_are_the_fused_step(L, V, B):
    want = fused_step_mask(L, V, B)
    got = branch_step_mask(L, V, request_branches(V + B, V, []))
    np.testing.assert_array_equal(got, want)
    if B:
        np.testing.assert_array_equal(branch_step_mask(L, V, [(V, 0, B)]), want)


def _random_case(rng, L, V, branches, Hq=4, Hkv=2, D=16, spare=3):
    n = V + sum(b[2] for b in branches)
    T = L + n
    pages = -(-T // PS)
    pool = pages + spare
    perm = rng.permutation(pool)[:pages].astype(np.int32)
    q = _bf16_bits(rng.standard_normal((n, Hq, D)) * 0.7)
    k = _bf16_bits(rng.standard_normal((pool, Hkv, PS, D)) * 0.7)
    v = _bf16_bits(rng.standard_normal((pool, Hkv, D, PS)))
    return dict(q=q, k=k, v=v, perm=perm, n=n, T=T, pages=pages)


def _token_kv(c, j, h):
    page, slot = c["perm"][j // PS], j % PS
    return c["k"][page, h, slot, :], c["v"][page, h, :, slot]


@pytest.mark.parametrize("seed,L,V,branches", [
    (0, 37, 5, [(2, 1, 4), (5, 0, 3), (0, 1, 2)]),
    (1, 0, 3, [(3, 0, 5), (1, 1, 1)]),
    (2, 20, 0, [(0, 0, 6), (0, 1, 3)]),
    (3, 70, 8, [(8, 0, 9)]),
])
def test_each_branch_equals_the_plain_step_on_its_own_sequence(seed, L, V, branches):
    """Branch b's rows, recomputed by the plain fused-step oracle on a request
    whose context is the kept canonical prefix, whose verify rows are the
    branch's lead rows and whose draft block is the rest of the branch --
    with every key copied into a fresh, identity-mapped page pool."""
    rng = np.random.default_rng(seed)
    c = _random_case(rng, L, V, branches)
    Hq, Hkv, D = c["q"].shape[1], c["k"].shape[1], c["q"].shape[2]
    res = oracle_branch_attention(c["q"], c["k"], c["v"], np.array([0, c["n"]]), np.array([V]),
                                  np.array([L]), np.array([0, c["pages"]]), c["perm"], [branches])
    row, key = V, L + V
    for prefix, lead, rows in branches:
        keys = list(range(L + prefix)) + list(range(key, key + rows))
        T2 = len(keys)
        pages2 = -(-T2 // PS)
        k2 = np.zeros((pages2, Hkv, PS, D), dtype=np.uint16)
        v2 = np.zeros((pages2, Hkv, D, PS), dtype=np.uint16)
        for t, j in enumerate(keys):
            for h in range(Hkv):
                kk, vv = _token_kv(c, j, h)
                k2[t // PS, h, t % PS, :] = kk
                v2[t // PS, h, :, t % PS] = vv
        ref = oracle_attention(c["q"][row:row + rows], k2, v2, np.array([0, rows]), np.array([lead]),
                               np.array([L + prefix]), np.array([0, pages2]), np.arange(pages2, dtype=np.int32))
        np.testing.assert_allclose(res["out"][row:row + rows], ref["out"], rtol=0, atol=1e-12)
        np.testing.assert_allclose(res["lse"][row:row + rows], ref["lse"], rtol=0, atol=1e-12)
        row += rows
        key += rows
    # verify rows: the plain step with no draft rows
    if V:
        ref = oracle_attention(c["q"][:V], c["k"], c["v"], np.array([0, V]), np.array([V]), np.array([L]),
                               np.array([0, c["pages"]]), c["perm"])
        np.testing.assert_allclose(res["out"][:V], ref["out"], rtol=0, atol=1e-12)


def test_branches_are_isolated():
    """Changing one branch's keys and values, or the verify rows past a
    branch's prefix, leaves the other rows' outputs unchanged."""
    rng = np.random.default_rng(7)
    L, V = 25, 6
    branches = [(2, 1, 3), (6, 0, 4)]
    c = _random_case(rng, L, V, branches)
    args = lambda cc: (cc["q"], cc["k"], cc["v"], np.array([0, cc["n"]]), np.array([V]), np.array([L]),
                       np.array([0, cc["pages"]]), cc["perm"], [branches])
    base = oracle_branch_attention(*args(c))["out"]
    # perturb branch 1's rows (keys L+V+3 .. L+V+6)
    c2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
    for j in range(L + V + 3, L + V + 7):
        page, slot = c["perm"][j // PS], j % PS
        c2["k"][page, :, slot, :] = _bf16_bits(rng.standard_normal(c["k"][page, :, slot, :].shape))
        c2["v"][page, :, :, slot] = _bf16_bits(rng.standard_normal(c["v"][page, :, :, slot].shape))
    out2 = oracle_branch_attention(*args(c2))["out"]
    np.testing.assert_array_equal(out2[:V + 3], base[:V + 3])      # verify rows and branch 0
    assert not np.allclose(out2[V + 3:], base[V + 3:])              # branch 1 does see them
    # perturb verify rows 2..5 (past branch 0's prefix of 2)
    c3 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
    for j in range(L + 2, L + V):
        page, slot = c["perm"][j // PS], j % PS
        c3["k"][page, :, slot, :] = _bf16_bits(rng.standard_normal(c["k"][page, :, slot, :].shape))
        c3["v"][page, :, :, slot] = _bf16_bits(rng.standard_normal(c["v"][page, :, :, slot].shape))
    out3 = oracle_branch_attention(*args(c3))["out"]
    np.testing.assert_array_equal(out3[:2], base[:2])               # verify rows 0, 1 are causal
    np.testing.assert_array_equal(out3[V:V + 3], base[V:V + 3])     # branch 0 keeps only 2 verify rows


def test_draft_rows_of_a_branch_are_permutation_equivariant():
    """Permuting a branch's draft rows jointly (q, k, v) permutes their
    outputs (they form Eq. 1's bidirectional draft set)."""
    rng = np.random.default_rng(9)
    L, V = 18, 3
    branches = [(1, 1, 5)]
    c = _random_case(rng, L, V, branches)
    res = oracle_branch_attention(c["q"], c["k"], c["v"], np.array([0, c["n"]]), np.array([V]), np.array([L]),
                                  np.array([0, c["pages"]]), c["perm"], [branches])["out"]
    draft = np.arange(V + 1, V + 5)            # the branch's rows after its lead row
    p = rng.permutation(len(draft))
    c2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
    c2["q"][draft] = c["q"][draft[p]]
    for a, b in zip(draft, draft[p]):
        ja, jb = L + a, L + b
        pa, sa, pb, sb = c["perm"][ja // PS], ja % PS, c["perm"][jb // PS], jb % PS
        c2["k"][pa, :, sa, :] = c["k"][pb, :, sb, :]
        c2["v"][pa, :, :, sa] = c["v"][pb, :, :, sb]
    res2 = oracle_branch_attention(c2["q"], c2["k"], c2["v"], np.array([0, c["n"]]), np.array([V]),
                                   np.array([L]), np.array([0, c["pages"]]), c["perm"], [branches])["out"]
    np.testing.assert_allclose(res2[draft], res[draft[p]], rtol=0, atol=1e-12)
    np.testing.assert_allclose(res2[:V + 1], res[:V + 1], rtol=0, atol=1e-12)


def test_plan_branches_rules():
    delta = np.float32(0.5)
    margin = np.array([0.9, 0.4, 0.7, 0.2, 0.1,      # request 0: risky 1, 3, 4 (three)
                       0.6, 0.5, 0.49,               # request 1: risky 2 only (0.5 is not < 0.5)
                       0.8, 0.9,                     # request 2: none
                       0.3, 0.3],                    # request 3: risky 0, 1 (two)
                      dtype=np.float32)
    top2 = np.arange(100, 100 + len(margin))
    rp = np.array([0, 5, 8, 10, 12, 12])             # request 4 is empty
    res = oracle_plan_branches(margin, top2, rp, delta)
    np.testing.assert_array_equal(res["n_risky"], [3, 1, 0, 2, 0])
    np.testing.assert_array_equal(res["n_corr"], [2, 1, 0, 2, 0])
    np.testing.assert_array_equal(res["corr_pos"], [[1, 3], [2, -1], [-1, -1], [0, 1], [-1, -1]])
    np.testing.assert_array_equal(res["corr_tok"], [[101, 103], [107, -1], [-1, -1], [110, 111], [-1, -1]])
    np.testing.assert_array_equal(res["continuation"], [0, 1, 1, 1, 1])


def test_match_branches_rules():
    n_corr = np.array([2, 2, 2, 1, 0, 2])
    corr_pos = np.array([[1, 3], [1, 3], [1, 3], [0, -1], [-1, -1], [1, 3]])
    corr_tok = np.array([[7, 9], [7, 9], [7, 9], [5, -1], [-1, -1], [7, 9]])
    cont = np.array([0, 1, 1, 1, 1, 1])
    cont_first = np.array([4, 4, 4, 4, 4, 4])
    block_len = np.array([5, 5, 5, 6, 4, 5])
    accept = np.array([3, 1, 5, 6, 4, 3])
    nxt = np.array([9, 8, 4, 4, 3, 8])
    got = oracle_match_branches(accept, nxt, block_len, n_corr, corr_pos, corr_tok, cont, cont_first)
    # 0: rejected at 3 with token 9 -> correction branch 1
    # 1: rejected at 1 but token 8 != 7 -> none
    # 2: all accepted, bonus 4 == continuation's first token -> continuation (index 2)
    # 3: all 6 accepted, bonus 4 == 4 -> continuation (index 1)
    # 4: all accepted, bonus 3 != 4 -> none
    # 5: rejected at 3 with token 8 != 9 -> none
    np.testing.assert_array_equal(got, [1, -1, 2, 1, -1, -1])
