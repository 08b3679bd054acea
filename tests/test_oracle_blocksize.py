"""Pins for the oracle of verification-guided block sizing and bucketing
(Sec. 5.2 Eq. 2 and 3, Sec. 5.3), CPU only.

Hand-made cases with answers worked out by hand cover each rule: the state of
Eq. 2 in closed form, the bin lookup at and between edges, the block-size
index of z and the full-acceptance flag, the argmax of Eq. 3 with its tie
rule, and the cost term's sign and weight.  Bucketing is checked against
Python's stable sort and against the definition on every small input.
"""
import itertools

import numpy as np
import pytest

from oracle import (oracle_block_state, oracle_bucket, oracle_plan_block_sizes, oracle_route,
                    oracle_utilities, s_bin)

CAND = [8, 16, 32]


def test_state_closed_form():
    s, zb, full = oracle_block_state(1.0, 3.0, 16, 16, CAND)
    assert s == np.float32(-2.0) and zb == 1 and full == 1
    s, zb, full = oracle_block_state(0.25, 0.5, 32, 7, CAND)
    assert s == np.float32(-0.375) and zb == 2 and full == 0
    # the definition's real-number mean: the sum is not rounded to float32
    # (in float32 1 + 2^-24 rounds to 1 and s would be -0.5)
    s, _, _ = oracle_block_state(np.float32(1.0), np.float32(2.0 ** -24), 8, 0, CAND)
    assert s == -(0.5 + 2.0 ** -25)


@pytest.mark.parametrize("prev,want", [(8, 0), (12, 0), (16, 1), (31, 1), (32, 2), (64, 2), (4, 0), (0, 0)])
def test_block_index_of_z(prev, want):
    assert oracle_block_state(0.0, 0.0, prev, 0, CAND)[1] == want


@pytest.mark.parametrize("accept,prev,want", [(0, 8, 0), (7, 8, 0), (8, 8, 1), (9, 8, 1), (0, 0, 1)])
def test_full_acceptance_flag(accept, prev, want):
    assert oracle_block_state(0.0, 0.0, prev, accept, CAND)[2] == want


@pytest.mark.parametrize("s,want", [(-10.0, 0), (-1.0, 1), (-0.75, 1), (-0.5, 2), (0.0, 2), (-1.5, 0)])
def test_bins(s, want):
    # edges -1.0 and -0.5: bin 0 below -1, bin 1 in [-1, -0.5), bin 2 at or above -0.5
    assert s_bin(np.float32(s), [-1.0, -0.5]) == want


def _table(rows):
    """value[b, bin, zb, full] with one bin and z = (0, 0) only."""
    v = np.zeros((len(rows), 1, 3, 2), dtype=np.float32)
    v[:, 0, 0, 0] = rows
    return v


def test_route_argmax_and_cost():
    v = _table([4.0, 6.0, 9.0])
    cost = [1.0, 2.0, 4.0]
    # utilities 3, 4, 5 -> 32
    assert oracle_route(np.float32(0), 0, 0, CAND, [], v, cost, 1.0) == 32
    # rho 2: 2, 2, 1 -> tie between 8 and 16 goes to 8
    assert oracle_route(np.float32(0), 0, 0, CAND, [], v, cost, 2.0) == 8
    # rho 1.5: 2.5, 3, 3 -> tie between 16 and 32 goes to 16
    assert oracle_route(np.float32(0), 0, 0, CAND, [], v, cost, 1.5) == 16
    # rho 0: the value alone decides
    assert oracle_route(np.float32(0), 0, 0, CAND, [], v, cost, 0.0) == 32


def test_route_decides_by_the_real_number_utilities():
    """Eq. 3's argmax is taken over the utilities as real numbers.  Here
    rho * cost = fp32(0.3) * 10 = 3 + 2^-23 exactly, so candidate 16 has
    utility 4 - 3 - 2^-23 = 1 - 2^-23, below candidate 8's 1 - 2^-24: the
    definition picks 8.  Evaluated in float32 the product rounds (a tie at
    half an ulp, to even) to 3, candidate 16 gets 1 > 1 - 2^-24 and wins --
    the kind of mistake a float32 oracle would make."""
    rho = np.float32(0.3)
    assert float(rho) * 10 == 3 + 2.0 ** -23 and np.float32(rho * np.float32(10)) == np.float32(3)
    v = _table([1 - 2.0 ** -24, 4.0, -100.0])
    cost = [0.0, 10.0, 0.0]
    assert oracle_route(0.0, 0, 0, CAND, [], v, cost, rho) == 8
    k, u = oracle_utilities(0.0, 0, 0, CAND, [], v, cost, rho)
    assert k == 0 and u[0] == 1 - 2.0 ** -24 and u[1] == 1 - 2.0 ** -23 and u[2] == -100.0


def test_bin_edges_are_compared_exactly():
    # s = -(e1 + e2) / 2 lands exactly on an edge: the bin at or above it
    s, _, _ = oracle_block_state(np.float32(1.5), np.float32(0.5), 8, 0, CAND)
    assert s == -1.0 and s_bin(s, [-1.0, -0.5]) == 1
    # 2^-25 below the edge (in float32, 1.5 + (0.5 + 2^-24) rounds to 2 and s
    # would land on the edge): the bin below
    e2 = np.float32(0.5 + 2.0 ** -24)
    assert float(e2) == 0.5 + 2.0 ** -24 and np.float32(np.float32(1.5) + e2) == np.float32(2.0)
    s, _, _ = oracle_block_state(np.float32(1.5), e2, 8, 0, CAND)
    assert s == -1.0 - 2.0 ** -25 and s_bin(s, [-1.0, -0.5]) == 0


def test_route_reads_the_right_cell():
    v = np.zeros((3, 2, 3, 2), dtype=np.float32)
    cost = [0.0, 0.0, 0.0]
    # only cell (b=1, bin 1, zb 2, full 1) is positive
    v[1, 1, 2, 1] = 1.0
    assert oracle_route(np.float32(0.5), 2, 1, CAND, [0.0], v, cost, 1.0) == 16
    assert oracle_route(np.float32(-0.5), 2, 1, CAND, [0.0], v, cost, 1.0) == 8   # bin 0
    assert oracle_route(np.float32(0.5), 1, 1, CAND, [0.0], v, cost, 1.0) == 8    # other zb
    assert oracle_route(np.float32(0.5), 2, 0, CAND, [0.0], v, cost, 1.0) == 8    # other F


def test_bucket_matches_stable_sort():
    rng = np.random.default_rng(0)
    nb = rng.choice(CAND, size=500)
    order, offsets = oracle_bucket(nb, CAND)
    want = sorted(range(len(nb)), key=lambda r: nb[r])  # Python's sort is stable
    np.testing.assert_array_equal(order, want)
    np.testing.assert_array_equal(offsets, np.concatenate([[0], np.cumsum([np.sum(nb == c) for c in CAND])]))


def test_bucket_definition_on_all_small_inputs():
    for R in range(0, 5):
        for nb in itertools.product(CAND, repeat=R):
            order, offsets = oracle_bucket(list(nb), CAND)
            assert sorted(order.tolist()) == list(range(R))
            for k, c in enumerate(CAND):
                part = order[offsets[k]:offsets[k + 1]].tolist()
                assert all(nb[r] == c for r in part) and part == sorted(part)


def test_plan_round_composes_and_shifts_history():
    rng = np.random.default_rng(1)
    R = 40
    value = rng.standard_normal((3, 4, 3, 2)).astype(np.float32)
    cost = [0.1, 0.3, 0.9]
    edges = [-2.0, -1.0, -0.5]
    acc = rng.integers(0, 33, size=R)
    ent = rng.random(R).astype(np.float32) * 3
    hist = rng.random(R).astype(np.float32) * 3
    prev = rng.choice(CAND, size=R)
    res = oracle_plan_block_sizes(acc, ent, prev, hist, CAND, edges, value, cost, 1.0)
    for r in range(R):
        s, zb, full = oracle_block_state(ent[r], hist[r], prev[r], acc[r], CAND)
        assert res["next_block"][r] == oracle_route(s, zb, full, CAND, edges, value, cost, 1.0)
    np.testing.assert_array_equal(res["entropy_hist"], ent)
    order, offsets = oracle_bucket(res["next_block"], CAND)
    np.testing.assert_array_equal(res["order"], order)
    np.testing.assert_array_equal(res["bucket_offsets"], offsets)
    assert len(set(res["next_block"].tolist())) > 1
