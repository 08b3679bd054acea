"""GPU parity of rg_plan_block_sizes (Sec. 5.2 Eq. 2-3, Sec. 5.3) against the
fp64 oracle.

The kernel evaluates Eq. 2's state and Eq. 3's utilities in float32 (one
rounding per operation); the oracle evaluates them as real numbers (float64).
A planned size must be the oracle's, except where the float32 rounding bound
admits another decision: when s lies within that bound of a bin edge (either
bin), or when two candidates' utilities lie within the sum of their bounds
of each other (either candidate).  The bounds: float32 s is the exact
-(e1 + e2) / 2 with one rounding of the sum, so |s32 - s| <= 2^-24 |s|;
a float32 utility fl(v - fl(rho c)) is within 2^-24 (|rho c| + |u|) of
the exact one; both are taken as 2^-23 x (the operands' magnitudes).  The
updated entropy history is bit-exact (a copy), and the grouping and bucket
offsets are bit-exact against the oracle's stable bucketing of the sizes the
kernel planned."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
COST = [1.0, 2.0, 4.0]


def _t(a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a), dtype=dtype, device=DEV)


def _run(d, cost, rho, bucket=True, hist=None):
    pol = binding.make_block_policy(d["candidates"], d["s_edges"], cost, rho, _t(d["value"], torch.float32))
    h = _t(d["entropy_hist"] if hist is None else hist, torch.float32)
    out = binding.plan_block_sizes(pol, _t(d["accept_len"], torch.int32), _t(d["accept_entropy"], torch.float32),
                                   _t(d["prev_block"], torch.int32), h, bucket=bucket)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["entropy_hist"] = h.cpu().numpy()
    return res


def _want(d, cost, rho, hist=None):
    return oracle.oracle_plan_block_sizes(d["accept_len"], d["accept_entropy"], d["prev_block"],
                                          d["entropy_hist"] if hist is None else hist, d["candidates"],
                                          d["s_edges"], d["value"], cost, rho)


EPS = 2.0 ** -23  # relative bound on a float32 evaluation's rounding (twice the unit roundoff)


def _admissible(d, cost, rho, want, hist):
    """[R, NB] mask of the candidates a float32 evaluation of Eq. 2-3 may
    return for each request (the oracle's choice always among them)."""
    cand = np.asarray(d["candidates"])
    edges = np.asarray(d["s_edges"], dtype=np.float64)
    value = np.asarray(d["value"], dtype=np.float64)
    R, NB = len(d["accept_len"]), len(cand)
    ok = np.zeros((R, NB), dtype=bool)
    rc = float(rho) * np.asarray(cost, dtype=np.float32).astype(np.float64)
    for r in range(R):
        _, zb, full = oracle.oracle_block_state(d["accept_entropy"][r], hist[r], d["prev_block"][r],
                                                d["accept_len"][r], cand)
        s, k = want["s"][r], int(want["bin"][r])
        bins = {k}
        if k > 0 and abs(s - edges[k - 1]) <= EPS * abs(s):
            bins.add(k - 1)
        if k < len(edges) and abs(s - edges[k]) <= EPS * abs(s):
            bins.add(k + 1)
        for kb in bins:
            v = value[:, kb, zb, full]
            u = v - rc
            eps = EPS * (np.abs(v) + np.abs(rc))
            ok[r] |= u + eps >= np.max(u - eps)
    return ok


def _compare(got, want, bucket=True, d=None, cost=None, rho=None, hist=None):
    """Planned sizes against the fp64 oracle within the float32 rounding
    bound; history, grouping and offsets bit-exact."""
    cand = np.asarray(d["candidates"])
    nb_got, nb_want = got["next_block"].astype(np.int64), want["next_block"]
    differ = np.nonzero(nb_got != nb_want)[0]
    if len(differ):
        ok = _admissible(d, cost, rho, want, d["entropy_hist"] if hist is None else hist)
        idx = np.searchsorted(cand, nb_got[differ])
        assert (idx < len(cand)).all() and (cand[np.minimum(idx, len(cand) - 1)] == nb_got[differ]).all()
        bad = differ[~ok[differ, idx]]
        assert len(bad) == 0, f"requests {bad[:8].tolist()} planned {nb_got[bad[:8]].tolist()}, " \
                              f"oracle {nb_want[bad[:8]].tolist()}, outside the float32 rounding bound"
        # near-ties are rare on these inputs: a systematic disagreement is a bug, not rounding
        assert len(differ) <= max(2, len(nb_got) // 1000), f"{len(differ)} of {len(nb_got)} differ"
    np.testing.assert_array_equal(got["entropy_hist"], want["entropy_hist"])
    if bucket:
        order, offsets = oracle.oracle_bucket(nb_got, cand)
        np.testing.assert_array_equal(got["order"], order)
        np.testing.assert_array_equal(got["bucket_offsets"], offsets)


@pytest.mark.parametrize("R,ns,rho", [(1, 8, 0.5), (5, 1, 0.5), (128, 8, 0.5), (1000, 8, 2.0), (1024, 16, 0.3),
                                      (1025, 8, 0.5), (4099, 64, 1.0), (65536, 8, 0.5)])
def test_matches_oracle(R, ns, rho):
    d = W.make_block_policy_inputs(seed=R, num_requests=R, num_s_bins=ns)
    got = _run(d, COST, rho)
    want = _want(d, COST, rho)
    _compare(got, want, d=d, cost=COST, rho=rho)
    if R >= 128:
        assert len(set(want["next_block"].tolist())) == 3  # every bucket is used


def test_without_bucketing_and_empty_batch():
    d = W.make_block_policy_inputs(seed=7, num_requests=300)
    _compare(_run(d, COST, 0.5, bucket=False), _want(d, COST, 0.5), bucket=False, d=d, cost=COST, rho=0.5)
    e = W.make_block_policy_inputs(seed=8, num_requests=0)
    got = _run(e, COST, 0.5)
    np.testing.assert_array_equal(got["bucket_offsets"], [0, 0, 0, 0])


def test_ties_go_to_the_smaller_block_and_edges_are_exact():
    d = W.make_block_policy_inputs(seed=9, num_requests=2000, num_s_bins=4)
    # utilities equal for every candidate: value = rho * cost + c
    rho = 0.5
    d["value"][:] = np.float32(3.0)
    for b, c in enumerate(COST):
        d["value"][b] += np.float32(rho) * np.float32(c)
    # some states exactly on a bin edge (s = -(e1 + e2) / 2)
    d["accept_entropy"][:100] = np.float32(-d["s_edges"][1])
    d["entropy_hist"][:100] = np.float32(-d["s_edges"][1])
    got, want = _run(d, COST, rho), _want(d, COST, rho)
    # all utilities are exactly 3 in float32 and in float64 (no rounding anywhere): ties go to the smallest
    assert (want["utility"] == 3.0).all()
    np.testing.assert_array_equal(got["next_block"], want["next_block"])
    assert (want["next_block"] == 8).all()
    _compare(got, want, d=d, cost=COST, rho=rho)
    d2 = W.make_block_policy_inputs(seed=9, num_requests=2000, num_s_bins=4)
    d2["accept_entropy"][:100] = np.float32(-d2["s_edges"][1])
    d2["entropy_hist"][:100] = np.float32(-d2["s_edges"][1])
    _compare(_run(d2, COST, 0.5), _want(d2, COST, 0.5), d=d2, cost=COST, rho=0.5)


def test_two_rounds_carry_the_history():
    d = W.make_block_policy_inputs(seed=11, num_requests=777)
    r1 = _run(d, COST, 0.5)
    w1 = _want(d, COST, 0.5)
    _compare(r1, w1, d=d, cost=COST, rho=0.5)
    d2 = W.make_block_policy_inputs(seed=12, num_requests=777)
    d2["prev_block"] = w1["next_block"].astype(np.int32)
    r2 = _run(d2, COST, 0.5, hist=r1["entropy_hist"])
    w2 = _want(d2, COST, 0.5, hist=w1["entropy_hist"])
    _compare(r2, w2, d=d2, cost=COST, rho=0.5, hist=w1["entropy_hist"])


def test_previous_blocks_outside_the_candidates():
    d = W.make_block_policy_inputs(seed=13, num_requests=500)
    rng = np.random.default_rng(13)
    d["prev_block"] = rng.integers(1, 70, size=500).astype(np.int32)
    d["accept_len"] = np.array([rng.integers(0, p + 2) for p in d["prev_block"]], dtype=np.int32)
    _compare(_run(d, COST, 0.5), _want(d, COST, 0.5), d=d, cost=COST, rho=0.5)


def test_float32_near_tie_is_admitted_only_within_the_bound():
    """rho * cost = fp32(0.3) * 10 is 3 + 2^-23 exactly; in float32 it rounds
    to 3.  Candidate 16's utility is then 1 - 2^-23 as a real number (below
    candidate 8's 1 - 2^-24: the definition picks 8) but 1 in float32 (16
    wins).  Both lie within the float32 bound, so either is accepted (and the
    grouping follows the sizes the kernel planned); with candidate 32 far
    ahead instead, the sizes must be the oracle's exactly."""
    R = 300
    d = W.make_block_policy_inputs(seed=21, num_requests=R)
    cost = [0.0, 10.0, 0.0]
    rho = float(np.float32(0.3))
    d["value"][0] = np.float32(1 - 2.0 ** -24)
    d["value"][1] = np.float32(4.0)
    d["value"][2] = np.float32(-100.0)
    got, want = _run(d, cost, rho), _want(d, cost, rho)
    assert (want["next_block"] == 8).all()
    assert set(got["next_block"].tolist()) <= {8, 16}
    ok = _admissible(d, cost, rho, want, d["entropy_hist"])
    assert ok[:, 0].all() and ok[:, 1].all() and not ok[:, 2].any()
    order, offsets = oracle.oracle_bucket(got["next_block"], d["candidates"])
    np.testing.assert_array_equal(got["order"], order)
    np.testing.assert_array_equal(got["bucket_offsets"], offsets)
    # away from the tie (candidate 32 far ahead) the planned sizes are the oracle's exactly
    d["value"][2] = np.float32(50.0)
    got2, want2 = _run(d, cost, rho), _want(d, cost, rho)
    assert (want2["next_block"] == 32).all()
    np.testing.assert_array_equal(got2["next_block"], want2["next_block"])
