"""GPU parity of rg_plan_block_sizes (Sec. 5.2 Eq. 2-3, Sec. 5.3) against the
oracle: planned block sizes, the updated entropy history, the stable grouping
and the bucket offsets, all bit-exact (the decisions are fp32 on both
sides)."""
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


def _compare(got, want, bucket=True):
    np.testing.assert_array_equal(got["next_block"], want["next_block"])
    np.testing.assert_array_equal(got["entropy_hist"], want["entropy_hist"])
    if bucket:
        np.testing.assert_array_equal(got["order"], want["order"])
        np.testing.assert_array_equal(got["bucket_offsets"], want["bucket_offsets"])


@pytest.mark.parametrize("R,ns,rho", [(1, 8, 0.5), (5, 1, 0.5), (128, 8, 0.5), (1000, 8, 2.0), (1024, 16, 0.3),
                                      (1025, 8, 0.5), (4099, 64, 1.0), (65536, 8, 0.5)])
def test_matches_oracle(R, ns, rho):
    d = W.make_block_policy_inputs(seed=R, num_requests=R, num_s_bins=ns)
    got = _run(d, COST, rho)
    want = _want(d, COST, rho)
    _compare(got, want)
    if R >= 128:
        assert len(set(want["next_block"].tolist())) == 3  # every bucket is used


def test_without_bucketing_and_empty_batch():
    d = W.make_block_policy_inputs(seed=7, num_requests=300)
    _compare(_run(d, COST, 0.5, bucket=False), _want(d, COST, 0.5), bucket=False)
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
    _compare(got, want)
    d2 = W.make_block_policy_inputs(seed=9, num_requests=2000, num_s_bins=4)
    d2["accept_entropy"][:100] = np.float32(-d2["s_edges"][1])
    d2["entropy_hist"][:100] = np.float32(-d2["s_edges"][1])
    _compare(_run(d2, COST, 0.5), _want(d2, COST, 0.5))


def test_two_rounds_carry_the_history():
    d = W.make_block_policy_inputs(seed=11, num_requests=777)
    r1 = _run(d, COST, 0.5)
    w1 = _want(d, COST, 0.5)
    _compare(r1, w1)
    d2 = W.make_block_policy_inputs(seed=12, num_requests=777)
    d2["prev_block"] = w1["next_block"].astype(np.int32)
    r2 = _run(d2, COST, 0.5, hist=r1["entropy_hist"])
    w2 = _want(d2, COST, 0.5, hist=w1["entropy_hist"])
    _compare(r2, w2)


def test_previous_blocks_outside_the_candidates():
    d = W.make_block_policy_inputs(seed=13, num_requests=500)
    rng = np.random.default_rng(13)
    d["prev_block"] = rng.integers(1, 70, size=500).astype(np.int32)
    d["accept_len"] = np.array([rng.integers(0, p + 2) for p in d["prev_block"]], dtype=np.int32)
    _compare(_run(d, COST, 0.5), _want(d, COST, 0.5))
