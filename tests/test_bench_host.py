"""Host-side parts of bench.py (no GPU): the one-GPU guard, the algorithmic
work the roofline divides by, the counter record's source check and the
oracle baseline's per-function split."""
import json
import re

import numpy as np

import bench
from paper_2609_34388_amd import workloads as W


def test_more_than_one_gpu_exits_with_a_message(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


def _visible_pairs(lay):
    """Allowed (row, key) pairs of every request, counted on a dense mask
    built from Eq. 1 of the fused step: verify row i sees keys 0 .. L + i,
    a draft row sees all T keys."""
    total = 0
    for r in range(lay.num_requests):
        L, V, B = int(lay.ctx_len[r]), int(lay.n_verify[r]), int(lay.n_draft[r])
        T = L + V + B
        keys = np.arange(T)[None, :]
        rows = np.arange(V + B)[:, None]
        lim = np.where(rows < V, L + rows + 1, T)
        total += int((keys < lim).sum())
    return total


def test_attention_flops_count_only_visible_pairs():
    for spec, seed, n in (("tiny", 0, None), ("mid", 3, 5), ("high", 1, 9)):
        lay = W.make_layout(spec, seed=seed, num_requests=n) if n else W.make_layout(spec, seed=seed)
        s = lay.spec
        work = bench.algorithmic_work(lay)
        # QK^T and PV: 2 flops per multiply-add, D per pair each, per query head
        assert work["attn_flops"] == 4 * s.head_dim * s.num_q_heads * _visible_pairs(lay)


def test_attention_bytes_read_each_key_once():
    lay = W.make_layout("mid", seed=2, num_requests=4)
    s = lay.spec
    kv = sum(int(t) for t in lay.kv_len) * s.num_kv_heads * s.head_dim * 2 * 2
    qo = lay.total_q * s.num_q_heads * s.head_dim * 2 * 2
    pages = sum((int(t) + 15) // 16 for t in lay.kv_len) * 4
    lse = lay.total_q * s.num_q_heads * 4
    assert bench.algorithmic_work(lay)["attn_bytes"] == kv + qo + pages + lse


def test_traffic_record_reported_only_for_its_workload_and_source():
    recs = bench.traffic_records()
    assert recs
    h = bench.attention_source_hash()
    for rec in recs:
        current = [r for r in recs if r["workload"] == rec["workload"] and r["source_sha256"] == h]
        if current:
            assert bench.measured_traffic(rec["workload"]) == current[0]["hbm_bytes_per_call"]
        else:
            assert bench.measured_traffic(rec["workload"]) is None
    assert bench.measured_traffic("no-such-workload") is None


def test_cpu_baseline_reports_each_oracle_function():
    lay = W.make_layout("tiny", seed=0)
    inputs = W.make_attention_inputs(lay, "cpu")
    inputs.update(W.make_logit_inputs(lay, "cpu"))
    cb = bench.cpu_baseline(lay, inputs, 0.2)
    assert cb["requests_timed"] >= 1 and cb["blas_threads"] >= 1 and cb["visible_cores"] >= 1
    split = [cb[k] for k in ("oracle_attention_ms", "oracle_accept_ms", "oracle_confidence_ms")]
    assert sum(split) <= cb["step_s"] * 1e3 + 0.05


def test_cpu_baseline_samples_requests_and_scales_to_the_batch():
    """A batch of several requests is timed request by request on a sample
    and scaled by the number of requests."""
    lay = W.make_layout("high", seed=0, num_requests=6, ctx=("uniform", 16, 64))
    inputs = W.make_attention_inputs(lay, "cpu")
    inputs.update(W.make_logit_inputs(lay, "cpu"))
    cb = bench.cpu_baseline(lay, inputs, 0.0)
    assert cb["requests_timed"] == 1 and cb["distinct_requests"] == 1
    assert "x 6 requests" in cb["sample"]
