#!/usr/bin/env python3
"""Benchmark of one fused draft-verify step on one MI355X.

A step is the whole hot path over one batch: hybrid-mask paged attention
(rg_draft_verify_attention), then greedy verification / acceptance and draft
confidence, both logit passes of the round in one call
(rg_verify_and_confidence: the same results as rg_verify_accept followed by
rg_draft_confidence, in two launches instead of four).  The separate calls
are timed too.  Inputs are seeded synthetic tensors resident in HBM before
timing starts; several copies of every input are rotated through the steps
so that the working set exceeds the 256 MB Infinity Cache and the numbers
are HBM numbers.  Where one copy of the inputs fits in that cache,
``warm_cache`` reports the step, the attention call and the logit round with
one copy reused by every call, labelled as such (context only).

The default workload is ``long`` (64 requests, 16k-32k context tokens, the
largest configuration); ``all_configs`` reports every configuration's step,
attention and logit-round figures from the same run.

Prints one JSON line.  ``value`` is the step's achieved fraction of the HBM
roofline (algorithmic bytes of all three calls / step time / 8 TB/s), in
percent; the attention call's TFLOP/s and GB/s and the logit passes' GB/s
are reported beside it.  The timed region replays a HIP graph of exactly
``--steps`` steps between two HIP events on the capturing stream; each entry
point is then timed the same way from a graph of ``--steps`` calls of it
alone.  Beside these means, ``*_event_median`` is the median over
``--steps`` eager calls, each between its own pair of HIP events.
``attention_host`` is the host time of the attention entry point (planning
alone, and call to return).  ``roofline`` covers the attention call (the
dominant one): its algorithmic bytes over its per-call time.
``roofline.traffic`` is the HBM traffic per call measured with rocprofv3
counters (FETCH_SIZE + WRITE_SIZE, scaled by what the same counters read for
a plain copy of known size); it is read from the committed profile
summaries and reported only while the attention sources still hash to the
ones the counters were taken with.

The ``overlap`` object measures the predictive draft-verify overlap on the
same workload (rg_multibranch_attention over every request's verify rows and
three branches, against the same rows served as separate requests, plus
rg_plan_branches and rg_match_branches, and the quadratic layout -- one draft
block per hypothetical accepted length -- through the same entry point);
``--no-overlap`` skips it.  The
``block_sizing`` object measures T_C(B) of this path at the workload's load,
one rg_plan_block_sizes round, and the mixed-size batch it plans as one ragged
batch, per size bucket and padded; ``--no-block-sizing`` skips it.

``--copy-calibration-mb N`` instead runs a plain device-to-device copy of N
MiB a few times (for calibrating those counters) and exits.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
CACHE_DEFEAT_BYTES = 512 << 20
WARM_FIT_BYTES = 128 << 20  # one input copy this small stays in the 256 MB Infinity Cache


PROFILES = os.path.join(ROOT, "profiles")
ATTN_SOURCES = ("attention.hip", "rg_internal.h", "api.cpp")


def attention_source_hash():
    """sha256 over the sources that decide what the attention call launches."""
    import hashlib

    h = hashlib.sha256()
    for name in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_34388_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_records():
    """Every TRAFFIC_JSON record of the committed counter summaries."""
    import glob

    recs = []
    for path in sorted(glob.glob(os.path.join(PROFILES, "*.md"))):
        for line in open(path):
            if line.startswith("TRAFFIC_JSON "):
                recs.append(json.loads(line[len("TRAFFIC_JSON "):]))
    return recs


def measured_traffic(workload):
    """HBM bytes per attention call from the committed counter summaries, or
    None when there is none for this workload or the sources changed since."""
    h = attention_source_hash()
    for rec in traffic_records():
        if rec.get("workload") == workload and rec.get("source_sha256") == h:
            return rec["hbm_bytes_per_call"]
    return None


def copy_calibration(mib):
    import torch

    n = (mib << 20) // 2
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read_per_copy": 2 * n, "bytes_written_per_copy": 2 * n,
                                           "copies": 3}}), flush=True)
    return 0


def algorithmic_work(lay):
    """Bytes and flops the step must move / do, counting only allowed
    (query, key) pairs: K and V of every key once per request, q and out
    once, the page table; logits once."""
    s = lay.spec
    D, hq, hkv = s.head_dim, s.num_q_heads, s.num_kv_heads
    attn_bytes = attn_flops = 0
    for r in range(lay.num_requests):
        L, V, B = int(lay.ctx_len[r]), int(lay.n_verify[r]), int(lay.n_draft[r])
        n, T = V + B, L + V + B
        attn_bytes += T * hkv * D * 2 * 2 + n * hq * D * 2 * 2 + math.ceil(T / 16) * 4 + n * hq * 4
        attn_flops += 4 * D * hq * (V * L + V * (V + 1) // 2 + B * T)
    rows_v, rows_d = lay.total_verify_rows, lay.total_draft_rows
    verify_bytes = rows_v * s.vocab * 2 + rows_v * (4 + 4 + 4 + 4) + lay.num_requests * 12
    draft_bytes = rows_d * s.vocab * 2 + rows_d * 6 * 4
    return dict(attn_bytes=attn_bytes, attn_flops=attn_flops, verify_bytes=verify_bytes,
                draft_bytes=draft_bytes)



def overlap_work(ov, branches):
    """Bytes and flops of the overlap round's attention, counting each key of
    a request once for all its rows (the shared-prefix access) and only the
    allowed (query, key) pairs: verify row i sees L + i + 1 keys; a branch's
    j-th lead row L + prefix + j + 1, its draft rows L + prefix + rows."""
    s = ov.spec
    D, hq, hkv = s.head_dim, s.num_q_heads, s.num_kv_heads
    nbytes = pairs = 0
    for r, br in enumerate(branches):
        L, V = int(ov.ctx_len[r]), int(ov.n_verify[r])
        n = int(ov.q_indptr[r + 1] - ov.q_indptr[r])
        T = L + n
        nbytes += T * hkv * D * 2 * 2 + n * hq * D * 2 * 2 + math.ceil(T / 16) * 4 + n * hq * 4
        pairs += V * L + V * (V + 1) // 2
        for prefix, lead, rows in br:
            pairs += lead * (L + prefix) + lead * (lead + 1) // 2 + (rows - lead) * (L + prefix + rows)
    return nbytes, 4 * D * hq * pairs


def overlap_leg(lay, dev, steps, warmup, capture, timed, step_outputs, quadratic=True):
    """Sec. 5.1 / 5.3 measured on the step's workload: every request's rows
    after its verify rows become overlap branches (two corrections and a
    continuation, each with the request's draft block size), served by one
    rg_multibranch_attention call that reads each request's keys once, and
    -- for comparison -- the same rows and keys served as separate requests
    (verify rows alone, each branch with its own copy of the kept prefix in
    its page table) through rg_draft_verify_attention.  Branch planning and
    reuse matching are timed on the step's own confidence and acceptance
    outputs."""
    import numpy as np
    import torch

    from paper_2609_34388_amd import binding
    from paper_2609_34388_amd import workloads as W

    branches = W.overlap_branches(lay)
    ov = W.make_overlap_layout(lay, branches)
    sep, origin = W.make_separate_layout(ov, branches)
    base = W.make_attention_inputs(ov, dev)
    kb, vb = W.make_separate_kv(ov, branches, sep, origin, base["k_cache"], base["v_cache"])
    per_copy = sum(t.numel() * t.element_size() for t in base.values()) + \
        kb.numel() * kb.element_size() * 2
    copies = max(1, math.ceil(CACHE_DEFEAT_BYTES / per_copy))
    sets = [dict(base, k_sep=kb, v_sep=vb)]
    for _ in range(copies - 1):
        sets.append({k: t.clone() for k, t in sets[0].items()})
    indptr = np.concatenate([[0], np.cumsum([len(b) for b in branches])]).astype(np.int32)
    flat = [b for br in branches for b in br]
    col = lambda i: np.array([b[i] for b in flat], dtype=np.int32)
    B = binding.make_branches(indptr, col(0), col(1), col(2))
    pidx = torch.as_tensor(ov.page_indices, device=dev)
    sidx = torch.as_tensor(sep.page_indices, device=dev)
    lays_ov = [binding.make_layout(c["q"], c["k_cache"], ov.q_indptr, ov.n_verify, ov.ctx_len, ov.page_indptr,
                                   pidx) for c in sets]
    lays_sep = [binding.make_layout(c["q"], c["k_sep"], sep.q_indptr, sep.n_verify, sep.ctx_len, sep.page_indptr,
                                    sidx) for c in sets]
    ws_ov = binding.new_workspace(binding.multibranch_workspace_bytes(lays_ov[0], B), dev)
    ws_sep = binding.new_workspace(binding.attention_workspace_bytes(lays_sep[0]), dev)
    out_ov, out_sep = torch.empty_like(base["q"]), torch.empty_like(base["q"])
    lse_ov = torch.empty(base["q"].shape[0], ov.spec.num_q_heads, dtype=torch.float32, device=dev)
    lse_sep = torch.empty_like(lse_ov)

    def multibranch(i):
        c = sets[i % copies]
        binding.multibranch_attention(c["q"], c["k_cache"], c["v_cache"], lays_ov[i % copies], B, out=out_ov,
                                      lse=lse_ov, workspace=ws_ov)

    def separate(i):
        c = sets[i % copies]
        binding.draft_verify_attention(c["q"], c["k_sep"], c["v_sep"], None, None, None, None, sidx, out=out_sep,
                                       lse=lse_sep, workspace=ws_sep, layout=lays_sep[i % copies])

    vout, dout, draft_indptr = step_outputs
    block_len = torch.as_tensor(np.diff(lay.draft_row_indptr).astype(np.int32), device=dev)
    plan_out = binding.plan_branches(dout["margin"], dout["top2"], draft_indptr, 0.5)
    cont_first = dout["top1"][:1].expand(lay.num_requests).contiguous()
    reused = torch.empty(lay.num_requests, dtype=torch.int32, device=dev)

    def plan(i):
        binding.plan_branches(dout["margin"], dout["top2"], draft_indptr, 0.5, out=plan_out)

    def match(i):
        binding.match_branches(vout["accept_len"], vout["next_token"], block_len, plan_out, cont_first, out=reused)

    for i in range(warmup):
        multibranch(i)
        separate(i)
    torch.cuda.synchronize()
    # the two paths must agree on every row (same keys, same rows)
    multibranch(0)
    separate(0)
    torch.cuda.synchronize()
    a, b = out_ov.float(), out_sep.float()
    row_err = ((a - b).abs().amax(-1) / b.norm(dim=-1).clamp_min(1e-6)).max().item()
    if not row_err <= 2e-2:
        raise RuntimeError(f"multi-branch and separate-request outputs differ (max row error {row_err:.3e})")
    mb_ms = timed(multibranch)
    sep_ms = timed(separate)
    plan_ms = timed(plan)
    match_ms = timed(match)
    ov_bytes, ov_flops = overlap_work(ov, branches)
    sep_bytes = algorithmic_work(sep)["attn_bytes"]
    del sets, base, kb, vb
    result = {
        "branches": len(flat), "requests": lay.num_requests, "rows": ov.total_q,
        "kv_tokens": int(ov.kv_len.sum()), "input_copies_rotated": copies,
        "multibranch": {"us": round(mb_ms * 1e3, 3), "bytes": ov_bytes, "flops": ov_flops,
                        "gbps": round(ov_bytes / (mb_ms * 1e-3) / 1e9, 1),
                        "frac_hbm": round(ov_bytes / (mb_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                        "tflops": round(ov_flops / (mb_ms * 1e-3) / 1e12, 3)},
        "separate_requests": {"us": round(sep_ms * 1e3, 3), "requests": sep.num_requests,
                              "bytes": sep_bytes, "gbps": round(sep_bytes / (sep_ms * 1e-3) / 1e9, 1)},
        "speedup_vs_separate": round(sep_ms / mb_ms, 3),
        "bytes_saved": sep_bytes - ov_bytes,
        "max_row_diff_vs_separate": float(f"{row_err:.3e}"),
        "plan_branches_us": round(plan_ms * 1e3, 3), "match_branches_us": round(match_ms * 1e3, 3),
    }
    if not quadratic:
        return result

    # The quadratic layout of Sec. 6.2 on the same requests: one draft block
    # per hypothetical accepted length, through the same entry point.
    qbr = W.quadratic_branches(lay)
    qov = W.make_overlap_layout(lay, qbr)
    qin = W.make_attention_inputs(qov, dev)
    qcopies = max(1, math.ceil(CACHE_DEFEAT_BYTES / sum(t.numel() * t.element_size() for t in qin.values())))
    qsets = [qin] + [{k: t.clone() for k, t in qin.items()} for _ in range(qcopies - 1)]
    qflat = [b for br in qbr for b in br]
    qptr = np.concatenate([[0], np.cumsum([len(b) for b in qbr])]).astype(np.int32)
    qcol = lambda i: np.array([b[i] for b in qflat], dtype=np.int32)
    QB = binding.make_branches(qptr, qcol(0), qcol(1), qcol(2))
    qlay = binding.make_layout(qin["q"], qin["k_cache"], qov.q_indptr, qov.n_verify, qov.ctx_len, qov.page_indptr,
                               torch.as_tensor(qov.page_indices, device=dev))
    qws = binding.new_workspace(binding.multibranch_workspace_bytes(qlay, QB), dev)
    qout = torch.empty_like(qin["q"])
    qlse = torch.empty(qin["q"].shape[0], qov.spec.num_q_heads, dtype=torch.float32, device=dev)

    def quadratic(i):
        c = qsets[i % qcopies]
        binding.multibranch_attention(c["q"], c["k_cache"], c["v_cache"], qlay, QB, out=qout, lse=qlse,
                                      workspace=qws)
    q_ms = timed(quadratic)
    q_bytes, q_flops = overlap_work(qov, qbr)
    del qin, qsets
    result["quadratic_layout"] = {"branches": len(qflat), "rows": qov.total_q, "input_copies_rotated": qcopies,
                                  "us": round(q_ms * 1e3, 3), "bytes": q_bytes, "flops": q_flops,
                                  "gbps": round(q_bytes / (q_ms * 1e-3) / 1e9, 1),
                                  "tflops": round(q_flops / (q_ms * 1e-3) / 1e12, 3),
                                  "time_vs_three_branches": round(q_ms / mb_ms, 3)}
    return result


def _gather(L, inputs, reqs):
    """Requests ``reqs`` of batch ``L`` as a batch of their own: same K/V
    pool, their query rows and logit rows copied out."""
    import numpy as np
    import torch

    from paper_2609_34388_amd import workloads as W

    sub = W.subset(L, reqs)
    cat = lambda ptr: torch.as_tensor(np.concatenate([np.arange(ptr[r], ptr[r + 1]) for r in reqs]).astype(np.int64),
                                      device=inputs["q"].device)
    qi, vi, di = cat(L.q_indptr), cat(L.row_indptr), cat(L.draft_row_indptr)
    return sub, dict(q=inputs["q"][qi].contiguous(), k_cache=inputs["k_cache"], v_cache=inputs["v_cache"],
                     verify_logits=inputs["verify_logits"][vi].contiguous(),
                     draft_tokens=inputs["draft_tokens"][vi].contiguous(),
                     draft_logits=inputs["draft_logits"][di].contiguous())


def block_sizing_leg(lay, dev, timed):
    """Sec. 5.2 / 5.3 on the step's workload: T_C(B) measured for this path
    (uniform blocks of each candidate size at this load), one planning round
    of rg_plan_block_sizes on synthetic request states with a synthetic value
    table, and the resulting mixed-size batch timed as one ragged batch, as
    one batch per size bucket, and padded to the largest planned size."""
    import numpy as np
    import torch

    from paper_2609_34388_amd import binding
    from paper_2609_34388_amd import workloads as W
    from paper_2609_34388_amd.cost_profile import make_step

    R = lay.num_requests
    cand = list(W.BLOCK_CANDIDATES)

    def batch(nv, nd):
        L = W.with_blocks(lay, nv, nd)
        inp = W.make_attention_inputs(L, dev)
        inp.update(W.make_logit_inputs(L, dev))
        return L, inp

    cost_us = []
    for B in cand:
        L, inp = batch(np.full(R, B), np.full(R, B))
        cost_us.append(timed(make_step(L, inp, dev)) * 1e3)
        del inp
    # rho_C: the cost of a 16-token block at this load is worth 8 tokens of progress
    rho = 8.0 / cost_us[1]
    d = W.make_block_policy_inputs(seed=lay.seed, num_requests=R)
    t = lambda a, dt: torch.as_tensor(np.ascontiguousarray(a), dtype=dt, device=dev)
    pol = binding.make_block_policy(d["candidates"], d["s_edges"], cost_us, rho, t(d["value"], torch.float32))
    acc, ent, prev = t(d["accept_len"], torch.int32), t(d["accept_entropy"], torch.float32), t(d["prev_block"], torch.int32)
    hist = t(d["entropy_hist"], torch.float32)
    hist0 = hist.clone()
    res = binding.plan_block_sizes(pol, acc, ent, prev, hist)
    planned = res["next_block"].cpu().numpy()
    order = res["order"].cpu().numpy()
    offs = res["bucket_offsets"].cpu().numpy()

    def plan(i):
        hist.copy_(hist0)
        binding.plan_block_sizes(pol, acc, ent, prev, hist, out=res)
    plan_us = timed(plan) * 1e3
    copy_us = timed(lambda i: hist.copy_(hist0)) * 1e3

    L, inp = batch(d["prev_block"], planned)
    ragged_us = timed(make_step(L, inp, dev)) * 1e3
    parts = []
    for b in range(len(cand)):
        reqs = order[offs[b]:offs[b + 1]]
        if len(reqs):
            sub, sinp = _gather(L, inp, reqs)
            parts.append(make_step(sub, sinp, dev))
    bucketed_us = timed(lambda i: [f(i) for f in parts]) * 1e3
    del inp, parts
    Lp, pinp = batch(d["prev_block"], np.full(R, int(planned.max())))
    padded_us = timed(make_step(Lp, pinp, dev)) * 1e3
    del pinp
    return {
        "candidates": cand, "T_C_us": [round(x, 3) for x in cost_us], "rho_per_us": round(rho, 6),
        "planned": {str(c): int((planned == c).sum()) for c in cand},
        "plan_block_sizes_us": round(max(plan_us - copy_us, 0.0), 3),
        "mixed_step_us": {"ragged_one_batch": round(ragged_us, 3), "bucketed": round(bucketed_us, 3),
                          "padded_to_largest": round(padded_us, 3)},
    }

def _request_problem(lay, inputs, r):
    """Request r of the batch as a problem of its own, as host bf16 bits: its
    query rows, its pages of the K/V pools (renumbered 0 .. p-1), its verify
    rows with the tokens they judge, and its next-block draft rows.  Input
    preparation only (a gather and a copy), outside any timed region."""
    import numpy as np
    import torch

    from paper_2609_34388_amd import workloads as W

    p0, p1 = int(lay.page_indptr[r]), int(lay.page_indptr[r + 1])
    q0, q1 = int(lay.q_indptr[r]), int(lay.q_indptr[r + 1])
    v0, v1 = int(lay.row_indptr[r]), int(lay.row_indptr[r + 1])
    d0, d1 = int(lay.draft_row_indptr[r]), int(lay.draft_row_indptr[r + 1])
    pages = torch.as_tensor(lay.page_indices[p0:p1].astype(np.int64), device=inputs["k_cache"].device)
    return dict(q=W.bf16_bits(inputs["q"][q0:q1]), k=W.bf16_bits(inputs["k_cache"][pages]),
                v=W.bf16_bits(inputs["v_cache"][pages]), q_indptr=np.array([0, q1 - q0], np.int32),
                page_indptr=np.array([0, p1 - p0], np.int32), page_indices=np.arange(p1 - p0, dtype=np.int32),
                n_verify=lay.n_verify[r:r + 1], ctx_len=lay.ctx_len[r:r + 1],
                verify=W.bf16_bits(inputs["verify_logits"][v0:v1]), row_indptr=np.array([0, v1 - v0], np.int32),
                tokens=inputs["draft_tokens"][v0:v1].cpu().numpy(), draft=W.bf16_bits(inputs["draft_logits"][d0:d1]))


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(lay, inputs, budget_s: float):
    """The fp64 oracle as it stands, timed on this host over the step's
    three parts request by request (attention, acceptance, confidence of
    request r's rows), requests in a seeded random order, until about
    ``budget_s`` seconds of oracle time are spent (each request at most once
    per pass; a batch of one request is run several times).  Requests are
    independent draws of the workload, so the whole step's oracle time is
    estimated as the mean time per request times the number of requests."""
    import numpy as np

    import oracle

    R = lay.num_requests
    order = np.random.default_rng(12345).permutation(R)
    parts = [0.0, 0.0, 0.0]  # attention, accept, confidence
    done = 0
    while done == 0 or (sum(parts) < budget_s and done < max(R, 50)):
        r = int(order[done % R])
        pb = _request_problem(lay, inputs, r)
        t0 = time.perf_counter()
        oracle.oracle_attention(pb["q"], pb["k"], pb["v"], pb["q_indptr"], pb["n_verify"], pb["ctx_len"],
                                pb["page_indptr"], pb["page_indices"])
        t1 = time.perf_counter()
        oracle.oracle_accept(pb["verify"], pb["row_indptr"], pb["tokens"])
        t2 = time.perf_counter()
        oracle.oracle_confidence(pb["draft"])
        t3 = time.perf_counter()
        for j, dt in enumerate((t1 - t0, t2 - t1, t3 - t2)):
            parts[j] += dt
        done += 1
    per_req = [p / done for p in parts]
    distinct = min(done, R)
    return {"step_s": sum(per_req) * R, "requests_timed": done, "distinct_requests": distinct,
            "oracle_attention_ms": round(per_req[0] * R * 1e3, 2),
            "oracle_accept_ms": round(per_req[1] * R * 1e3, 2),
            "oracle_confidence_ms": round(per_req[2] * R * 1e3, 2),
            "blas_threads": blas_threads(), "visible_cores": len(os.sched_getaffinity(0)),
            "sample": (f"{done} request run(s) ({distinct} distinct of {R}; all heads and rows of each) of the "
                       f"fp64 numpy oracle, {sum(parts):.1f} s in all; whole-step time = mean time per request "
                       f"x {R} requests")}


def cpu_baseline_rows(lay, dev, budget_s: float):
    """The oracle beside the rows built past the step, on the same workload:
    the overlap round's multi-branch attention (request by request, within
    ``budget_s``; inputs drawn on the device, each timed request's keys and
    rows copied to the host first) and one block-sizing round for every
    request."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_34388_amd import workloads as W

    branches = W.overlap_branches(lay)
    ov = W.make_overlap_layout(lay, branches)
    inp = W.make_attention_inputs(ov, dev)
    done, t_total = 0, 0.0
    order = np.random.default_rng(12345).permutation(ov.num_requests)
    for r in order:
        r = int(r)
        p0, p1 = int(ov.page_indptr[r]), int(ov.page_indptr[r + 1])
        q0, q1 = int(ov.q_indptr[r]), int(ov.q_indptr[r + 1])
        pages = torch.as_tensor(ov.page_indices[p0:p1].astype(np.int64), device=inp["k_cache"].device)
        qb, kb, vb = (W.bf16_bits(t) for t in (inp["q"][q0:q1], inp["k_cache"][pages], inp["v_cache"][pages]))
        t0 = time.perf_counter()
        oracle.oracle_branch_attention(qb, kb, vb, np.array([0, q1 - q0], np.int32), ov.n_verify[r:r + 1],
                                       ov.ctx_len[r:r + 1], np.array([0, p1 - p0], np.int32),
                                       np.arange(p1 - p0, dtype=np.int32), [branches[r]])
        t_total += time.perf_counter() - t0
        done += 1
        if t_total >= budget_s:
            break
    del inp
    overlap = {"us_per_request": round(t_total / done * 1e6, 1), "requests_timed": done,
               "us_all_requests_estimated": round(t_total / done * ov.num_requests * 1e6, 1),
               "sample": f"{done} of {ov.num_requests} request(s) of the overlap round (verify rows and three "
                         f"branches each), fp64 numpy oracle"}
    d = W.make_block_policy_inputs(seed=lay.seed, num_requests=lay.num_requests)
    cost = [1.0] * len(d["candidates"])
    t0 = time.perf_counter()
    oracle.oracle_plan_block_sizes(d["accept_len"], d["accept_entropy"], d["prev_block"], d["entropy_hist"],
                                   d["candidates"], d["s_edges"], d["value"], cost, 0.5)
    plan_us = (time.perf_counter() - t0) * 1e6
    sizing = {"us": round(plan_us, 1), "sample": f"one round for all {lay.num_requests} request(s), oracle"}
    return {"overlap_multibranch_attention": overlap, "plan_block_sizes": sizing}


def host_call_times(layout, q, k, v, out, lse, ws, stream, n):
    """Host cost of the attention entry point (row a1, the planning): the
    mean time of rg_draft_verify_attention_plan (validation and planning, no
    GPU work), and of rg_draft_verify_attention itself from call to return
    (validation, planning and the kernel launches; the kernels run
    asynchronously), over n calls each, called through ctypes directly."""
    import ctypes

    import torch

    from paper_2609_34388_amd import binding

    lib = binding.library()
    info = binding.AttnPlanInfo()
    ref = ctypes.byref(layout.c)
    t0 = time.perf_counter()
    for _ in range(n):
        lib.rg_draft_verify_attention_plan(ref, ctypes.byref(info))
    plan_us = (time.perf_counter() - t0) / n * 1e6
    ws_ptr = ws.data_ptr() if ws is not None else None
    ws_bytes = ws.numel() if ws is not None else 0
    args = (ref, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), ws_ptr, ws_bytes,
            stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        st = lib.rg_draft_verify_attention(*args)
    call_us = (time.perf_counter() - t0) / n * 1e6
    torch.cuda.synchronize()
    if st != 0:
        raise RuntimeError(f"rg_draft_verify_attention returned {st}")
    return {"plan_us": round(plan_us, 2), "call_us": round(call_us, 2), "calls": n,
            "note": "host time per call (rg_draft_verify_attention_plan alone; the attention call from "
                    "call to return, its kernels running asynchronously)"}


def measure_workload(name, seed, dev, steps, warmup, copies_arg=0, detail=False):
    """Time one workload's step and its entry points.  Returns the results
    and, with ``detail``, the objects the extra legs reuse."""
    import torch

    from paper_2609_34388_amd import binding
    from paper_2609_34388_amd import workloads as W

    lay = W.make_layout(name, seed=seed)
    s = lay.spec
    base = W.make_attention_inputs(lay, dev)
    base.update(W.make_logit_inputs(lay, dev))
    per_copy = sum(t.numel() * t.element_size() for t in base.values())
    copies = copies_arg or max(1, math.ceil(CACHE_DEFEAT_BYTES / per_copy))
    sets = [base] + [{k: t.clone() for k, t in base.items()} for _ in range(copies - 1)]
    page_idx = torch.as_tensor(lay.page_indices, device=dev)
    row_indptr = torch.as_tensor(lay.row_indptr, device=dev)

    layouts = [binding.make_layout(c["q"], c["k_cache"], lay.q_indptr, lay.n_verify, lay.ctx_len,
                                   lay.page_indptr, page_idx) for c in sets]
    attn_ws = binding.new_workspace(binding.attention_workspace_bytes(layouts[0]), dev)
    ver_ws = binding.new_workspace(binding.verify_accept_workspace_bytes(
        lay.num_requests, lay.total_verify_rows, s.vocab), dev)
    dr_ws = binding.new_workspace(binding.draft_confidence_workspace_bytes(lay.total_draft_rows, s.vocab), dev)
    round_ws = binding.new_workspace(binding.verify_and_confidence_workspace_bytes(
        lay.num_requests, lay.total_verify_rows, lay.total_draft_rows, s.vocab), dev)
    out = torch.empty_like(base["q"])
    lse = torch.empty(base["q"].shape[0], s.num_q_heads, dtype=torch.float32, device=dev)
    vout = dict(row_argmax=torch.empty(lay.total_verify_rows, dtype=torch.int32, device=dev),
                accept_len=torch.empty(lay.num_requests, dtype=torch.int32, device=dev),
                next_token=torch.empty(lay.num_requests, dtype=torch.int32, device=dev),
                row_entropy=torch.empty(lay.total_verify_rows, dtype=torch.float32, device=dev),
                accept_entropy=torch.empty(lay.num_requests, dtype=torch.float32, device=dev))
    dout = {k: torch.empty(lay.total_draft_rows, dtype=dt, device=dev)
            for k, dt in (("top1", torch.int32), ("top2", torch.int32), ("p1", torch.float32),
                          ("p2", torch.float32), ("margin", torch.float32), ("entropy", torch.float32))}

    def attention(i):
        c = sets[i % copies]
        binding.draft_verify_attention(c["q"], c["k_cache"], c["v_cache"], None, None, None, None, page_idx,
                                       out=out, lse=lse, workspace=attn_ws, layout=layouts[i % copies])

    def verify(i):
        c = sets[i % copies]
        binding.verify_accept(c["verify_logits"], row_indptr, c["draft_tokens"], workspace=ver_ws, out=vout)

    def draft(i):
        c = sets[i % copies]
        binding.draft_confidence(c["draft_logits"], workspace=dr_ws, out=dout)

    def logit_round(i):
        c = sets[i % copies]
        binding.verify_and_confidence(c["verify_logits"], row_indptr, c["draft_tokens"], c["draft_logits"],
                                      workspace=round_ws, out_verify=vout, out_draft=dout)

    def step(i):
        attention(i)
        logit_round(i)

    # Warmup: eager steps (compiles nothing; loads the library, touches every buffer).
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    # The step is launch-bound at low concurrency, so the timed region replays a
    # HIP graph holding exactly `steps` captured steps (input copies rotated),
    # between two HIP events on the capturing stream.
    def capture(fn, n, first):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n):
                fn(first + i)
        torch.cuda.synchronize()
        return g

    def time_calls(fn):
        g = capture(fn, steps, warmup)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        g.replay()  # untimed: the first launch of a graph also uploads it
        torch.cuda.synchronize()
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / steps

    def event_median(fn):
        """Median over `steps` eager calls, each between its own pair of HIP
        events on the launching stream (launch gaps between calls excluded,
        each call's own launches included)."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            a.record(stream)
            fn(warmup + i)
            b.record(stream)
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) for a, b in ev)
        return t[len(t) // 2] if len(t) % 2 else 0.5 * (t[len(t) // 2 - 1] + t[len(t) // 2])

    ms_step = time_calls(step)
    attn_ms = time_calls(attention)
    round_ms = time_calls(logit_round)
    step_med = event_median(step)
    attn_med = event_median(attention)

    work = algorithmic_work(lay)
    step_bytes = work["attn_bytes"] + work["verify_bytes"] + work["draft_bytes"]
    logit_bytes = work["verify_bytes"] + work["draft_bytes"]
    gbps = lambda b, ms: b / (ms * 1e-3) / 1e9
    plan = binding.attention_plan(layouts[0])
    res = dict(
        lay=lay, work=work, step_bytes=step_bytes, copies=copies, per_copy=per_copy, plan=plan,
        ms_step=ms_step, attn_ms=attn_ms, round_ms=round_ms, step_med=step_med, attn_med=attn_med,
        summary={"step_us": round(ms_step * 1e3, 3), "step_us_event_median": round(step_med * 1e3, 3),
                 "value": round(100.0 * gbps(step_bytes, ms_step) / HBM_PEAK_GBPS, 3),
                 "attention_us": round(attn_ms * 1e3, 3), "attention_us_event_median": round(attn_med * 1e3, 3),
                 "attention_frac_hbm": round(gbps(work["attn_bytes"], attn_ms) / HBM_PEAK_GBPS, 4),
                 "attention_tflops": round(work["attn_flops"] / (attn_ms * 1e-3) / 1e12, 3),
                 "logit_round_us": round(round_ms * 1e3, 3),
                 "logits_frac_hbm": round(gbps(logit_bytes, round_ms) / HBM_PEAK_GBPS, 4),
                 "requests": lay.num_requests, "input_copies_rotated": copies})
    if not detail:
        del sets, layouts
        return res
    res["ver_ms"] = time_calls(verify)
    res["dr_ms"] = time_calls(draft)
    res["host"] = host_call_times(layouts[0], sets[0]["q"], sets[0]["k_cache"], sets[0]["v_cache"], out, lse,
                                  attn_ws, stream.cuda_stream, n=100 if lay.num_requests > 16 else 400)
    if plan["split_requests"] > 0:
        # The one-launch work-queue mode (split chunks merged in the same
        # launch), opt-in through RG_ATTN_PERSIST=1, timed the same way.
        prev = os.environ.get("RG_ATTN_PERSIST")
        os.environ["RG_ATTN_PERSIST"] = "1"
        try:
            one_ms = time_calls(attention)
            one_plan = binding.attention_plan(layouts[0])
        finally:
            if prev is None:
                del os.environ["RG_ATTN_PERSIST"]
            else:
                os.environ["RG_ATTN_PERSIST"] = prev
        res["attention_one_launch"] = {"us": round(one_ms * 1e3, 3),
                                       "persistent_launches": one_plan["persistent_launches"],
                                       "time_vs_two_launches": round(one_ms / attn_ms, 3)}
    if copies > 1 and per_copy <= WARM_FIT_BYTES:
        # Labelled warm-cache figures, never the headline: every call of the
        # graph reuses input copy 0, which then stays in the Infinity Cache.
        warm_step = time_calls(lambda i: step(0))
        warm_attn = time_calls(lambda i: attention(0))
        warm_round = time_calls(lambda i: logit_round(0))
        res["warm_cache"] = {
            "note": "inputs resident in the 256 MB Infinity Cache (one input copy reused by every call); "
                    "context only, the headline numbers above rotate copies past the cache",
            "input_bytes": per_copy, "ms_per_step": round(warm_step, 5),
            "attention_us": round(warm_attn * 1e3, 3),
            "attention_gbps": round(work["attn_bytes"] / (warm_attn * 1e-3) / 1e9, 1),
            "logit_round_us": round(warm_round * 1e3, 3)}
    res.update(capture=capture, time_calls=time_calls, vout=vout, dout=dout,
               host_inputs={k: base[k] for k in ("q", "k_cache", "v_cache", "verify_logits", "draft_logits",
                                                 "draft_tokens")})
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long",
                    help="tiny | low | low_sigma2 | mid | high | long (default: long, the largest configuration: "
                         "64 requests, 16k-32k context tokens)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copies", type=int, default=0, help="input copies rotated (0 = enough for 512 MB)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overlap", action="store_true", help="skip the overlap-round measurement")
    ap.add_argument("--no-quadratic", action="store_true",
                    help="in the overlap-round measurement, skip the quadratic layout")
    ap.add_argument("--no-block-sizing", action="store_true", help="skip the block-sizing measurement")
    ap.add_argument("--no-all-configs", action="store_true",
                    help="skip the per-workload summary of the other configurations")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run a plain copy of this many MiB (counter calibration) and exit")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(requests and KV heads would shard across GPUs with no exchange).", file=sys.stderr)
        return 2

    if args.copy_calibration_mb > 0:
        return copy_calibration(args.copy_calibration_mb)

    import torch

    from paper_2609_34388_amd import binding

    if not os.path.exists(binding.LIB_PATH):
        from paper_2609_34388_amd import build_lib
        build_lib.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_start = time.perf_counter()

    m = measure_workload(args.workload, args.seed, dev, args.steps, args.warmup, args.copies, detail=True)
    lay, work, plan = m["lay"], m["work"], m["plan"]
    s = lay.spec
    ms_step, attn_ms, round_ms = m["ms_step"], m["attn_ms"], m["round_ms"]
    ver_ms, dr_ms = m["ver_ms"], m["dr_ms"]
    step_bytes = m["step_bytes"]
    step_gbps = step_bytes / (ms_step * 1e-3) / 1e9
    attn_gbps = work["attn_bytes"] / (attn_ms * 1e-3) / 1e9
    attn_tflops = work["attn_flops"] / (attn_ms * 1e-3) / 1e12
    traffic = measured_traffic(args.workload) if args.seed == 0 else None
    kernels = "attn_fwd_kernel + attn_combine_kernel" if plan["split_requests"] else "attn_fwd_kernel"

    result = {
        "metric": "draft-verify attention TFLOP/s + logits GB/s, % of MI355X roofline, 1 GPU",
        "value": round(100.0 * step_gbps / HBM_PEAK_GBPS, 3),
        "unit": "% of MI355X HBM roofline (whole step: attention + verify + draft bytes / step time / 8 TB/s)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "timing": "mean over a HIP graph replay of exactly `steps` captured steps between two HIP events, "
                  "after one untimed replay of the same graph (its first launch also uploads it; each entry "
                  "point timed the same way alone); *_event_median: median over `steps` eager calls, each "
                  "between its own HIP event pair",
        "config": {"workload": args.workload, "requests": lay.num_requests, "q_heads": s.num_q_heads,
                   "kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "page_size": 16,
                   "context_tokens": int(lay.ctx_len.sum()), "verify_rows": int(lay.n_verify.sum()),
                   "draft_rows": int(lay.n_draft.sum()), "vocab": s.vocab, "seed": args.seed,
                   "input_copies_rotated": m["copies"], "attn_chunk_keys": plan["chunk_keys"],
                   "attn_work_items": plan["work_items"]},
        "step_ms_event_median": round(m["step_med"], 5),
        "attention": {"ms": round(attn_ms, 5), "ms_event_median": round(m["attn_med"], 5),
                      "tflops": round(attn_tflops, 3), "gbps": round(attn_gbps, 1),
                      "bytes": work["attn_bytes"], "flops": work["attn_flops"],
                      "frac_hbm": round(attn_gbps / HBM_PEAK_GBPS, 4),
                      "frac_mfma_bf16": round(attn_tflops / BF16_PEAK_TFLOPS, 5)},
        "attention_host": m["host"],
        "verify_accept": {"ms": round(ver_ms, 5), "bytes": work["verify_bytes"],
                          "gbps": round(work["verify_bytes"] / (ver_ms * 1e-3) / 1e9, 1)},
        "draft_confidence": {"ms": round(dr_ms, 5), "bytes": work["draft_bytes"],
                             "gbps": round(work["draft_bytes"] / (dr_ms * 1e-3) / 1e9, 1)},
        "logit_round": {"ms": round(round_ms, 5), "bytes": work["verify_bytes"] + work["draft_bytes"],
                        "gbps": round((work["verify_bytes"] + work["draft_bytes"]) / (round_ms * 1e-3) / 1e9, 1)},
        "logits_gbps": round((work["verify_bytes"] + work["draft_bytes"]) / (round_ms * 1e-3) / 1e9, 1),
        "roofline": {"kernel": f"rg_draft_verify_attention ({kernels})",
                     "bound": "hbm", "achieved": round(attn_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(attn_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes": work["attn_bytes"], "us_per_call": round(attn_ms * 1e3, 3)},
    }
    for k in ("attention_one_launch", "warm_cache"):
        if k in m:
            result[k] = m[k]
    if not args.no_overlap:
        result["overlap"] = overlap_leg(lay, dev, args.steps, args.warmup, m["capture"], m["time_calls"],
                                        (m["vout"], m["dout"], torch.as_tensor(lay.draft_row_indptr, device=dev)),
                                        quadratic=not args.no_quadratic)
    if not args.no_block_sizing:
        result["block_sizing"] = block_sizing_leg(lay, dev, m["time_calls"])
    if not args.no_cpu_baseline:
        cb = cpu_baseline(lay, m["host_inputs"], args.cpu_budget)
        cpu_gbps = step_bytes / cb["step_s"] / 1e9
        result["cpu_baseline"] = {"value": round(100.0 * cpu_gbps / HBM_PEAK_GBPS, 6), "unit": result["unit"],
                                  "cores": cb["blas_threads"], "kind": "oracle",
                                  "ms_per_step": round(cb["step_s"] * 1e3, 2),
                                  "cores_note": "threads of the BLAS library the oracle's matrix products ran on; "
                                                "the rest of the oracle is single-threaded Python",
                                  **{k: cb[k] for k in ("blas_threads", "visible_cores", "oracle_attention_ms",
                                                        "oracle_accept_ms", "oracle_confidence_ms",
                                                        "requests_timed", "sample")}}
        if not args.no_overlap or not args.no_block_sizing:
            result["cpu_baseline"]["beside_next_rows"] = cpu_baseline_rows(lay, dev, min(4.0, args.cpu_budget / 3))
    headline_summary = m["summary"]
    del m
    torch.cuda.empty_cache()
    if not args.no_all_configs:
        # Every configuration timed the same way in the same run (summary
        # figures; the headline above is the one named in `config.workload`).
        allc = {}
        for name in W_CONFIGS:
            if name == args.workload:
                allc[name] = headline_summary
                continue
            r = measure_workload(name, args.seed, dev, args.steps, args.warmup)
            allc[name] = r["summary"]
            del r
            torch.cuda.empty_cache()
        result["all_configs"] = allc
    result["bench_wall_s"] = round(time.perf_counter() - t_start, 1)
    print(json.dumps(result), flush=True)
    return 0


W_CONFIGS = ("tiny", "low", "mid", "high", "long")


if __name__ == "__main__":
    sys.exit(main())
