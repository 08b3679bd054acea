"""Summaries of the rocprofv3 runs of profile_runs.sh as the markdown kept
under profiles/ (kernel trace, HBM traffic with the copy calibration and the
record bench.py reads, compute-side counters).

Usage: python -m paper_2609_34388_amd.profile_summary <out-dir> <workload | overlap:workload> [...]
(<out-dir> and entries as given to profile_runs.sh; writes profiles/*_<workload>*.md).
"""
from __future__ import annotations

import csv
import glob
import json
import os
import statistics
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

RUNS = "bash paper_2609_34388_amd/profile_runs.sh <out-dir> {wl}"
BENCH = "python3 bench.py --no-block-sizing --no-cpu-baseline --no-all-configs --no-overlap --workload {wl}"
BENCH_OV = "python3 bench.py --no-block-sizing --no-cpu-baseline --no-all-configs --no-quadratic --workload {wl}"


def short(name: str) -> str:
    n = name.replace("(anonymous namespace)::", "").replace("rg::", "")
    if n.startswith("void "):
        n = n[5:]
    return n.split("(")[0]


def one(pattern: str) -> str:
    hits = glob.glob(pattern)
    if len(hits) != 1:
        raise FileNotFoundError(pattern)
    return hits[0]


def counter_rows(path: str):
    return list(csv.DictReader(open(path)))


def per_kernel(rows, counter):
    agg = defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            agg[short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return agg


def bench_line(log: str):
    for line in open(log):
        if line.startswith("{"):
            return json.loads(line)
    raise ValueError(f"no bench line in {log}")


def calibration(out: str):
    f = {}
    for c, known in (("FETCH_SIZE", 262144.0), ("WRITE_SIZE", 262144.0)):
        vals = per_kernel(counter_rows(one(f"{out}/copy_{c}/*counter_collection.csv")), c)["__amd_rocclr_copyBuffer"]
        f[c] = (vals, known, known / statistics.mean(vals))
    return f


def trace_md(out: str, wl: str) -> str:
    rows = list(csv.DictReader(open(one(f"{out}/trace_{wl}/*kernel_stats.csv"))))
    b = bench_line(f"{out}/trace_{wl}.log")
    lines = [f"# Kernel trace of the `{wl}` step (rocprofv3 --kernel-trace --stats)", "",
             f"Workload `{wl}`: {b['config']['requests']} request(s), 32 query / 8 KV heads, head_dim 128, "
             f"{b['config']['context_tokens']} context tokens, {b['config']['verify_rows']} verify + "
             f"{b['config']['draft_rows']} draft rows, vocab {b['config']['vocab']}, seed 0.", "",
             "Command (repository root on the GPU host; the trace pass of):", "", "```", RUNS.format(wl=wl),
             "# i.e. rocprofv3 --kernel-trace --stats --output-format csv -d <out-dir>/trace_" + wl + " -o " + wl
             + " -- " + BENCH.format(wl=wl) + " --steps 20 --warmup 5", "```", "",
             "Library kernels (every dispatch of the run: warmup, graph replays, per-call timings, host-cost calls):",
             "", "| kernel | calls | mean us | min us | max us |", "|---|---|---|---|---|"]
    for r in rows:
        n = short(r["Name"])
        if any(k in n for k in ("attn_", "rows_kernel", "finalize_kernel")):
            lines.append(f"| {n} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                         f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} |")
    lines += ["", "The benchmark line of the same run (under the profiler):", "",
              f"- step {b['ms_per_step'] * 1e3:.1f} us (graph-replay mean), `value` {b['value']} % of the HBM roofline;",
              f"- attention {b['attention']['ms'] * 1e3:.1f} us per call ({b['attention']['gbps']} GB/s, "
              f"{b['attention']['tflops']} TFLOP/s), event median {b['attention']['ms_event_median'] * 1e3:.1f} us;",
              f"- logit round {b['logit_round']['ms'] * 1e3:.1f} us ({b['logit_round']['gbps']} GB/s).", ""]
    return "\n".join(lines)


def traffic_md(out: str, wl: str) -> str:
    cal = calibration(out)
    fetch = per_kernel(counter_rows(one(f"{out}/pmc_FETCH_SIZE_{wl}/*counter_collection.csv")), "FETCH_SIZE")
    write = per_kernel(counter_rows(one(f"{out}/pmc_WRITE_SIZE_{wl}/*counter_collection.csv")), "WRITE_SIZE")
    b = bench_line(f"{out}/trace_{wl}.log")
    ff, wf = cal["FETCH_SIZE"][2], cal["WRITE_SIZE"][2]
    lines = [f"# HBM traffic of the attention call, workload `{wl}` (rocprofv3 counters)", "",
             "Commands (one counter per pass; the counter passes of):", "", "```", RUNS.format(wl=wl),
             "# i.e. for c in FETCH_SIZE WRITE_SIZE:", "#   rocprofv3 --pmc $c --output-format csv -d <out-dir>/copy_$c -o copy"
             " -- python3 bench.py --copy-calibration-mb 256",
             "#   rocprofv3 --pmc $c --output-format csv -d <out-dir>/pmc_${c}_" + wl + " -o " + wl + " -- "
             + BENCH.format(wl=wl) + " --steps 3 --warmup 1", "```", "",
             "Calibration: a 256 MiB device-to-device copy (`__amd_rocclr_copyBuffer`) reads and writes 262144 KiB.",
             "", "| counter | copy kernel reads (KiB per dispatch) | known KiB | factor |", "|---|---|---|---|"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        vals, known, fac = cal[c]
        lines.append(f"| {c} | {', '.join(f'{v:.1f}' for v in vals)} | {known:.0f} | {fac:.5f} |")
    lines += ["", "Per dispatch of the library kernels (mean over the dispatches of the run, KiB as the counter reads):",
              "", "| kernel | FETCH_SIZE | WRITE_SIZE | scaled bytes (fetch x factor + write x factor) |",
              "|---|---|---|---|"]
    attn_bytes = 0.0
    for k in fetch:
        if not any(t in k for t in ("attn_", "rows_kernel", "finalize_kernel")):
            continue
        fv, wv = statistics.mean(fetch[k]), statistics.mean(write.get(k, [0.0]))
        by = (fv * ff + wv * wf) * 1024
        lines.append(f"| {k} | {fv:.1f} | {wv:.1f} | {by / 1e6:.3f} MB |")
        if k.startswith("attn_fwd_kernel<128, AttnPlanT<AttnReq, 128>") or k.startswith("attn_combine_kernel<128"):
            if "AttnReqBr" not in k:
                attn_bytes += by
    alg = b["attention"]["bytes"]
    lines += ["", f"Attention call (attn_fwd_kernel and, for split requests, attn_combine_kernel): "
              f"{attn_bytes / 1e6:.3f} MB of HBM traffic per call against {alg / 1e6:.3f} MB of algorithmic bytes "
              f"(K and V of every key once, q, out, page table, lse): {attn_bytes / alg:.4f}x.", "",
              "Machine-readable record read by bench.py (reported as `roofline.traffic` only while the attention "
              "sources hash to `source_sha256`):", "",
              "TRAFFIC_JSON " + json.dumps({"workload": wl, "hbm_bytes_per_call": int(round(attn_bytes)),
                                           "fetch_factor": round(ff, 5), "write_factor": round(wf, 5),
                                           "source_sha256": bench.attention_source_hash()}), ""]
    return "\n".join(lines)


def sq_md(out: str, wl: str) -> str:
    rows = counter_rows(one(f"{out}/sq_{wl}/*counter_collection.csv"))
    b = bench_line(f"{out}/trace_{wl}.log")
    cs = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "SQ_INSTS_VALU",
          "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAVE_CYCLES", "GRBM_GUI_ACTIVE")
    agg = {c: per_kernel(rows, c) for c in cs}
    lines = [f"# Compute-side counters, workload `{wl}` (rocprofv3 --pmc)", "",
             "Command (the SQ pass of):", "", "```", RUNS.format(wl=wl),
             "# i.e. rocprofv3 --pmc " + " ".join(cs) + " --output-format csv -d <out-dir>/sq_" + wl + " -o " + wl
             + " -- " + BENCH.format(wl=wl) + " --steps 3 --warmup 1", "```", "",
             "Means per dispatch.  MFMA flops = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512.  MFMA busy = "
             "SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs).  Entries = vocabulary entries "
             "of the logit rows.", "",
             "| kernel | MFMA GFLOP | MFMA busy | VALU instr | LDS instr | LDS bank conflicts | GRBM_GUI_ACTIVE / 8 |",
             "|---|---|---|---|---|---|---|"]
    for k in agg["GRBM_GUI_ACTIVE"]:
        if not any(t in k for t in ("attn_", "rows_kernel", "finalize_kernel")):
            continue
        m = lambda c: statistics.mean(agg[c].get(k, [0.0]))
        cyc = m("GRBM_GUI_ACTIVE") / 8
        busy = m("SQ_VALU_MFMA_BUSY_CYCLES") / (1024 * cyc) if cyc else 0.0
        lines.append(f"| {k} | {m('SQ_INSTS_VALU_MFMA_MOPS_BF16') * 512 / 1e9:.2f} | {100 * busy:.1f} % | "
                     f"{m('SQ_INSTS_VALU'):.4g} | {m('SQ_INSTS_LDS'):.4g} | {m('SQ_LDS_BANK_CONFLICT'):.4g} | "
                     f"{cyc:.4g} |")
    ent = (b["config"]["verify_rows"] + b["config"]["draft_rows"]) * b["config"]["vocab"]
    lines += ["", f"Algorithmic attention flops of the workload: {b['attention']['flops'] / 1e9:.2f} GFLOP.  "
              f"The logit rows hold {ent / 1e6:.1f} M vocabulary entries ((verify + draft rows) x vocab); "
              "VALU instructions per entry (wave instructions x 64 lanes / entries):", ""]
    for k in ("round_rows_kernel", "verify_rows_kernel", "draft_rows_kernel"):
        rows_k = b["config"]["verify_rows"] if k.startswith("verify") else (
            b["config"]["draft_rows"] if k.startswith("draft") else
            b["config"]["verify_rows"] + b["config"]["draft_rows"])
        vr = statistics.mean(agg["SQ_INSTS_VALU"].get(k, [0.0]))
        e = rows_k * b["config"]["vocab"]
        lines.append(f"- {k}: {vr:.4g} VALU wave instructions over {e / 1e6:.1f} M entries, "
                     f"{vr * 64 / e:.2f} per entry")
    lines.append("")
    return "\n".join(lines)


def overlap_md(out: str, wl: str) -> str:
    tag = f"overlap_{wl}"
    rows = list(csv.DictReader(open(one(f"{out}/trace_{tag}/*kernel_stats.csv"))))
    b = bench_line(f"{out}/trace_{tag}.log")
    ov = b["overlap"]
    cal = calibration(out)
    ff, wf = cal["FETCH_SIZE"][2], cal["WRITE_SIZE"][2]
    fetch = per_kernel(counter_rows(one(f"{out}/pmc_FETCH_SIZE_{tag}/*counter_collection.csv")), "FETCH_SIZE")
    write = per_kernel(counter_rows(one(f"{out}/pmc_WRITE_SIZE_{tag}/*counter_collection.csv")), "WRITE_SIZE")
    launches = (ov["requests"] + 63) // 64  # the branched plan holds 64 requests per launch
    lines = [f"# Multi-branch attention of the overlap round, workload `{wl}`: kernel trace and HBM traffic", "",
             f"The overlap round of the benchmark on `{wl}` ({ov['requests']} requests, {ov['branches']} branches, "
             f"{ov['rows']} query rows, {ov['kv_tokens']} keys): every request keeps its verify rows and gets two "
             "correction branches (a committed replacement token plus a draft block of the request's block size) "
             "and a continuation branch, served by one rg_multibranch_attention call that reads each request's "
             "keys once; the comparison serves the same rows and keys as separate requests through "
             "rg_draft_verify_attention.", "",
             "Commands (repository root on the GPU host; the overlap entry of):", "", "```",
             f"bash paper_2609_34388_amd/profile_runs.sh <out-dir> overlap:{wl}",
             f"# i.e. rocprofv3 --kernel-trace --stats --output-format csv -d <out-dir>/trace_{tag} -o {tag} -- "
             + BENCH_OV.format(wl=wl) + " --steps 20 --warmup 5",
             f"#   and for c in FETCH_SIZE WRITE_SIZE: rocprofv3 --pmc $c --output-format csv -d "
             f"<out-dir>/pmc_${{c}}_{tag} -o {tag} -- " + BENCH_OV.format(wl=wl) + " --steps 3 --warmup 1",
             "```", "", "| kernel | calls | mean us |", "|---|---|---|"]
    for r in rows:
        n = short(r["Name"])
        if "AttnReqBr" in n or "branches_kernel" in n:
            lines.append(f"| {n} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} |")
    by = 0.0
    fk = wk = 0.0
    for k in fetch:
        if "AttnReqBr" in k:
            f_, w_ = statistics.mean(fetch[k]), statistics.mean(write.get(k, [0.0]))
            fk += f_
            wk += w_
            by += (f_ * ff + w_ * wf) * 1024
    by *= launches  # every branched kernel runs once per launch
    fk *= launches
    wk *= launches
    alg = ov["multibranch"]["bytes"]
    lines += ["", f"rg_multibranch_attention = {launches} launch(es) per call (at most 64 requests per launch).", "",
              "| per call | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM MB (scaled) | algorithmic MB | ratio |",
              "|---|---|---|---|---|---|",
              f"| rg_multibranch_attention | {fk:.0f} | {wk:.0f} | {by / 1e6:.1f} | {alg / 1e6:.1f} | {by / alg:.3f} |",
              "", f"Counter scaling from the plain-copy calibration of the same run: FETCH_SIZE x {ff:.4f}, "
              f"WRITE_SIZE x {wf:.4f}.", "", "Bench (graph replay, profiler attached):", "", "```",
              json.dumps(ov), "```", ""]
    return "\n".join(lines)


def main(argv):
    out, entries = argv[0], argv[1:]
    for e in entries:
        if e.startswith("overlap:"):
            wl = e.split(":", 1)[1]
            path = os.path.join(ROOT, "profiles", f"multibranch_{wl}_trace_and_traffic.md")
            with open(path, "w") as f:
                f.write(overlap_md(out, wl))
            print("wrote", path)
            continue
        wl = e
        for name, fn in ((f"step_{wl}_kernel_trace.md", trace_md), (f"attention_{wl}_traffic.md", traffic_md),
                         (f"compute_counters_{wl}.md", sq_md)):
            path = os.path.join(ROOT, "profiles", name)
            with open(path, "w") as f:
                f.write(fn(out, wl))
            print("wrote", path)


if __name__ == "__main__":
    main(sys.argv[1:])
