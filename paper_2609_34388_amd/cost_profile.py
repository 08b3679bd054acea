"""Offline execution-cost profile T_C(B) of this path (Sec. 5.2, Eq. 3).

The block-size policy weighs each candidate block size B by the profiled
cost of a step at serving load C.  This tool measures that cost for the part
of the step this library runs -- the draft-verify attention and both logit
passes -- on the local GPU: for each concurrency C and candidate B, a batch
of C requests, each with B verify rows and a B-row draft block over a
context drawn from U[512, 4096] tokens, in the 8B-style shape (32 query /
8 KV heads, head dim 128, vocabulary 128256), timed by replaying a HIP
graph of repeated steps.

    python -m paper_2609_34388_amd.cost_profile [--loads 1,2,4,...] [--blocks 8,16,32] [--steps 50]

prints one JSON object {"T_C_us": {C: {B: microseconds}}, ...}.
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np
import torch

from . import binding
from . import workloads as W


def make_step(L, inputs, dev):
    """A function running one step of batch ``L`` on ``inputs`` (attention,
    then verification and draft confidence in one call); its buffers are
    allocated once, here."""
    s = L.spec
    pidx = torch.as_tensor(L.page_indices, device=dev)
    lt = binding.make_layout(inputs["q"], inputs["k_cache"], L.q_indptr, L.n_verify, L.ctx_len, L.page_indptr, pidx)
    aws = binding.new_workspace(binding.attention_workspace_bytes(lt), dev)
    rws = binding.new_workspace(binding.verify_and_confidence_workspace_bytes(
        L.num_requests, L.total_verify_rows, L.total_draft_rows, s.vocab), dev)
    rp = torch.as_tensor(L.row_indptr, device=dev)
    out = torch.empty_like(inputs["q"])
    lse = torch.empty(inputs["q"].shape[0], s.num_q_heads, dtype=torch.float32, device=dev)
    vout = dict(row_argmax=torch.empty(L.total_verify_rows, dtype=torch.int32, device=dev),
                accept_len=torch.empty(L.num_requests, dtype=torch.int32, device=dev),
                next_token=torch.empty(L.num_requests, dtype=torch.int32, device=dev),
                row_entropy=torch.empty(L.total_verify_rows, dtype=torch.float32, device=dev),
                accept_entropy=torch.empty(L.num_requests, dtype=torch.float32, device=dev))
    dout = {k: torch.empty(L.total_draft_rows, dtype=dt, device=dev)
            for k, dt in (("top1", torch.int32), ("top2", torch.int32), ("p1", torch.float32),
                          ("p2", torch.float32), ("margin", torch.float32), ("entropy", torch.float32))}

    def step(i):
        binding.draft_verify_attention(inputs["q"], inputs["k_cache"], inputs["v_cache"], None, None, None, None,
                                       pidx, out=out, lse=lse, workspace=aws, layout=lt)
        binding.verify_and_confidence(inputs["verify_logits"], rp, inputs["draft_tokens"], inputs["draft_logits"],
                                      workspace=rws, out_verify=vout, out_draft=dout)
    return step


def graph_time_ms(fn, steps: int, warmup: int = 2) -> float:
    """Milliseconds per call of ``fn``: a HIP graph of ``steps`` calls,
    replayed once untimed (its first launch also uploads it), then once
    between two events on the capturing stream."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(steps):
            fn(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g.replay()
    torch.cuda.synchronize()
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def profile(loads, blocks, steps: int = 50, seed: int = 0, dev=None):
    dev = dev or torch.device("cuda:0")
    table = {}
    for C in loads:
        base = W.make_layout("high", seed=seed, num_requests=C)
        table[C] = {}
        for B in blocks:
            L = W.with_blocks(base, np.full(C, B), np.full(C, B))
            inp = W.make_attention_inputs(L, dev)
            inp.update(W.make_logit_inputs(L, dev))
            table[C][B] = graph_time_ms(make_step(L, inp, dev), steps) * 1e3
            del inp
            print(json.dumps({"C": C, "B": B, "us": round(table[C][B], 3)}), file=sys.stderr, flush=True)
    return table


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--loads", default="1,2,4,8,16,32,64,128")
    ap.add_argument("--blocks", default="8,16,32")
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    loads = [int(x) for x in args.loads.split(",")]
    blocks = [int(x) for x in args.blocks.split(",")]
    if not torch.cuda.is_available():
        raise SystemExit("cost_profile needs a GPU")
    table = profile(loads, blocks, args.steps, args.seed)
    print(json.dumps({"path": "draft-verify attention + verification + draft confidence",
                      "shape": "32 q / 8 kv heads, head_dim 128, vocab 128256, contexts U[512, 4096]",
                      "T_C_us": {str(c): {str(b): round(t, 3) for b, t in row.items()} for c, row in table.items()}}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
