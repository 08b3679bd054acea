"""The entry points captured in a HIP graph: every replay (with eager work
and synchronisations in between) must reproduce the eager results bit for
bit.  The benchmark times such replays."""
import numpy as np
import pytest
import torch

from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


@pytest.mark.parametrize("fused", [False, True])
def test_graph_replays_match_eager(fused):
    lay = W.make_layout("mid", seed=12, num_requests=6, ctx=("uniform", 300, 2500))
    inp = W.make_attention_inputs(lay, DEV)
    inp.update(W.make_logit_inputs(lay, DEV))
    page_idx = torch.as_tensor(lay.page_indices, device=DEV)
    rp = torch.as_tensor(lay.row_indptr, device=DEV)
    layout = binding.make_layout(inp["q"], inp["k_cache"], lay.q_indptr, lay.n_verify, lay.ctx_len,
                                 lay.page_indptr, page_idx)
    ws = binding.new_workspace(binding.attention_workspace_bytes(layout), DEV)
    vws = binding.new_workspace(binding.verify_accept_workspace_bytes(
        lay.num_requests, lay.total_verify_rows, lay.spec.vocab), DEV)
    dws = binding.new_workspace(binding.draft_confidence_workspace_bytes(lay.total_draft_rows, lay.spec.vocab), DEV)
    rws = binding.new_workspace(binding.verify_and_confidence_workspace_bytes(
        lay.num_requests, lay.total_verify_rows, lay.total_draft_rows, lay.spec.vocab), DEV)
    out = torch.empty_like(inp["q"])
    lse = torch.empty(inp["q"].shape[0], lay.spec.num_q_heads, dtype=torch.float32, device=DEV)
    vout = dict(row_argmax=torch.empty(lay.total_verify_rows, dtype=torch.int32, device=DEV),
                accept_len=torch.empty(lay.num_requests, dtype=torch.int32, device=DEV),
                next_token=torch.empty(lay.num_requests, dtype=torch.int32, device=DEV),
                row_entropy=torch.empty(lay.total_verify_rows, dtype=torch.float32, device=DEV),
                accept_entropy=torch.empty(lay.num_requests, dtype=torch.float32, device=DEV))
    dout = {k: torch.empty(lay.total_draft_rows, dtype=dt, device=DEV)
            for k, dt in (("top1", torch.int32), ("top2", torch.int32), ("p1", torch.float32),
                          ("p2", torch.float32), ("margin", torch.float32), ("entropy", torch.float32))}

    def step():
        binding.draft_verify_attention(inp["q"], inp["k_cache"], inp["v_cache"], None, None, None, None,
                                       page_idx, out=out, lse=lse, workspace=ws, layout=layout)
        if fused:
            binding.verify_and_confidence(inp["verify_logits"], rp, inp["draft_tokens"], inp["draft_logits"],
                                          workspace=rws, out_verify=vout, out_draft=dout)
        else:
            binding.verify_accept(inp["verify_logits"], rp, inp["draft_tokens"], workspace=vws, out=vout)
            binding.draft_confidence(inp["draft_logits"], workspace=dws, out=dout)

    step()
    torch.cuda.synchronize()
    eager = [out.clone(), lse.clone()] + [t.clone() for t in vout.values()] + [t.clone() for t in dout.values()]
    assert binding.attention_plan(layout)["split_requests"] > 0  # the combine kernel is part of the graph

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in [out, lse] + list(vout.values()) + list(dout.values()):
            t.zero_()
        noise = torch.randn(1 << 20, device=DEV).sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [out, lse] + list(vout.values()) + list(dout.values())
        for a, b in zip(got, eager):
            assert torch.equal(a, b), f"replay {rep} differs"
        assert torch.isfinite(noise)
