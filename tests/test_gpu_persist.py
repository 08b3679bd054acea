"""GPU parity of the one-launch work-queue attention (RG_ATTN_PERSIST=1: split
requests merged in the same launch) against the fp64 oracle, and of the
default two-launch mode beside it.

Besides the output tolerance of the attention tests (per row and head,
max |error| <= 1e-2 x the oracle row's L2 norm; lse within 2e-3), every call
must leave the workspace's synchronisation words at zero (queue head, exit
count, per-column-group counters) and its error word clear, so the next call
on the same workspace starts clean.  Reuse is checked with different inputs
on one workspace, call after call and under graph replay.
"""
import numpy as np
import pytest
import torch

from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W
from tests.test_gpu_attention import _custom, check, reference

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def _layout_handle(lay, inp):
    return binding.make_layout(inp["q"], inp["k_cache"], lay.q_indptr, lay.n_verify, lay.ctx_len,
                               lay.page_indptr, torch.as_tensor(lay.page_indices, device=DEV))


def _run(lay, inp, ws, handle=None):
    handle = handle or _layout_handle(lay, inp)
    page_idx = torch.as_tensor(lay.page_indices, device=DEV)
    out, lse = binding.draft_verify_attention(inp["q"], inp["k_cache"], inp["v_cache"], lay.q_indptr,
                                              lay.n_verify, lay.ctx_len, lay.page_indptr, page_idx,
                                              workspace=ws, layout=handle)
    return out, lse


def _sync_words(ws, info):
    off, n = info["sync_offset"], info["sync_words"]
    assert off >= 0 and off % 4 == 0 and n > 0
    return ws[off:off + 4 * n].view(torch.int32)


@pytest.mark.parametrize("persist", ["1", "0"])
@pytest.mark.parametrize("case", [
    dict(kind="mid", n=4, ctx=(200, 1500)),
    dict(ctx=[129], nv=[32], nd=[38]),                   # 280 columns: two column groups
    dict(ctx=[700, 0, 33], nv=[8, 0, 3], nd=[8, 0, 2], D=64, hq=4, hkv=1),
    dict(ctx=[1000, 5], nv=[2, 1], nd=[2, 0], hq=4, hkv=4),
    dict(ctx=[900], nv=[0], nd=[1]),                     # one query row
    dict(ctx=[40000], nv=[4], nd=[4]),                   # one request, 626 items: queue past the first round
])
def test_split_parity_both_modes(monkeypatch, persist, case):
    monkeypatch.setenv("RG_ATTN_PERSIST", persist)
    monkeypatch.setenv("RG_ATTN_CHUNK", "128")  # every request longer than 128 keys is split
    if "kind" in case:
        lay = W.make_layout(case["kind"], seed=21, num_requests=case["n"], ctx=("uniform",) + case["ctx"])
    else:
        kw = {k: case[k] for k in ("hq", "hkv", "D") if k in case}
        lay = _custom(len(case["ctx"]), case["ctx"], case["nv"], case["nd"], seed=22, **kw)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    handle = _layout_handle(lay, inp)
    info = binding.attention_plan(handle)
    assert info["split_requests"] >= 1
    assert info["persistent_launches"] == (info["num_launches"] if persist == "1" else 0)
    ws = binding.new_workspace(info["workspace_bytes"], DEV)
    out, lse = _run(lay, inp, ws, handle)
    torch.cuda.synchronize()
    check(out, lse, reference(lay, inp))
    assert int(_sync_words(ws, info).abs().sum()) == 0
    assert binding.attention_check(ws) == 0


def test_check_reports_and_clears_the_report_word(monkeypatch):
    """rg_draft_verify_attention_check reads the report word a one-launch
    call leaves when a wait gave up (raised here from the host: no wait is
    made to give up on the device), returns RG_ERR_WAIT once and clears it;
    the next one-launch call on the workspace runs normally."""
    monkeypatch.setenv("RG_ATTN_PERSIST", "1")
    monkeypatch.setenv("RG_ATTN_CHUNK", "128")
    lay = _custom(2, [700, 300], [8, 4], [8, 4], seed=23)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    handle = _layout_handle(lay, inp)
    info = binding.attention_plan(handle)
    ws = binding.new_workspace(info["workspace_bytes"], DEV)
    _sync_words(ws, info)[3] = 7
    assert binding.attention_check(ws) == 6
    assert int(_sync_words(ws, info)[3]) == 0
    assert binding.attention_check(ws) == 0
    out, lse = _run(lay, inp, ws, handle)
    check(out, lse, reference(lay, inp))
    assert binding.attention_check(ws) == 0
    assert int(_sync_words(ws, info).abs().sum()) == 0


def test_modes_agree_and_full_size_low(monkeypatch):
    """The bench's batch-1 shape: both modes within bf16 rounding of each other."""
    lay = W.make_layout("low", seed=0)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    res = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("RG_ATTN_PERSIST", mode)
        handle = _layout_handle(lay, inp)
        info = binding.attention_plan(handle)
        ws = binding.new_workspace(info["workspace_bytes"], DEV)
        res[mode] = _run(lay, inp, ws, handle)
        torch.cuda.synchronize()
        if mode == "1":
            assert info["persistent_launches"] == 1
            assert int(_sync_words(ws, info).abs().sum()) == 0
    a, b = res["1"][0].float(), res["0"][0].float()
    norm = b.norm(dim=-1).clamp_min(1e-6)
    assert float(((a - b).abs().amax(dim=-1) / norm).max()) <= 2e-2 * 0.5
    assert float((res["1"][1] - res["0"][1]).abs().max()) <= 2e-3


@pytest.mark.parametrize("persist", ["1", "0"])
def test_workspace_reuse_with_changing_inputs(monkeypatch, persist):
    """Alternate two different problems (different split counts) on one workspace."""
    monkeypatch.setenv("RG_ATTN_PERSIST", persist)
    monkeypatch.setenv("RG_ATTN_CHUNK", "256")
    lays = [W.make_layout("mid", seed=31, num_requests=3, ctx=("uniform", 300, 1400)),
            W.make_layout("mid", seed=32, num_requests=5, ctx=("uniform", 600, 2000))]
    inps = [W.make_attention_inputs(l, DEV, poison=float("nan")) for l in lays]
    handles = [_layout_handle(l, i) for l, i in zip(lays, inps)]
    infos = [binding.attention_plan(h) for h in handles]
    ws = binding.new_workspace(max(i["workspace_bytes"] for i in infos), DEV)
    refs = [reference(l, i) for l, i in zip(lays, inps)]
    for k in range(6):
        j = k % 2
        out, lse = _run(lays[j], inps[j], ws, handles[j])
        torch.cuda.synchronize()
        check(out, lse, refs[j])
        assert int(_sync_words(ws, infos[j]).abs().sum()) == 0


@pytest.mark.parametrize("persist", ["1", "0"])
def test_graph_replay_alternating_inputs(monkeypatch, persist):
    """A captured call replayed with its inputs rewritten between replays."""
    monkeypatch.setenv("RG_ATTN_PERSIST", persist)
    monkeypatch.setenv("RG_ATTN_CHUNK", "256")
    lay = W.make_layout("mid", seed=41, num_requests=4, ctx=("uniform", 500, 1500))
    # two different problems over the same layout (the second with sharper scores)
    variants = [W.make_attention_inputs(lay, DEV, poison=float("nan"), qk_std=s) for s in (None, 0.4)]
    refs = [reference(lay, v) for v in variants]
    q = variants[0]["q"].clone()
    k = variants[0]["k_cache"].clone()
    v = variants[0]["v_cache"].clone()
    live = dict(q=q, k_cache=k, v_cache=v)
    handle = _layout_handle(lay, live)
    info = binding.attention_plan(handle)
    assert info["persistent_launches"] == (1 if persist == "1" else 0)
    ws = binding.new_workspace(info["workspace_bytes"], DEV)
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=DEV)
    page_idx = torch.as_tensor(lay.page_indices, device=DEV)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        binding.draft_verify_attention(q, k, v, lay.q_indptr, lay.n_verify, lay.ctx_len, lay.page_indptr,
                                       page_idx, out=out, lse=lse, workspace=ws, layout=handle)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        binding.draft_verify_attention(q, k, v, lay.q_indptr, lay.n_verify, lay.ctx_len, lay.page_indptr,
                                       page_idx, out=out, lse=lse, workspace=ws, layout=handle)
    for rep in range(6):
        j = rep % 2
        q.copy_(variants[j]["q"])
        k.copy_(variants[j]["k_cache"])
        v.copy_(variants[j]["v_cache"])
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        check(out, lse, refs[j])
        assert int(_sync_words(ws, info).abs().sum()) == 0


def test_many_requests_several_persistent_launches(monkeypatch):
    monkeypatch.setenv("RG_ATTN_PERSIST", "1")
    monkeypatch.setenv("RG_ATTN_CHUNK", "128")
    lay = W.make_layout("high", seed=51, num_requests=300, ctx=("uniform", 100, 400))
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    handle = _layout_handle(lay, inp)
    info = binding.attention_plan(handle)
    assert info["num_launches"] == 3 and info["persistent_launches"] == 3
    ws = binding.new_workspace(info["workspace_bytes"], DEV)
    out, lse = _run(lay, inp, ws, handle)
    torch.cuda.synchronize()
    check(out, lse, reference(lay, inp))
    assert int(_sync_words(ws, info).abs().sum()) == 0
