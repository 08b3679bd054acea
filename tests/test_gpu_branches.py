"""GPU parity of the predictive draft-verify overlap entry points against the
fp64 oracle: rg_multibranch_attention (branches sharing the canonical
prefix), rg_plan_branches and rg_match_branches.

Tolerances as for the fused step: per (row, head) max |error| <= 1e-2 x the
row's L2 norm, lse within 2e-3; integer outputs bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
ATOL_ROW = 1e-2
LSE_ATOL = 2e-3  # log1p(2^-9): bf16-rounded probabilities in the row sum


def _layout(ctx, nv, branches, hq=8, hkv=2, D=128, seed=0):
    """A synthetic request batch whose rows after the verify rows are the
    listed branches."""
    nd = [sum(b[2] for b in br) for br in branches]
    R = len(ctx)
    spec = W.WorkloadSpec("custom", 9, R, hq, hkv, D, 1024, ("fixed", 0), ("fixed", 0), ("fixed", 0),
                          ("fixed", 1.0), 1.0 / np.sqrt(D))
    lay = W.make_layout(spec, seed=seed)
    lay.ctx_len = np.asarray(ctx, dtype=np.int32)
    lay.n_verify = np.asarray(nv, dtype=np.int32)
    lay.n_draft = np.asarray(nd, dtype=np.int32)
    q_len = lay.n_verify + lay.n_draft
    T = lay.ctx_len + q_len
    pages = (T + 15) // 16
    lay.q_indptr = np.concatenate([[0], np.cumsum(q_len)]).astype(np.int32)
    lay.page_indptr = np.concatenate([[0], np.cumsum(pages)]).astype(np.int32)
    lay.num_pages = int(pages.sum()) + 5
    rng = np.random.default_rng(seed + 100)
    lay.page_indices = rng.permutation(lay.num_pages)[:int(pages.sum())].astype(np.int32)
    lay.row_indptr = np.concatenate([[0], np.cumsum(lay.n_verify)]).astype(np.int32)
    lay.draft_row_indptr = np.concatenate([[0], np.cumsum(lay.n_draft)]).astype(np.int32)
    return lay


def _branch_arrays(branches):
    indptr = np.concatenate([[0], np.cumsum([len(b) for b in branches])]).astype(np.int32)
    flat = [b for br in branches for b in br]
    col = lambda i: np.array([b[i] for b in flat], dtype=np.int32)
    return indptr, col(0), col(1), col(2)


def _run(lay, inp, branches):
    pidx = torch.as_tensor(lay.page_indices, device=DEV)
    L = binding.make_layout(inp["q"], inp["k_cache"], lay.q_indptr, lay.n_verify, lay.ctx_len,
                            lay.page_indptr, pidx)
    B = binding.make_branches(*_branch_arrays(branches))
    out, lse = binding.multibranch_attention(inp["q"], inp["k_cache"], inp["v_cache"], L, B)
    torch.cuda.synchronize()
    return out, lse


def _check(out, lse, ref, rows=None):
    got, want = out.double().cpu().numpy(), ref["out"]
    gl, wl = lse.double().cpu().numpy(), ref["lse"]
    if rows is not None:
        got, want, gl, wl = got[rows], want[rows], gl[rows], wl[rows]
    assert np.isfinite(got).all()
    norm = np.maximum(np.linalg.norm(want, axis=-1), 1e-6)
    err = np.abs(got - want).max(axis=-1) / norm
    assert err.max() <= ATOL_ROW, f"max row error {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}"
    assert np.abs(gl - wl).max() <= LSE_ATOL


def _reference(lay, inp, branches, requests=None):
    return oracle.oracle_branch_attention(W.bf16_bits(inp["q"]), W.bf16_bits(inp["k_cache"]),
                                          W.bf16_bits(inp["v_cache"]), lay.q_indptr, lay.n_verify, lay.ctx_len,
                                          lay.page_indptr, lay.page_indices, branches, requests=requests)


CASES = {
    # two corrections (lead 1) and a continuation per request, one request without branches
    "overlap": ([300, 57, 1000], [8, 4, 16],
                [[(2, 1, 6), (5, 1, 6), (8, 0, 8)], [], [(0, 1, 3), (16, 0, 12)]]),
    # a branch that keeps no verify row, tiny rows, a lead-only branch
    "edges": ([0, 5, 40], [3, 1, 0], [[(0, 0, 2), (3, 2, 2)], [(1, 1, 1)], [(0, 1, 1), (0, 0, 4)]]),
    # long context: split over chunks, branches in the last chunk
    "split": ([2500, 1300], [16, 4], [[(3, 1, 16), (9, 1, 16), (16, 0, 16)], [(4, 0, 9)]]),
    # many columns: 64 rows = 256 columns of one KV head (8 tiles)
    "wide": ([700], [16], [[(5, 1, 16), (11, 1, 16), (16, 0, 16)]]),
    # chunk boundaries between a branch's kept prefix and its own rows (the
    # first branch spans more keys than any chunk)
    "gap": ([3000, 700], [4, 2], [[(0, 0, 600), (1, 1, 5), (4, 0, 7)], [(0, 1, 300), (2, 0, 3)]]),
    # one draft block per hypothetical accepted length (a regular family of V + 1 branches)
    "quadratic": ([260, 31], [8, 3], [[(a, 0, 4) for a in range(9)], [(a, 0, 5) for a in range(4)]]),
    # two single branches, then a family with prefix step 2 and lead rows
    "family": ([500], [9], [[(4, 1, 3), (0, 0, 2)] + [(a, 1, 3) for a in range(1, 10, 2)]]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_multibranch_attention_matches_oracle(name):
    ctx, nv, branches = CASES[name]
    lay = _layout(ctx, nv, branches, seed=len(name))
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    out, lse = _run(lay, inp, branches)
    _check(out, lse, _reference(lay, inp, branches))


def _random_branch_case(i):
    """Seeded random batch i: per request up to three branches of any shape,
    or a regular family (equal rows and lead, prefixes growing by a step),
    over random contexts, GQA groups and head sizes, with a forced or
    automatic chunk size."""
    r = np.random.default_rng(2000 + i)
    R = int(r.integers(1, 5))
    hkv = int(r.choice([1, 2, 4]))
    g = int(r.choice([1, 2, 4]))
    D = int(r.choice([64, 128]))
    ctx, nv, branches = [], [], []
    for _ in range(R):
        v = int(r.integers(0, 12))
        kind = r.choice(["none", "free", "family"], p=[0.2, 0.45, 0.35])
        br = []
        if kind == "free" or (kind == "none" and v == 0):
            for _ in range(int(r.integers(1, 4))):
                rows = int(r.integers(1, 20))
                br.append((int(r.integers(0, v + 1)), int(r.integers(0, min(rows, 15) + 1)), rows))
        elif kind == "family":
            k, rows = int(r.integers(2, 7)), int(r.integers(1, 9))
            lead = int(r.integers(0, min(rows, 15) + 1))
            step = int(r.integers(0, v // (k - 1) + 1))  # prefixes p0 + j step stay within 0 .. V
            p0 = int(r.integers(0, v - (k - 1) * step + 1))
            br = [(p0 + j * step, lead, rows) for j in range(k)]
        ctx.append(int(r.integers(0, 1500)))
        nv.append(v)
        branches.append(br)
    chunk = str(int(r.choice([0, 128, 256, 512])))
    return ctx, nv, branches, dict(hq=hkv * g, hkv=hkv, D=D), chunk


@pytest.mark.parametrize("i", range(16))
def test_random_branch_layouts(monkeypatch, i):
    ctx, nv, branches, shape, chunk = _random_branch_case(i)
    if chunk != "0":
        monkeypatch.setenv("RG_ATTN_CHUNK", chunk)
    lay = _layout(ctx, nv, branches, seed=i, **shape)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    out, lse = _run(lay, inp, branches)
    _check(out, lse, _reference(lay, inp, branches))


@pytest.mark.parametrize("name", ["overlap", "split", "gap", "quadratic"])
def test_multibranch_one_launch_mode_matches_oracle(monkeypatch, name):
    """The branched plans in the one-launch work-queue mode (RG_ATTN_PERSIST=1),
    every request split over 128-key chunks, against the oracle."""
    monkeypatch.setenv("RG_ATTN_PERSIST", "1")
    monkeypatch.setenv("RG_ATTN_CHUNK", "128")
    ctx, nv, branches = CASES[name]
    lay = _layout(ctx, nv, branches, seed=len(name) + 40)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    out, lse = _run(lay, inp, branches)
    _check(out, lse, _reference(lay, inp, branches))


def test_no_branches_is_the_fused_step_bit_for_bit():
    ctx, nv = [300, 57, 1000], [8, 4, 16]
    branches = [[(nv[0], 0, 11)], [], []]
    lay = _layout(ctx, nv, [[(nv[0], 0, 11)], [(nv[1], 0, 7)], [(nv[2], 0, 16)]], seed=3)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    out_b, lse_b = _run(lay, inp, branches)
    pidx = torch.as_tensor(lay.page_indices, device=DEV)
    out_p, lse_p = binding.draft_verify_attention(inp["q"], inp["k_cache"], inp["v_cache"], lay.q_indptr,
                                                  lay.n_verify, lay.ctx_len, lay.page_indptr, pidx)
    torch.cuda.synchronize()
    assert torch.equal(out_b, out_p) and torch.equal(lse_b, lse_p)


def test_branch_keys_never_leak_into_other_branches():
    """Huge values in one branch's K/V (and in the verify rows past another
    branch's prefix) leave the rows that must not see them unchanged."""
    ctx, nv, branches = [200], [8], [[(3, 1, 5), (8, 0, 6)]]
    lay = _layout(ctx, nv, branches, seed=5)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    base, _ = _run(lay, inp, branches)
    k2, v2 = inp["k_cache"].clone(), inp["v_cache"].clone()
    L, V = ctx[0], nv[0]
    for j in list(range(L + V + 5, L + V + 11)) + list(range(L + 3, L + V)):  # branch 1's rows, verify rows 3..7
        page = int(lay.page_indices[int(lay.page_indptr[0]) + j // 16])
        k2[page, :, j % 16, :] = 30.0
        v2[page, :, :, j % 16] = 1e4
    inp2 = dict(inp, k_cache=k2, v_cache=v2)
    out2, _ = _run(lay, inp2, branches)
    rows_b0 = slice(V, V + 5)
    assert torch.equal(out2[rows_b0], base[rows_b0])
    assert torch.equal(out2[:3], base[:3])


def test_multibranch_full_size_low_shape_sampled():
    """The batch-1 shape of the benchmark with an overlap round: 16 verify
    rows, two correction branches (1 + 15 rows) and a 16-row continuation,
    4096 context tokens, 32 / 8 heads; the oracle recomputes it."""
    ctx, nv = [4096], [16]
    branches = [[(3, 1, 16), (9, 1, 16), (16, 0, 16)]]
    lay = _layout(ctx, nv, branches, hq=32, hkv=8, seed=11)
    inp = W.make_attention_inputs(lay, DEV, poison=float("nan"))
    out, lse = _run(lay, inp, branches)
    ref = oracle.oracle_branch_attention(W.bf16_bits(inp["q"]), W.bf16_bits(inp["k_cache"]),
                                         W.bf16_bits(inp["v_cache"]), lay.q_indptr, lay.n_verify, lay.ctx_len,
                                         lay.page_indptr, lay.page_indices, branches, heads=[0, 5, 13, 31])
    for h in (0, 5, 13, 31):
        _check(out[:, h:h + 1], lse[:, h:h + 1], dict(out=ref["out"][:, h:h + 1], lse=ref["lse"][:, h:h + 1]))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_plan_and_match_branches_match_oracle(seed):
    rng = np.random.default_rng(seed)
    R = 300
    lens = rng.integers(0, 70, size=R)               # some blocks empty, some past one wave
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    rows = int(rp[-1])
    margin = (rng.random(rows) ** 3).astype(np.float32)  # many below 0.5
    margin[rng.random(rows) < 0.05] = np.float32(0.5)    # the threshold itself is not risky
    top2 = rng.integers(0, 128256, size=rows).astype(np.int32)
    delta = 0.5
    got = binding.plan_branches(torch.as_tensor(margin, device=DEV), torch.as_tensor(top2, device=DEV),
                                torch.as_tensor(rp, device=DEV), delta)
    torch.cuda.synchronize()
    want = oracle.oracle_plan_branches(margin, top2, rp, np.float32(delta))
    for k in ("n_risky", "n_corr", "corr_pos", "corr_tok", "continuation"):
        np.testing.assert_array_equal(got[k].cpu().numpy(), want[k], err_msg=k)
    # outcomes: every prepared branch hit, and near misses
    accept = np.zeros(R, dtype=np.int32)
    nxt = np.zeros(R, dtype=np.int32)
    cont_first = rng.integers(0, 50, size=R).astype(np.int32)
    for r in range(R):
        kind = r % 5
        if kind == 0 and want["n_corr"][r] > 0:
            c = r % int(want["n_corr"][r])
            accept[r], nxt[r] = want["corr_pos"][r, c], want["corr_tok"][r, c]
        elif kind == 1 and want["n_corr"][r] > 0:
            accept[r], nxt[r] = want["corr_pos"][r, 0], want["corr_tok"][r, 0] + 1
        elif kind == 2:
            accept[r], nxt[r] = lens[r], cont_first[r]
        elif kind == 3:
            accept[r], nxt[r] = lens[r], cont_first[r] + 1
        else:
            accept[r], nxt[r] = rng.integers(0, lens[r] + 1), rng.integers(0, 50)
    tt = lambda a: torch.as_tensor(np.ascontiguousarray(a, dtype=np.int32), device=DEV)
    reused = binding.match_branches(tt(accept), tt(nxt), tt(lens), got, tt(cont_first))
    torch.cuda.synchronize()
    want_r = oracle.oracle_match_branches(accept, nxt, lens, want["n_corr"], want["corr_pos"], want["corr_tok"],
                                          want["continuation"], cont_first)
    np.testing.assert_array_equal(reused.cpu().numpy(), want_r)
    assert (want_r >= 0).sum() > R // 10  # the outcomes above do hit branches


@pytest.mark.parametrize("workload", ["mid", "high", "long"])
def test_overlap_round_full_size(workload):
    """A full-size overlap round (every request with two correction branches
    and a continuation, the layout the benchmark times): sampled requests
    against the oracle, and every row against the same rows served as
    separate requests (each branch with its own copy of the kept prefix)
    through rg_draft_verify_attention.  At `long` the sampled requests
    include the one with the most rows (several 256-column groups) and the
    one with the most keys."""
    lay = W.make_layout(workload, seed=4)
    branches = W.overlap_branches(lay)
    ov = W.make_overlap_layout(lay, branches)
    inp = W.make_attention_inputs(ov, DEV, poison=float("nan"))
    out, lse = _run(ov, inp, branches)
    rng = np.random.default_rng(4)
    reqs = sorted(rng.choice(ov.num_requests, size=min(3, ov.num_requests), replace=False).tolist())
    if workload == "long":
        reqs = sorted(set(reqs) | {int(np.argmax(ov.q_len)), int(np.argmax(ov.kv_len))})
        assert int(ov.q_len.max()) * (ov.spec.num_q_heads // ov.spec.num_kv_heads) > 256
    heads = [0, 13, 31]
    ref = oracle.oracle_branch_attention(W.bf16_bits(inp["q"]), W.bf16_bits(inp["k_cache"]),
                                         W.bf16_bits(inp["v_cache"]), ov.q_indptr, ov.n_verify, ov.ctx_len,
                                         ov.page_indptr, ov.page_indices, branches, requests=reqs, heads=heads)
    for r in reqs:
        q0, q1 = int(ov.q_indptr[r]), int(ov.q_indptr[r + 1])
        for h in heads:
            _check(out[q0:q1, h:h + 1], lse[q0:q1, h:h + 1],
                   dict(out=ref["out"][q0:q1, h:h + 1], lse=ref["lse"][q0:q1, h:h + 1]))
    sep, origin = W.make_separate_layout(ov, branches)
    k2, v2 = W.make_separate_kv(ov, branches, sep, origin, inp["k_cache"], inp["v_cache"])
    sidx = torch.as_tensor(sep.page_indices, device=DEV)
    out_s, lse_s = binding.draft_verify_attention(inp["q"], k2, v2, sep.q_indptr, sep.n_verify, sep.ctx_len,
                                                  sep.page_indptr, sidx)
    torch.cuda.synchronize()
    a, b = out.double(), out_s.double()
    err = ((a - b).abs().amax(-1) / b.norm(dim=-1).clamp_min(1e-6)).max().item()
    assert err <= 2 * ATOL_ROW
    assert (lse.double() - lse_s.double()).abs().max().item() <= 2 * LSE_ATOL


def test_quadratic_layout_full_size_low_shape():
    """The batch-1 shape (4096 context tokens, V = B = 16, 32 / 8 heads) in the
    quadratic layout: 17 draft blocks of 16 rows, 288 rows in all, so five
    256-column groups; sampled heads against the oracle."""
    lay = W.make_layout("low", seed=6)
    branches = W.quadratic_branches(lay)
    ov = W.make_overlap_layout(lay, branches)
    assert ov.total_q == 16 + 17 * 16
    inp = W.make_attention_inputs(ov, DEV, poison=float("nan"))
    out, lse = _run(ov, inp, branches)
    heads = [0, 17, 31]
    ref = oracle.oracle_branch_attention(W.bf16_bits(inp["q"]), W.bf16_bits(inp["k_cache"]),
                                         W.bf16_bits(inp["v_cache"]), ov.q_indptr, ov.n_verify, ov.ctx_len,
                                         ov.page_indptr, ov.page_indices, branches, heads=heads)
    for h in heads:
        _check(out[:, h:h + 1], lse[:, h:h + 1], dict(out=ref["out"][:, h:h + 1], lse=ref["lse"][:, h:h + 1]))
