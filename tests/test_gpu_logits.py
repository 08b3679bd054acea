"""GPU parity of rg_verify_accept and rg_draft_confidence against the fp64
oracle.

Integer outputs (argmax, top-1/top-2 indices, accept lengths, next tokens)
must be bit-exact, ties broken to the lowest index.  p1, p2, entropies and
e_t within 1e-4 relative; the margin within 1e-4 * p1 absolute (it is a
difference); p2 gets an absolute floor of 1e-30 (fp32 underflow).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
RTOL = 1e-4


def rel_ok(got, want, rtol=RTOL, floor=0.0):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    bad = ~(np.abs(got - want) <= rtol * np.abs(want) + floor)  # NaN counts as a mismatch
    assert not bad.any(), f"{bad.sum()} mismatches, worst got {got[bad][:3]} want {want[bad][:3]}"


def check_verify(logits, row_indptr, tokens, res):
    ref = oracle.oracle_accept(W.bf16_bits(logits), row_indptr, tokens.cpu().numpy())
    np.testing.assert_array_equal(res["row_argmax"].cpu().numpy(), ref["row_argmax"])
    np.testing.assert_array_equal(res["accept_len"].cpu().numpy(), ref["accept_len"])
    np.testing.assert_array_equal(res["next_token"].cpu().numpy(), ref["next_token"])
    rel_ok(res["row_entropy"].cpu().numpy(), ref["row_entropy"])
    rel_ok(res["accept_entropy"].cpu().numpy(), ref["accept_entropy"], floor=1e-30)


def check_draft(logits, res):
    ref = oracle.oracle_confidence(W.bf16_bits(logits))
    np.testing.assert_array_equal(res["top1"].cpu().numpy(), ref["top1"])
    np.testing.assert_array_equal(res["top2"].cpu().numpy(), ref["top2"])
    rel_ok(res["p1"].cpu().numpy(), ref["p1"])
    rel_ok(res["p2"].cpu().numpy(), ref["p2"], floor=1e-30)
    m = res["margin"].double().cpu().numpy()
    assert (np.abs(m - ref["margin"]) <= RTOL * ref["p1"]).all()
    rel_ok(res["entropy"].cpu().numpy(), ref["entropy"])


def run_verify(lay, inp, **kw):
    rp = torch.as_tensor(lay.row_indptr, device=DEV)
    res = binding.verify_accept(inp["verify_logits"], rp, inp["draft_tokens"], **kw)
    torch.cuda.synchronize()
    return res


def run_draft(logits, **kw):
    res = binding.draft_confidence(logits, **kw)
    torch.cuda.synchronize()
    return res


@pytest.mark.parametrize("name", ["tiny", "low", "low_sigma2", "mid", "high", "long"])
def test_configs_full(name):
    lay = W.make_layout(name, seed=0)
    inp = W.make_logit_inputs(lay, DEV)
    res = run_verify(lay, inp)
    check_verify(inp["verify_logits"], lay.row_indptr, inp["draft_tokens"], res)
    check_draft(inp["draft_logits"], run_draft(inp["draft_logits"]))


@pytest.mark.parametrize("variant", ["sigma0", "ties", "spike", "bonus"])
def test_variants(variant):
    kw = dict(num_requests=6)
    lay = W.make_layout("mid", seed=3, bonus_rows=(variant == "bonus"), **kw)
    inp = W.make_logit_inputs(lay, DEV, sigma=0.0 if variant in ("sigma0", "bonus") else None,
                              ties=(variant == "ties"), spike=12.0 if variant == "spike" else None)
    res = run_verify(lay, inp)
    check_verify(inp["verify_logits"], lay.row_indptr, inp["draft_tokens"], res)
    if variant == "sigma0":
        assert (res["accept_len"].cpu().numpy() == lay.n_verify).all()
    check_draft(inp["draft_logits"], run_draft(inp["draft_logits"]))


def test_peaked_rows_entropy_accuracy():
    g = torch.Generator(device=DEV).manual_seed(1)
    x = torch.randn(64, 50000, generator=g, device=DEV) * 2.0
    x[torch.arange(64), torch.arange(64) * 700] += torch.linspace(5, 60, 64, device=DEV)
    logits = x.to(torch.bfloat16)
    check_draft(logits, run_draft(logits))


def test_extremes_at_every_lane_row_and_wave():
    """Maxima, runners-up and duplicated maxima placed in each 16-lane row of
    each wave of a chunk's work group (thread t of the group holds entries
    (u * 256 + t) * 8 + j of its chunk), so every step of the in-wave
    reductions and of the merge across waves decides some row."""
    vocab = 2 * 8192 + 100
    lanes = [0, 15, 16, 31, 32, 47, 48, 63]
    rows = []
    g = torch.Generator(device="cpu").manual_seed(11)
    for w in range(4):
        for li, lane in enumerate(lanes):
            for chunk in (0, 1):
                base = torch.randn(vocab, generator=g) * 0.5
                at = chunk * 8192 + ((li % 4) * 256 + w * 64 + lane) * 8 + (li % 8)
                other = ((li + 1) % 4 * 256 + (w + 1) % 4 * 64 + lanes[(li + 3) % 8]) * 8 + 5
                base[at] = 6.0
                base[other] = 5.0  # runner-up in another wave, row and chunk
                rows.append(base.clone())
                dup = base.clone()
                dup[other] = 6.0  # the maximum twice: the lower index is top-1
                rows.append(dup)
    logits = torch.stack(rows).to(torch.bfloat16).to(DEV)
    check_draft(logits, run_draft(logits))
    n = logits.shape[0]
    rp = torch.tensor([0, n // 2, n], dtype=torch.int32, device=DEV)
    tok = torch.argmax(logits.float(), dim=1).to(torch.int32)
    tok[n // 2 + 7] = (tok[n // 2 + 7] + 1) % vocab
    res = binding.verify_accept(logits, rp, tok)
    torch.cuda.synchronize()
    check_verify(logits, rp.cpu().numpy(), tok, res)


@pytest.mark.parametrize("vocab", [2, 7, 1000, 8192, 8193, 16384, 16385, 128250])
def test_vocab_sizes_and_tails(vocab):
    g = torch.Generator(device=DEV).manual_seed(vocab)
    logits = (torch.randn(9, vocab, generator=g, device=DEV) * 2).to(torch.bfloat16)
    logits[3] = 0.0  # all tied
    check_draft(logits, run_draft(logits))
    rp = torch.tensor([0, 4, 4, 9], dtype=torch.int32, device=DEV)
    tok = torch.argmax(logits.float(), dim=1).to(torch.int32)
    tok[6] = (tok[6] + 1) % vocab
    res = binding.verify_accept(logits, rp, tok)
    torch.cuda.synchronize()
    check_verify(logits, rp.cpu().numpy(), tok, res)


def test_verify_single_entry_vocabulary():
    """rg_verify_accept accepts vocab = 1: every row's argmax is 0 and its
    entropy 0, so a row matches exactly when its token is 0."""
    logits = torch.tensor([[1.5], [-2.0], [0.0], [7.0], [3.0]], dtype=torch.bfloat16, device=DEV)
    rp = torch.tensor([0, 2, 2, 5], dtype=torch.int32, device=DEV)
    tok = torch.tensor([0, 0, 0, -1, 0], dtype=torch.int32, device=DEV)
    res = binding.verify_accept(logits, rp, tok)
    torch.cuda.synchronize()
    check_verify(logits, rp.cpu().numpy(), tok, res)
    assert res["row_argmax"].cpu().tolist() == [0] * 5
    assert res["accept_len"].cpu().tolist() == [2, 0, 1]


def test_masked_vocabulary_entries():
    """Most of each row masked to -1e30 (a finite mask value, as samplers
    write them): the masked entries carry no probability and the statistics
    are those of the unmasked ones; a row with a single unmasked entry has
    p1 = 1 and entropy 0, and the runner-up is the first masked index."""
    g = torch.Generator(device=DEV).manual_seed(11)
    vocab = 40000
    x = torch.randn(8, vocab, generator=g, device=DEV) * 2
    keep = torch.rand(8, vocab, generator=g, device=DEV) < 0.1
    keep[:, 0] = True
    keep[5] = False
    keep[5, 123] = True                  # one unmasked entry
    keep[6] = False
    keep[6, 7] = True
    keep[6, 39999] = True                # two, in different chunks
    x = torch.where(keep, x, torch.full_like(x, -1e30))
    logits = x.to(torch.bfloat16)
    check_draft(logits, run_draft(logits))
    rp = torch.tensor([0, 3, 8], dtype=torch.int32, device=DEV)
    tok = torch.argmax(logits.float(), dim=1).to(torch.int32)
    tok[1] = (tok[1] + 1) % vocab
    res = binding.verify_accept(logits, rp, tok)
    torch.cuda.synchronize()
    check_verify(logits, rp.cpu().numpy(), tok, res)


def test_row_stride_and_unaligned_rows():
    g = torch.Generator(device=DEV).manual_seed(5)
    base = (torch.randn(12, 20011, generator=g, device=DEV) * 2).to(torch.bfloat16)
    strided = base[:, :20000]            # row stride 20011 > vocab, rows not 16-byte aligned
    assert strided.stride(0) == 20011
    check_draft(strided, run_draft(strided))
    shifted = base.view(-1)[1:1 + 12 * 20000].view(12, 20000)  # misaligned base
    check_draft(shifted, run_draft(shifted))
    rp = torch.tensor([0, 5, 12], dtype=torch.int32, device=DEV)
    tok = torch.argmax(shifted.float(), dim=1).to(torch.int32)
    res = binding.verify_accept(shifted, rp, tok)
    torch.cuda.synchronize()
    check_verify(shifted, rp.cpu().numpy(), tok, res)


def test_empty_requests_and_workspace_reuse():
    lay = W.make_layout("high", seed=4, num_requests=40)
    counts = lay.n_verify.copy()
    counts[::3] = 0
    lay.row_indptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    rows = int(lay.row_indptr[-1])
    inp = W.make_logit_inputs(lay, DEV)
    ws = binding.new_workspace(binding.verify_accept_workspace_bytes(40, rows, lay.spec.vocab), DEV)
    first = run_verify(lay, inp, workspace=ws)
    check_verify(inp["verify_logits"], lay.row_indptr, inp["draft_tokens"], first)
    ws.fill_(0xFF)  # workspace contents must not matter
    second = run_verify(lay, inp, workspace=ws)
    for k in first:
        assert torch.equal(first[k], second[k]), k
    dws = binding.new_workspace(binding.draft_confidence_workspace_bytes(rows, lay.spec.vocab), DEV)
    a = run_draft(inp["verify_logits"], workspace=dws)
    b = run_draft(inp["verify_logits"], workspace=dws)
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("rows,reqs", [(16, 9), (17, 9), (16, 1), (40, 300), (16, 200), (8, 255), (8, 256)])
def test_finalize_group_layouts(rows, reqs):
    """Requests of many sizes (empty ones among them, more requests than a
    work group has threads) over a 16-chunk vocabulary give the oracle's
    accept lengths, next tokens and e_t (200 to 256 requests over 8 or 16
    rows: mostly empty requests, every one finalised)."""
    vocab = 128250  # 16 chunks of 8192 entries: 16 lanes per row
    g = torch.Generator(device=DEV).manual_seed(rows * 1000 + reqs)
    logits = (torch.randn(rows, vocab, generator=g, device=DEV) * 2).to(torch.bfloat16)
    cuts = np.sort(np.random.default_rng(rows + reqs).integers(0, rows + 1, size=reqs - 1))
    rp = np.concatenate([[0], cuts, [rows]]).astype(np.int32)  # some requests empty
    tok = torch.argmax(logits.float(), dim=1).to(torch.int32)
    tok[rows // 2] = (tok[rows // 2] + 1) % vocab
    res = binding.verify_accept(logits, torch.as_tensor(rp, device=DEV), tok)
    torch.cuda.synchronize()
    check_verify(logits, rp, tok, res)


def test_no_verify_rows_at_all():
    rp = torch.zeros(4, dtype=torch.int32, device=DEV)
    logits = torch.empty(0, 128, dtype=torch.bfloat16, device=DEV)
    tok = torch.empty(0, dtype=torch.int32, device=DEV)
    res = binding.verify_accept(logits, rp, tok)
    torch.cuda.synchronize()
    assert res["accept_len"].tolist() == [0, 0, 0]
    assert res["next_token"].tolist() == [-1, -1, -1]
    assert res["accept_entropy"].tolist() == [0.0, 0.0, 0.0]


def _same(a, b):
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("case", ["tiny", "low", "high", "bonus_ties", "no_draft_rows", "empty_requests"])
def test_fused_round_matches_separate_calls(case):
    """rg_verify_and_confidence gives the two separate calls' results bit for
    bit (same arithmetic, fewer launches), and so matches the oracle."""
    if case == "bonus_ties":
        lay = W.make_layout("mid", seed=8, num_requests=5, bonus_rows=True)
        inp = W.make_logit_inputs(lay, DEV, ties=True)
    elif case == "empty_requests":
        lay = W.make_layout("high", seed=9, num_requests=7, verify=("choice", (0, 4), None))
        inp = W.make_logit_inputs(lay, DEV)
    else:
        lay = W.make_layout("mid" if case == "no_draft_rows" else case, seed=7, num_requests=None if case != "no_draft_rows" else 3,
                            draft=("fixed", 0) if case == "no_draft_rows" else None)
        inp = W.make_logit_inputs(lay, DEV)
    rp = torch.as_tensor(lay.row_indptr, device=DEV)
    ws = binding.new_workspace(binding.verify_and_confidence_workspace_bytes(
        lay.num_requests, lay.total_verify_rows, lay.total_draft_rows, lay.spec.vocab), DEV)
    ws.fill_(0xFF)  # contents must not matter
    fv, fd = binding.verify_and_confidence(inp["verify_logits"], rp, inp["draft_tokens"], inp["draft_logits"],
                                           workspace=ws)
    torch.cuda.synchronize()
    sv = run_verify(lay, inp)
    _same(sv, fv)
    if lay.total_draft_rows:
        sd = run_draft(inp["draft_logits"])
        _same(sd, fd)
        check_draft(inp["draft_logits"], fd)
    check_verify(inp["verify_logits"], lay.row_indptr, inp["draft_tokens"], fv)


@pytest.mark.parametrize("i", range(12))
def test_random_rounds(i):
    """Seeded random rounds through rg_verify_and_confidence: vocabulary size,
    requests (some without verify rows), row counts, sharp or flat rows, exact
    ties and draft tokens that match the argmax for a random prefix of each
    request, against the oracle."""
    r = np.random.default_rng(3000 + i)
    vocab = int(r.choice([2, 3, 100, 4097, 8191, 8192, 20000, 65537, 128256, 151936]))
    R = int(r.integers(1, 24))
    nv = r.integers(0, 10, R)
    nv[r.random(R) < 0.2] = 0
    nd_total = int(r.integers(0, 60))
    rows_v = int(nv.sum())
    g = torch.Generator(device="cpu").manual_seed(i)
    def rows(n):
        x = torch.randn(n, vocab, generator=g) * float(r.choice([0.5, 2.0, 6.0]))
        if n and vocab > 4:
            k = torch.randint(0, vocab, (n,), generator=g)
            x[torch.arange(n), k] += float(r.choice([0.0, 8.0, 30.0]))  # sharp rows
            x[: n // 3, 1] = x[: n // 3].max(dim=1).values  # exact ties with the maximum
        return x.to(torch.bfloat16).to(DEV)
    vlog, dlog = rows(rows_v), rows(nd_total)
    rp = torch.as_tensor(np.concatenate([[0], np.cumsum(nv)]).astype(np.int32), device=DEV)
    tok = torch.argmax(vlog.float(), dim=1).to(torch.int32) if rows_v else torch.zeros(0, dtype=torch.int32, device=DEV)
    if rows_v:
        flip = torch.as_tensor(r.random(rows_v) < 0.3, device=DEV)
        tok = torch.where(flip, (tok + 1) % vocab, tok)
        tok[torch.as_tensor(r.random(rows_v) < 0.05, device=DEV)] = -1  # bonus rows
    ws = binding.new_workspace(binding.verify_and_confidence_workspace_bytes(R, rows_v, nd_total, vocab), DEV)
    fv, fd = binding.verify_and_confidence(vlog, rp, tok, dlog, workspace=ws)
    torch.cuda.synchronize()
    check_verify(vlog, rp.cpu().numpy(), tok, fv)
    if nd_total:
        check_draft(dlog, fd)
