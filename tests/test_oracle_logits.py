"""Pins for the oracle's verification / acceptance and draft-confidence
statistics (CPU only): brute force over tiny inputs, closed forms, and
library routines (scipy entropy, torch Categorical, stable argsort)."""
import itertools
import math

import numpy as np
import pytest
import scipy.stats
import torch

from oracle import bf16_bits_to_f64, oracle_accept, oracle_confidence
from paper_2609_34388_amd import workloads as W


def _bits(x) -> np.ndarray:
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _accept_brute(argmaxes, tokens):
    """Accept length as the longest prefix on which every token equals the
    row argmax (max over prefix lengths, not a first-mismatch scan)."""
    V = len(tokens)
    best = 0
    for k in range(V + 1):
        if all(tokens[i] >= 0 and argmaxes[i] == tokens[i] for i in range(k)):
            best = k
    return best


def test_accept_brute_force_all_small_patterns():
    """vocab 3, up to 4 rows, logits from {0, 1} (lots of ties) and every
    token pattern including bonus rows (-1)."""
    vocab = 3
    rng = np.random.default_rng(0)
    cases = 0
    for V in range(0, 5):
        rows_choices = list(itertools.product([0.0, 1.0], repeat=vocab))
        for _ in range(60 if V else 1):
            logits = np.array([rows_choices[rng.integers(len(rows_choices))] for _ in range(V)],
                              dtype=np.float64).reshape(V, vocab)
            toks = rng.integers(-1, vocab, size=V)
            res = oracle_accept(_bits(logits), np.array([0, V]), toks)
            # first-occurrence argmax by explicit scan
            am = []
            for row in logits:
                best = 0
                for v in range(vocab):
                    if row[v] > row[best]:
                        best = v
                am.append(best)
            a = _accept_brute(am, toks)
            assert list(res["row_argmax"]) == am
            assert res["accept_len"][0] == a
            assert res["next_token"][0] == (am[a] if a < V else -1)
            ents = [scipy.stats.entropy(np.exp(r - r.max()) / np.exp(r - r.max()).sum())
                    for r in logits]
            if V:
                np.testing.assert_allclose(res["accept_entropy"][0],
                                           np.mean(ents[:min(a, V - 1) + 1]), rtol=1e-13)
            else:
                assert res["accept_entropy"][0] == 0.0
            np.testing.assert_allclose(res["row_entropy"], ents, rtol=1e-13, atol=1e-15)
            cases += 1
    assert cases > 200


def test_accept_multi_request_ragged_and_empty():
    vocab = 7
    rng = np.random.default_rng(2)
    counts = [3, 0, 5, 1, 0]
    indptr = np.concatenate([[0], np.cumsum(counts)])
    logits = rng.normal(size=(indptr[-1], vocab))
    am = logits.argmax(1)
    toks = am.copy()
    toks[indptr[0] + 1] = (am[indptr[0] + 1] + 1) % vocab   # request 0 fails at row 1
    toks[indptr[3]] = -1                                      # request 3 is a bonus row only
    res = oracle_accept(_bits(logits), indptr, toks)
    bam = bf16_bits_to_f64(_bits(logits)).argmax(1)
    assert list(res["accept_len"]) == [1, 0, 5, 0, 0]
    assert list(res["next_token"]) == [bam[1], -1, -1, bam[indptr[3]], -1]
    assert res["accept_entropy"][1] == 0.0 and res["accept_entropy"][4] == 0.0


def test_sigma_zero_accepts_everything():
    lay = W.make_layout("tiny", seed=3, verify=("fixed", 6))
    inp = W.make_logit_inputs(lay, sigma=0.0)
    res = oracle_accept(W.bf16_bits(inp["verify_logits"]), lay.row_indptr,
                        inp["draft_tokens"].numpy())
    assert res["accept_len"][0] == 6 and res["next_token"][0] == -1


@pytest.mark.parametrize("k", [0, 2, 5])
def test_forced_mismatch_position(k):
    lay = W.make_layout("tiny", seed=4, verify=("fixed", 6))
    inp = W.make_logit_inputs(lay, sigma=0.0)
    toks = inp["draft_tokens"].numpy().copy()
    toks[k] = (toks[k] + 1) % lay.spec.vocab
    res = oracle_accept(W.bf16_bits(inp["verify_logits"]), lay.row_indptr, toks)
    assert res["accept_len"][0] == k
    assert res["next_token"][0] == inp["draft_tokens"].numpy()[k]


def test_bonus_row_gives_next_token_on_full_accept():
    lay = W.make_layout("tiny", seed=5, verify=("fixed", 3), bonus_rows=True)
    inp = W.make_logit_inputs(lay, sigma=0.0)
    toks = inp["draft_tokens"].numpy()
    assert toks[-1] == -1 and len(toks) == 4
    x = bf16_bits_to_f64(W.bf16_bits(inp["verify_logits"]))
    res = oracle_accept(W.bf16_bits(inp["verify_logits"]), lay.row_indptr, toks)
    assert res["accept_len"][0] == 3
    assert res["next_token"][0] == int(np.argmax(x[3]))


def test_confidence_all_equal_logits():
    vocab = 1000
    res = oracle_confidence(_bits(np.full((2, vocab), 0.75)))
    assert list(res["top1"]) == [0, 0] and list(res["top2"]) == [1, 1]
    np.testing.assert_allclose(res["p1"], 1.0 / vocab, rtol=1e-14)
    np.testing.assert_allclose(res["p2"], 1.0 / vocab, rtol=1e-14)
    assert (res["margin"] == 0).all()
    np.testing.assert_allclose(res["entropy"], math.log(vocab), rtol=1e-14)


@pytest.mark.parametrize("x", [0.5, 3.0, 12.0, 40.0])
def test_confidence_single_spike_closed_form(x):
    vocab, pos = 257, 100
    row = np.zeros(vocab)
    row[pos] = x
    res = oracle_confidence(_bits(row[None]))
    xb = float(bf16_bits_to_f64(_bits([x]))[0])
    z = math.exp(xb) + vocab - 1
    p1, p2 = math.exp(xb) / z, 1.0 / z
    # H = ln z - p1 * x, rewritten with delta = (vocab-1) e^-x to avoid cancellation
    delta = (vocab - 1) * math.exp(-xb)
    h = math.log1p(delta) + xb * delta / (1.0 + delta)
    assert res["top1"][0] == pos and res["top2"][0] == 0
    np.testing.assert_allclose([res["p1"][0], res["p2"][0], res["entropy"][0]], [p1, p2, h],
                               rtol=1e-12)
    np.testing.assert_allclose(res["margin"][0], p1 - p2, rtol=1e-12)


def test_confidence_against_library_routines():
    g = torch.Generator().manual_seed(0)
    logits = (torch.randn(16, 4096, generator=g) * 2.0).to(torch.bfloat16)
    logits[3, 17] = logits[3].max()          # tie at the top
    logits[5, :] = 0.0                        # all tied
    bits = logits.contiguous().view(torch.int16).numpy().view(np.uint16)
    res = oracle_confidence(bits)
    x = logits.double()
    ent = torch.distributions.Categorical(logits=x).entropy().numpy()
    np.testing.assert_allclose(res["entropy"], ent, rtol=1e-12)
    p = torch.softmax(x, dim=1).numpy()
    order = np.argsort(-x.numpy(), axis=1, kind="stable")
    np.testing.assert_array_equal(res["top1"], order[:, 0])
    np.testing.assert_array_equal(res["top2"], order[:, 1])
    rows = np.arange(16)
    np.testing.assert_allclose(res["p1"], p[rows, order[:, 0]], rtol=1e-12)
    np.testing.assert_allclose(res["p2"], p[rows, order[:, 1]], rtol=1e-12)
    assert res["p1"][3] == res["p2"][3] and res["margin"][3] == 0.0


def test_verify_entropy_two_way_closed_form():
    # logits (0, ln 3) -> p = (1/4, 3/4)
    row = np.array([[0.0, 1.0986328125]])  # ln 3 rounded to a bf16 value
    xb = bf16_bits_to_f64(_bits(row))[0]
    p = np.exp(xb) / np.exp(xb).sum()
    res = oracle_accept(_bits(row), np.array([0, 1]), np.array([1]))
    want = -(p[0] * math.log(p[0]) + p[1] * math.log(p[1]))
    assert abs(res["row_entropy"][0] - want) < 1e-15
    assert res["row_argmax"][0] == 1 and res["accept_len"][0] == 1
