"""C-ABI checks that need no GPU: the library loads, exports every function
include/recguide.h declares, rejects bad arguments with the documented
status before touching the device, and plans ragged batches consistently."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "recguide.h")

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIB_PATH), reason="library not built")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rg_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_function():
    lib = binding.library()
    names = _declared_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(binding.EXPORTS)


def test_abi_version_and_status_strings():
    m = re.search(r"#define RG_ABI_VERSION (\d+)", open(HEADER).read())
    assert binding.abi_version() == int(m.group(1))
    lib = binding.library()
    for s in range(7):
        assert lib.rg_status_string(s)
    assert lib.rg_status_string(99) == b"unknown status"


FAKE_DEV = ctypes.c_void_p(0x1000)  # never dereferenced on the validation paths


class _L:
    def __init__(self, R=2, hq=8, hkv=2, D=128, page=16, num_pages=64, ctx=(40, 17), nv=(3, 0), n=(7, 5),
                 pages=None):
        self.q_indptr = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
        self.n_verify = np.asarray(nv, dtype=np.int32)
        self.ctx_len = np.asarray(ctx, dtype=np.int32)
        if pages is None:
            pages = [math.ceil((c + k) / 16) for c, k in zip(ctx, n)]
        self.page_indptr = np.concatenate([[0], np.cumsum(pages)]).astype(np.int32)
        self.c = binding.AttnLayout(R, hq, hkv, D, page, num_pages, 0.0, self.q_indptr.ctypes.data,
                                    self.n_verify.ctypes.data, self.ctx_len.ctypes.data,
                                    self.page_indptr.ctypes.data, FAKE_DEV.value)


def _attn(l, q=FAKE_DEV, k=FAKE_DEV, v=FAKE_DEV, out=FAKE_DEV):
    return binding.library().rg_draft_verify_attention(ctypes.byref(l.c), q, k, v, out, None, None, 0, None)


def test_attention_validation_errors():
    lib = binding.library()
    assert lib.rg_draft_verify_attention(None, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, None, None, 0, None) == 1
    assert _attn(_L(), q=None) == 1
    assert _attn(_L(), out=None) == 1
    l = _L(); l.c.num_requests = 0
    assert _attn(l) == 2
    l = _L(); l.c.num_q_heads = 6; l.c.num_kv_heads = 4
    assert _attn(l) == 2
    l = _L(); l.c.head_dim = 96
    assert _attn(l) == 3
    l = _L(); l.c.page_size = 32
    assert _attn(l) == 3
    assert _attn(_L(nv=(8, 0))) == 2                       # more verify rows than rows
    assert _attn(_L(ctx=(-1, 3))) == 2
    assert _attn(_L(pages=[2, 2])) == 2                    # too few pages for 47 keys
    l = _L(); l.page_indptr[0] = 1
    assert _attn(l) == 2
    l = _L(); l.c.page_indices = None
    assert _attn(l) == 1
    # misaligned pointers are rejected, not read
    assert _attn(_L(), q=ctypes.c_void_p(0x1002)) == 3


@pytest.mark.parametrize("nv", [32767, 32768, 40000, 65535])
def test_verify_counts_up_to_16_bits_are_planned(nv):
    """A request's row count and verify count share one packed plan word
    (16 bits each); every verify count up to 65535 is accepted and planned
    like any other layout (the kernel reads the field unsigned)."""
    l = _L(R=1, hq=1, hkv=1, D=64, ctx=(16,), nv=(nv,), n=(nv,), num_pages=(16 + nv) // 16 + 2)
    info = _plan(l)
    assert info.work_items >= 1
    assert _attn(l, out=None) == 1  # validation passes up to the pointer checks


def test_row_counts_past_16_bits_are_rejected():
    l = _L(R=1, hq=1, hkv=1, D=64, ctx=(0,), nv=(0,), n=(65536,), num_pages=4097)
    st = binding.library().rg_draft_verify_attention_workspace(ctypes.byref(l.c), ctypes.byref(ctypes.c_size_t()))
    assert st == 3
    assert _attn(l) == 3


def test_attention_check_validation():
    lib = binding.library()
    assert lib.rg_draft_verify_attention_check(None, 1 << 20, None) == 1
    assert lib.rg_draft_verify_attention_check(ctypes.c_void_p(0x1000), 15, None) == 4
    assert lib.rg_status_string(6) == b"a one-launch attention wait gave up"


def _br(indptr, prefix, lead, rows):
    return binding.make_branches(indptr, prefix, lead, rows)


def _mb_ws(l, b):
    n = ctypes.c_size_t(123)
    st = binding.library().rg_multibranch_attention_workspace(ctypes.byref(l.c), ctypes.byref(b.c), ctypes.byref(n))
    return st, n.value


def test_multibranch_validation_errors():
    lib = binding.library()
    # request 0: V = 3, 4 rows after them; request 1: V = 0, 5 rows
    l = _L(nv=(3, 0), n=(7, 5))
    ok = _br([0, 2, 3], [1, 3, 0], [1, 0, 0], [2, 2, 5])
    st, n = _mb_ws(l, ok)
    assert st == 0 and n == 0                                    # nothing is split here
    assert _mb_ws(l, _br([0, 0, 0], [], [], []))[0] == 0         # no branches: the fused step
    assert _mb_ws(l, _br([0, 2, 3], [1, 3, 0], [1, 0, 0], [2, 3, 5]))[0] == 2   # rows sum to 5, not 4
    assert _mb_ws(l, _br([0, 2, 3], [4, 3, 0], [1, 0, 0], [2, 2, 5]))[0] == 2   # prefix past V
    assert _mb_ws(l, _br([0, 2, 3], [1, 3, 0], [3, 0, 0], [2, 2, 5]))[0] == 2   # lead past rows
    assert _mb_ws(l, _br([0, 2, 3], [1, 3, 0], [1, 0, 0], [0, 4, 5]))[0] == 2   # empty branch
    assert _mb_ws(l, _br([1, 2, 3], [1, 3, 0], [1, 0, 0], [2, 2, 5]))[0] == 2   # branch_indptr[0] != 0
    family = _br([0, 4, 5], [0, 1, 2, 3, 0], [0, 0, 0, 0, 0], [1, 1, 1, 1, 5])
    assert _mb_ws(l, family)[0] == 0                             # a regular family packs into one word
    mixed = _br([0, 4, 5], [3, 0, 1, 3, 0], [0, 0, 0, 0, 0], [1, 1, 1, 1, 5])
    assert _mb_ws(l, mixed)[0] == 0                              # two single words, then a family of two
    four = _br([0, 4, 5], [3, 0, 2, 1, 0], [0, 0, 0, 0, 0], [1, 1, 1, 1, 5])
    assert _mb_ws(l, four)[0] == 3                               # three single branches before the last
    big = _L(R=1, nv=(4100,), n=(4101,), ctx=(0,))
    assert _mb_ws(big, _br([0, 1], [4100], [0], [1]))[0] == 3    # prefix past its 12-bit field
    assert lib.rg_multibranch_attention_workspace(ctypes.byref(l.c), None, ctypes.byref(ctypes.c_size_t())) == 1
    # the attention call itself validates the same way before anything runs
    assert lib.rg_multibranch_attention(ctypes.byref(l.c), ctypes.byref(four.c), FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                        FAKE_DEV, None, None, 0, None) == 3
    assert lib.rg_multibranch_attention(ctypes.byref(l.c), ctypes.byref(ok.c), None, FAKE_DEV, FAKE_DEV,
                                        FAKE_DEV, None, None, 0, None) == 1


def test_branch_plan_and_match_validation_errors():
    lib = binding.library()
    d = FAKE_DEV
    assert lib.rg_plan_branches(d, d, d, 0, 4, ctypes.c_float(0.5), d, d, d, d, d, None) == 2
    assert lib.rg_plan_branches(d, d, None, 2, 4, ctypes.c_float(0.5), d, d, d, d, d, None) == 1
    assert lib.rg_plan_branches(None, d, d, 2, 4, ctypes.c_float(0.5), d, d, d, d, d, None) == 1
    assert lib.rg_match_branches(d, d, d, d, d, d, d, d, 0, d, None) == 2
    assert lib.rg_match_branches(d, d, d, d, d, d, d, None, 2, d, None) == 1


def _policy(cand=(8, 16, 32), edges=(-1.0, -0.5), cost=(1.0, 2.0, 3.0), nb=None, ns=None):
    c = np.asarray(cand, dtype=np.int32)
    e = np.asarray(edges, dtype=np.float32)
    k = np.asarray(cost, dtype=np.float32)
    pol = binding.BlockPolicy(len(c) if nb is None else nb, c.ctypes.data, (len(e) + 1) if ns is None else ns,
                              e.ctypes.data if len(e) else None, k.ctypes.data, 1.0, FAKE_DEV)
    return pol, (c, e, k)


def test_block_size_validation_errors():
    lib = binding.library()
    d = FAKE_DEV
    args = lambda pol, R=4, order=d, offs=d: (ctypes.byref(pol), d, d, d, d, R, d, order, offs, None)
    assert lib.rg_plan_block_sizes(None, d, d, d, d, 4, d, d, d, None) == 1
    pol, keep = _policy(cand=(16, 8, 32))
    assert lib.rg_plan_block_sizes(*args(pol)) == 2          # unsorted candidates
    pol, keep = _policy(cand=(8, 8, 32))
    assert lib.rg_plan_block_sizes(*args(pol)) == 2          # repeated candidate
    pol, keep = _policy(cand=(0, 8, 32))
    assert lib.rg_plan_block_sizes(*args(pol)) == 2          # block size below 1
    pol, keep = _policy(edges=(-0.5, -1.0))
    assert lib.rg_plan_block_sizes(*args(pol)) == 2          # decreasing edges
    pol, keep = _policy(nb=9)
    assert lib.rg_plan_block_sizes(*args(pol)) == 3          # too many candidates
    pol, keep = _policy(ns=65)
    assert lib.rg_plan_block_sizes(*args(pol)) == 3          # too many bins
    pol, keep = _policy()
    assert lib.rg_plan_block_sizes(*args(pol, R=-1)) == 2
    assert lib.rg_plan_block_sizes(*args(pol, R=65537)) == 3
    assert lib.rg_plan_block_sizes(*args(pol, order=None)) == 1   # offsets without order
    assert lib.rg_plan_block_sizes(*args(pol, offs=None)) == 1    # order without offsets
    assert lib.rg_plan_block_sizes(ctypes.byref(pol), d, None, d, d, 4, d, d, d, None) == 1
    assert lib.rg_plan_block_sizes(*args(pol, R=0, order=None, offs=None)) == 0  # nothing to do


def test_logit_validation_errors():
    lib = binding.library()
    ws = ctypes.c_void_p(0x2000)
    n = ctypes.c_size_t()
    assert lib.rg_verify_accept_workspace(0, 4, 100, ctypes.byref(n)) == 2
    assert lib.rg_verify_accept_workspace(1, 4, 100, None) == 1
    assert lib.rg_verify_accept_workspace(2, 4, 20000, ctypes.byref(n)) == 0 and n.value > 0
    need = n.value
    args = [FAKE_DEV, 20000, 20000, 2, 4, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, None, None]
    assert lib.rg_verify_accept(*args, ws, need - 1, None) == 4
    assert lib.rg_verify_accept(*args[:1], 100, 20000, *args[3:], ws, need, None) == 2  # stride < vocab
    bad = list(args); bad[5] = None
    assert lib.rg_verify_accept(*bad, ws, need, None) == 1
    assert lib.rg_draft_confidence_workspace(4, 1, ctypes.byref(n)) == 2
    assert lib.rg_draft_confidence_workspace(4, 2, ctypes.byref(n)) == 0
    need = n.value
    dargs = [FAKE_DEV, 2, 2, 4, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, None, None]
    assert lib.rg_draft_confidence(*dargs, ws, need - 1, None) == 4
    dargs[4] = None
    assert lib.rg_draft_confidence(*dargs, ws, need, None) == 1


def _plan(l):
    info = binding.AttnPlanInfo()
    assert binding.library().rg_draft_verify_attention_plan(ctypes.byref(l.c), ctypes.byref(info)) == 0
    return info


@pytest.mark.parametrize("name", ["tiny", "low", "mid", "high", "long"])
def test_plan_accounting(name):
    lay = W.make_layout(name, seed=1)
    s = lay.spec
    l = _L(R=lay.num_requests, hq=s.num_q_heads, hkv=s.num_kv_heads, D=s.head_dim,
           num_pages=lay.num_pages, ctx=lay.ctx_len, nv=lay.n_verify, n=lay.q_len,
           pages=np.diff(lay.page_indptr))
    info = _plan(l)
    g = s.num_q_heads // s.num_kv_heads
    ch = info.chunk_keys
    assert ch % 128 == 0 and 128 <= ch <= 65536
    cpg = 256
    items = split = part = 0
    for r in range(lay.num_requests):
        T, M = int(lay.kv_len[r]), int(lay.q_len[r]) * g
        nch = -(-T // ch)
        items += s.num_kv_heads * (-(-M // cpg)) * nch
        if nch > 1:
            split += 1
            part += s.num_kv_heads * nch * (-(-M // 32) * 32)  # partials per 32-column tile
    assert info.work_items == items
    assert info.split_requests == split
    assert info.partial_columns == part
    assert info.num_launches == -(-lay.num_requests // 128)
    if part:
        assert info.workspace_bytes >= part // info.num_launches * s.head_dim * 2  # bf16 partial outputs
    else:
        assert info.workspace_bytes == 0


def test_plan_chunk_override_and_workspace_monotone(monkeypatch):
    lay = W.make_layout("mid", seed=2)
    s = lay.spec
    mk = lambda: _L(R=lay.num_requests, hq=s.num_q_heads, hkv=s.num_kv_heads, D=s.head_dim,
                    num_pages=lay.num_pages, ctx=lay.ctx_len, nv=lay.n_verify, n=lay.q_len,
                    pages=np.diff(lay.page_indptr))
    sizes = []
    for ch in (8192, 2048, 512, 128):  # multiples of the 128-key buffer
        monkeypatch.setenv("RG_ATTN_CHUNK", str(ch))
        info = _plan(mk())
        assert info.chunk_keys == ch
        sizes.append(info.workspace_bytes)
    assert sizes == sorted(sizes)


@pytest.mark.parametrize("persist", ["1", "0"])
@pytest.mark.parametrize("name", ["low", "mid", "high"])
def test_plan_one_launch_mode_and_sync_words(monkeypatch, persist, name):
    """Launches with a split request run as one work-queue launch when
    RG_ATTN_PERSIST=1 (the default is the main kernel plus the merge
    kernel); the synchronisation words (queue head, exit count, error word,
    then two counters per merge item) open the workspace at a fixed place
    and size, before the partials."""
    monkeypatch.setenv("RG_ATTN_PERSIST", persist)
    lay = W.make_layout(name, seed=1)
    s = lay.spec
    info = _plan(_L(R=lay.num_requests, hq=s.num_q_heads, hkv=s.num_kv_heads, D=s.head_dim,
                    num_pages=lay.num_pages, ctx=lay.ctx_len, nv=lay.n_verify, n=lay.q_len,
                    pages=np.diff(lay.page_indptr)))
    if info.split_requests == 0:
        assert info.persistent_launches == 0 and info.sync_offset == -1 and info.workspace_bytes == 0
        assert info.sync_words == 0
        return
    assert info.persistent_launches == (info.num_launches if persist == "1" else 0)
    g = s.num_q_heads // s.num_kv_heads
    tiles = sum(s.num_kv_heads * -(-int(lay.q_len[r]) * g // 32)
                for r in range(lay.num_requests) if -(-int(lay.kv_len[r]) // info.chunk_keys) > 1)
    merge_items = tiles * (4 * s.head_dim // (256 if persist == "1" else 128))
    # fixed place and size whatever the layout, room for every merge item's two counters
    assert info.sync_offset == 0 and info.sync_words == 4 + 2 * 16384 >= 4 + 2 * merge_items
    assert info.workspace_bytes >= (4 * info.sync_words + info.partial_columns * (s.head_dim * 2 + 8))


def test_generators_are_deterministic():
    a = W.make_layout("high", seed=5)
    b = W.make_layout("high", seed=5)
    for f in ("ctx_len", "n_verify", "n_draft", "page_indices", "q_indptr"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    c = W.make_layout("high", seed=6)
    assert not np.array_equal(a.ctx_len, c.ctx_len)
    small = W.make_layout("tiny", seed=3)
    x = W.make_attention_inputs(small)
    y = W.make_attention_inputs(small)
    for k in x:
        np.testing.assert_array_equal(W.bf16_bits(x[k]), W.bf16_bits(y[k]))
    lx = W.make_logit_inputs(small)
    ly = W.make_logit_inputs(small)
    for k in lx:
        assert np.array_equal(lx[k].view(-1).float().numpy(), ly[k].view(-1).float().numpy())


def test_generated_layout_respects_spec_ranges():
    lay = W.make_layout("long", seed=0)
    assert lay.num_requests == 64
    assert lay.ctx_len.min() >= 16384 and lay.ctx_len.max() <= 32768
    assert set(np.unique(lay.n_verify)) <= {4, 8, 16, 32}
    # every page referenced once, random order
    assert len(np.unique(lay.page_indices)) == len(lay.page_indices)
    assert lay.page_indices.max() < lay.num_pages
    pages = np.diff(lay.page_indptr)
    assert (pages * 16 >= lay.kv_len).all() and ((pages - 1) * 16 < lay.kv_len).all()


def test_fused_round_validation_errors():
    lib = binding.library()
    n = ctypes.c_size_t()
    assert lib.rg_verify_and_confidence_workspace(2, 4, 6, 1, ctypes.byref(n)) == 2  # vocab < 2
    assert lib.rg_verify_and_confidence_workspace(0, 4, 6, 100, ctypes.byref(n)) == 2
    assert lib.rg_verify_and_confidence_workspace(2, 4, 6, 20000, None) == 1
    assert lib.rg_verify_and_confidence_workspace(2, 4, 6, 20000, ctypes.byref(n)) == 0
    need = n.value
    sep = ctypes.c_size_t()
    lib.rg_verify_accept_workspace(2, 4, 20000, ctypes.byref(sep))
    assert need >= sep.value
    D = FAKE_DEV
    def call(ws, ws_bytes, vocab=20000, row_indptr=D, top1=D):
        return lib.rg_verify_and_confidence(D, vocab, D, vocab, vocab, 2, 4, row_indptr, D, D, D, D, None, None,
                                            6, top1, D, D, D, None, None, ws, ws_bytes, None)
    assert call(ctypes.c_void_p(0x10000), need - 1) == 4
    assert call(ctypes.c_void_p(0x10010), need) == 4  # not 256-byte aligned
    assert call(ctypes.c_void_p(0x10000), need, row_indptr=None) == 1
    assert call(ctypes.c_void_p(0x10000), need, top1=None) == 1
    assert call(ctypes.c_void_p(0x10000), need, vocab=1) == 2
