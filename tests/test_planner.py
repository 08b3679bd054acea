"""The attention planner's chunk rule and item accounting on the host (no
GPU): the shortest chunk (a multiple of 128 keys, at least 256, at most one
CU's share of all keys) whose work items fit in two rounds of 256, or, when
even the longest allowed chunk gives more, that chunk."""
import numpy as np
import pytest

from paper_2609_34388_amd import workloads as W
from tests.test_abi import _L, _plan

CUS, ROUND2 = 256, 512


def _items(lay, chunk, g, hkv):
    n = 0
    for r in range(lay.num_requests):
        q, T = int(lay.q_len[r]), int(lay.kv_len[r])
        if q == 0:
            continue
        n += -(-(q * g) // 256) * -(-T // chunk)
    return n * hkv


@pytest.mark.parametrize("spec,seed,nreq", [
    ("tiny", 0, None), ("low", 0, None), ("low", 1, 3),
    ("mid", 0, None), ("mid", 5, None), ("mid", 12, None), ("mid", 1, 4), ("mid", 2, 8), ("mid", 3, 32),
    ("high", 0, None), ("high", 1, 16), ("high", 2, 80),
    ("long", 0, None), ("long", 1, 8), ("long", 2, 24),
])
def test_chunk_is_shortest_fitting_two_rounds(spec, seed, nreq):
    lay = W.make_layout(spec, seed=seed, num_requests=nreq) if nreq else W.make_layout(spec, seed=seed)
    s = lay.spec
    g, hkv = s.num_q_heads // s.num_kv_heads, s.num_kv_heads
    l = _L(R=lay.num_requests, hq=s.num_q_heads, hkv=hkv, D=s.head_dim, num_pages=lay.num_pages,
           ctx=lay.ctx_len, nv=lay.n_verify, n=lay.q_len, pages=np.diff(lay.page_indptr))
    info = _plan(l)
    chunk = info.chunk_keys
    assert info.work_items == _items(lay, chunk, g, hkv)
    up = lambda x: -(-x // 128) * 128
    groups = [(int(lay.kv_len[r]), -(-int(lay.q_len[r]) * g // 256)) for r in range(lay.num_requests)
              if lay.q_len[r] > 0]
    total = sum(T * c for T, c in groups) * hkv
    whole = max(256, up(max(T for T, _ in groups)))
    hi = min(whole, max(256, up(total // CUS)))
    if _items(lay, hi, g, hkv) > ROUND2:
        assert chunk == hi
    elif _items(lay, 256, g, hkv) <= ROUND2:
        assert chunk == 256
    else:
        assert 256 < chunk <= hi and chunk % 128 == 0
        assert _items(lay, chunk, g, hkv) <= ROUND2 < _items(lay, chunk - 128, g, hkv)
