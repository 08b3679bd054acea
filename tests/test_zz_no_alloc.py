"""The allocation-free logit round (rg_verify_and_confidence_noalloc) against
the same round with a caller workspace (rg_verify_and_confidence), through
the C ABI: two calls in a row, the second with a smaller batch, every output
bit for bit (same kernels; integer outputs exact, the statistics within the
oracle tolerance a fortiori)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_34388_amd import binding
from paper_2609_34388_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def _round(lay, inp, noalloc):
    rp = torch.as_tensor(lay.row_indptr, device=DEV)
    v, d = binding.verify_and_confidence(inp["verify_logits"], rp, inp["draft_tokens"], inp["draft_logits"],
                                         noalloc=noalloc)
    torch.cuda.synchronize()
    return v, d


@pytest.mark.parametrize("first,second", [(("mid", 3, None), ("high", 1, 5)), (("low", 0, None), ("tiny", 0, None))])
def test_noalloc_round_matches_workspace_round(first, second):
    for name, seed, nreq in (first, second):  # the second batch is smaller than the first
        lay = W.make_layout(name, seed=seed, num_requests=nreq) if nreq else W.make_layout(name, seed=seed)
        inp = W.make_logit_inputs(lay, DEV, ties=True)
        v0, d0 = _round(lay, inp, noalloc=False)
        v1, d1 = _round(lay, inp, noalloc=True)
        for k in v0:
            assert torch.equal(v0[k], v1[k]), (name, k)
        for k in d0:
            assert torch.equal(d0[k], d1[k]), (name, k)


def test_noalloc_round_refuses_batches_past_the_scratch():
    lib = binding.library()
    n = ctypes.c_size_t()
    assert lib.rg_verify_and_confidence_workspace(1, 16000, 16000, 128256, ctypes.byref(n)) == 0
    assert n.value > binding.NOALLOC_SCRATCH_BYTES
    D = ctypes.c_void_p(0x1000)  # never dereferenced: the size check comes first
    st = lib.rg_verify_and_confidence_noalloc(D, 128256, D, 128256, 128256, 1, 16000, D, D, D, D, D, None, None,
                                              16000, D, D, D, D, None, None, None)
    assert st == 3
