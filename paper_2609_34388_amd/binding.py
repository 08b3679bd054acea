"""ctypes binding of librecguide.so (include/recguide.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  If the library is missing or cannot be loaded the first call
raises; there is no fallback.

Tensors are torch tensors on the GPU (bf16 as torch.bfloat16, indices as
torch.int32); per-request sizes for attention planning are host arrays
(numpy or CPU tensors).  Calls enqueue on the current torch stream unless a
``stream`` (torch.cuda.Stream or raw handle) is given and return without
synchronising.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Tuple

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librecguide.so")

RG_OK = 0
NOALLOC_SCRATCH_BYTES = 4 << 20  # RG_NOALLOC_SCRATCH_BYTES
_STATUS = {0: "ok", 1: "RG_ERR_NULL", 2: "RG_ERR_SHAPE", 3: "RG_ERR_UNSUPPORTED",
           4: "RG_ERR_WORKSPACE", 5: "RG_ERR_HIP", 6: "RG_ERR_WAIT"}


class RGError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_STATUS.get(status, status)} ({_lib().rg_status_string(status).decode()})")


class AttnLayout(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("sm_scale", ctypes.c_float),
                ("q_indptr", ctypes.c_void_p), ("n_verify", ctypes.c_void_p),
                ("ctx_len", ctypes.c_void_p), ("page_indptr", ctypes.c_void_p),
                ("page_indices", ctypes.c_void_p)]


class BranchLayout(ctypes.Structure):
    _fields_ = [("branch_indptr", ctypes.c_void_p), ("prefix", ctypes.c_void_p),
                ("lead", ctypes.c_void_p), ("rows", ctypes.c_void_p)]


class BlockPolicy(ctypes.Structure):
    _fields_ = [("num_candidates", ctypes.c_int32), ("candidates", ctypes.c_void_p),
                ("num_s_bins", ctypes.c_int32), ("s_edges", ctypes.c_void_p), ("cost", ctypes.c_void_p),
                ("rho", ctypes.c_float), ("value", ctypes.c_void_p)]


class AttnPlanInfo(ctypes.Structure):
    _fields_ = [("num_launches", ctypes.c_int32), ("chunk_keys", ctypes.c_int32),
                ("work_items", ctypes.c_int64), ("split_requests", ctypes.c_int64),
                ("partial_columns", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
                ("persistent_launches", ctypes.c_int32), ("sync_words", ctypes.c_int32),
                ("sync_offset", ctypes.c_int64)]


EXPORTS = ("rg_abi_version", "rg_status_string", "rg_draft_verify_attention_workspace",
           "rg_draft_verify_attention", "rg_draft_verify_attention_plan", "rg_draft_verify_attention_check",
           "rg_verify_accept_workspace", "rg_verify_accept", "rg_draft_confidence_workspace",
           "rg_draft_confidence", "rg_verify_and_confidence_workspace", "rg_verify_and_confidence",
           "rg_verify_and_confidence_noalloc",
           "rg_multibranch_attention_workspace", "rg_multibranch_attention", "rg_plan_branches",
           "rg_match_branches", "rg_plan_block_sizes")

_LIB = None


def _lib():
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built (run `python -m paper_2609_34388_amd.build_lib`)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "rg_abi_version": (I32, []),
        "rg_status_string": (ctypes.c_char_p, [I32]),
        "rg_draft_verify_attention_workspace": (I32, [ctypes.POINTER(AttnLayout), ctypes.POINTER(SZ)]),
        "rg_draft_verify_attention_plan": (I32, [ctypes.POINTER(AttnLayout), ctypes.POINTER(AttnPlanInfo)]),
        "rg_draft_verify_attention": (I32, [ctypes.POINTER(AttnLayout), P, P, P, P, P, P, SZ, P]),
        "rg_draft_verify_attention_check": (I32, [P, SZ, P]),
        "rg_verify_accept_workspace": (I32, [I32, I32, I32, ctypes.POINTER(SZ)]),
        "rg_verify_accept": (I32, [P, I64, I32, I32, I32, P, P, P, P, P, P, P, P, SZ, P]),
        "rg_draft_confidence_workspace": (I32, [I32, I32, ctypes.POINTER(SZ)]),
        "rg_draft_confidence": (I32, [P, I64, I32, I32, P, P, P, P, P, P, P, SZ, P]),
        "rg_verify_and_confidence_workspace": (I32, [I32, I32, I32, I32, ctypes.POINTER(SZ)]),
        "rg_verify_and_confidence": (I32, [P, I64, P, I64, I32, I32, I32, P, P, P, P, P, P, P,
                                           I32, P, P, P, P, P, P, P, SZ, P]),
        "rg_verify_and_confidence_noalloc": (I32, [P, I64, P, I64, I32, I32, I32, P, P, P, P, P, P, P,
                                                   I32, P, P, P, P, P, P, P]),
        "rg_multibranch_attention_workspace": (I32, [ctypes.POINTER(AttnLayout), ctypes.POINTER(BranchLayout),
                                                     ctypes.POINTER(SZ)]),
        "rg_multibranch_attention": (I32, [ctypes.POINTER(AttnLayout), ctypes.POINTER(BranchLayout),
                                           P, P, P, P, P, P, SZ, P]),
        "rg_plan_branches": (I32, [P, P, P, I32, I32, ctypes.c_float, P, P, P, P, P, P]),
        "rg_match_branches": (I32, [P, P, P, P, P, P, P, P, I32, P, P]),
        "rg_plan_block_sizes": (I32, [ctypes.POINTER(BlockPolicy), P, P, P, P, I32, P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def library() -> ctypes.CDLL:
    """The loaded library (raises if it is not built)."""
    return _lib()


def abi_version() -> int:
    return int(_lib().rg_abi_version())


# ---------------------------------------------------------------------------
def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _host_i32(x, name: str) -> np.ndarray:
    if isinstance(x, torch.Tensor):
        if x.is_cuda:
            raise TypeError(f"{name} must be a host array")
        x = x.numpy()
    a = np.ascontiguousarray(np.asarray(x), dtype=np.int32)
    return a


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(status: int, where: str):
    if status != RG_OK:
        raise RGError(status, where)


class _Layout:
    """Keeps the host arrays alive while the C struct points at them."""

    def __init__(self, num_q_heads, num_kv_heads, head_dim, num_pages, q_indptr, n_verify,
                 ctx_len, page_indptr, page_indices: torch.Tensor, sm_scale=0.0):
        self.q_indptr = _host_i32(q_indptr, "q_indptr")
        self.n_verify = _host_i32(n_verify, "n_verify")
        self.ctx_len = _host_i32(ctx_len, "ctx_len")
        self.page_indptr = _host_i32(page_indptr, "page_indptr")
        self.page_indices = _dev(page_indices, "page_indices", torch.int32)
        R = self.ctx_len.shape[0]
        if self.q_indptr.shape[0] != R + 1 or self.page_indptr.shape[0] != R + 1 or \
                self.n_verify.shape[0] != R:
            raise ValueError("per-request arrays disagree on the number of requests")
        self.c = AttnLayout(R, num_q_heads, num_kv_heads, head_dim, 16, num_pages, float(sm_scale),
                            self.q_indptr.ctypes.data, self.n_verify.ctypes.data,
                            self.ctx_len.ctypes.data, self.page_indptr.ctypes.data,
                            self.page_indices.data_ptr())


def make_layout(q: torch.Tensor, k_cache: torch.Tensor, q_indptr, n_verify, ctx_len, page_indptr,
                page_indices: torch.Tensor, sm_scale: float = 0.0) -> _Layout:
    total, hq, d = q.shape
    num_pages, hkv, page, d2 = k_cache.shape
    if page != 16 or d2 != d:
        raise ValueError("k_cache must be [pages, Hkv, 16, D] with the query's D")
    return _Layout(hq, hkv, d, num_pages, q_indptr, n_verify, ctx_len, page_indptr, page_indices,
                   sm_scale)


def attention_workspace_bytes(layout: _Layout) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib().rg_draft_verify_attention_workspace(ctypes.byref(layout.c), ctypes.byref(n)),
           "rg_draft_verify_attention_workspace")
    return int(n.value)


def attention_plan(layout: _Layout) -> Dict[str, int]:
    info = AttnPlanInfo()
    _check(_lib().rg_draft_verify_attention_plan(ctypes.byref(layout.c), ctypes.byref(info)),
           "rg_draft_verify_attention_plan")
    return {f: int(getattr(info, f)) for f, _ in AttnPlanInfo._fields_}


def draft_verify_attention(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                           q_indptr, n_verify, ctx_len, page_indptr, page_indices: torch.Tensor, *,
                           sm_scale: float = 0.0, out: Optional[torch.Tensor] = None,
                           lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                           workspace: Optional[torch.Tensor] = None, layout: Optional[_Layout] = None,
                           stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Fused draft-verify attention (rg_draft_verify_attention).

    q [sum n, Hq, D], k_cache [pages, Hkv, 16, D], v_cache [pages, Hkv, D, 16]
    (bf16); returns (out [sum n, Hq, D] bf16, lse [sum n, Hq] fp32 or None).
    """
    _dev(q, "q", torch.bfloat16)
    _dev(k_cache, "k_cache", torch.bfloat16)
    _dev(v_cache, "v_cache", torch.bfloat16)
    if v_cache.shape != (k_cache.shape[0], k_cache.shape[1], k_cache.shape[3], 16):
        raise ValueError("v_cache must be [pages, Hkv, D, 16]")
    lay = layout or make_layout(q, k_cache, q_indptr, n_verify, ctx_len, page_indptr, page_indices, sm_scale)
    if int(lay.q_indptr[-1]) != q.shape[0]:
        raise ValueError("q_indptr[-1] must equal the number of query rows")
    if lay.page_indices.numel() < int(lay.page_indptr[-1]):
        raise ValueError("page_indices is shorter than page_indptr[-1]")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", torch.bfloat16)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    if lse is not None:
        _dev(lse, "lse", torch.float32)
    need = attention_workspace_bytes(lay)
    if workspace is None and need:
        workspace = new_workspace(need, q.device)
    ws_ptr = _ptr(workspace) if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = _lib().rg_draft_verify_attention(ctypes.byref(lay.c), q.data_ptr(), k_cache.data_ptr(),
                                          v_cache.data_ptr(), out.data_ptr(), _ptr(lse), ws_ptr,
                                          ws_bytes, _stream(stream))
    _check(st, "rg_draft_verify_attention")
    return out, lse


def attention_check(workspace: torch.Tensor, stream=None) -> int:
    """rg_draft_verify_attention_check: synchronises the stream and returns
    the status (RG_OK, or 6 = RG_ERR_WAIT when a one-launch wait gave up)."""
    return int(_lib().rg_draft_verify_attention_check(workspace.data_ptr(), workspace.numel(), _stream(stream)))


class _Branches:
    """Host arrays of the overlap branches, kept alive with the C struct."""

    def __init__(self, branch_indptr, prefix, lead, rows):
        self.branch_indptr = _host_i32(branch_indptr, "branch_indptr")
        self.prefix = _host_i32(prefix, "prefix")
        self.lead = _host_i32(lead, "lead")
        self.rows = _host_i32(rows, "rows")
        nb = int(self.branch_indptr[-1]) if self.branch_indptr.size else 0
        for name in ("prefix", "lead", "rows"):
            if getattr(self, name).shape[0] < nb:
                raise ValueError(f"{name} is shorter than branch_indptr[-1]")
        self.c = BranchLayout(self.branch_indptr.ctypes.data, self.prefix.ctypes.data,
                              self.lead.ctypes.data, self.rows.ctypes.data)


def make_branches(branch_indptr, prefix, lead, rows) -> _Branches:
    return _Branches(branch_indptr, prefix, lead, rows)


def multibranch_workspace_bytes(layout: _Layout, branches: _Branches) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib().rg_multibranch_attention_workspace(ctypes.byref(layout.c), ctypes.byref(branches.c),
                                                     ctypes.byref(n)), "rg_multibranch_attention_workspace")
    return int(n.value)


def multibranch_attention(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, layout: _Layout,
                          branches: _Branches, *, out: Optional[torch.Tensor] = None,
                          lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                          workspace: Optional[torch.Tensor] = None,
                          stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Attention of a step with overlap branches (rg_multibranch_attention);
    tensors as in draft_verify_attention, the layout from make_layout and
    the branch lists from make_branches."""
    _dev(q, "q", torch.bfloat16)
    _dev(k_cache, "k_cache", torch.bfloat16)
    _dev(v_cache, "v_cache", torch.bfloat16)
    if v_cache.shape != (k_cache.shape[0], k_cache.shape[1], k_cache.shape[3], 16):
        raise ValueError("v_cache must be [pages, Hkv, D, 16]")
    if int(layout.q_indptr[-1]) != q.shape[0]:
        raise ValueError("q_indptr[-1] must equal the number of query rows")
    if branches.branch_indptr.shape[0] != layout.ctx_len.shape[0] + 1:
        raise ValueError("branch_indptr must have num_requests + 1 entries")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", torch.bfloat16)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    if lse is not None:
        _dev(lse, "lse", torch.float32)
    need = multibranch_workspace_bytes(layout, branches)
    if workspace is None and need:
        workspace = new_workspace(need, q.device)
    ws_ptr = _ptr(workspace) if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = _lib().rg_multibranch_attention(ctypes.byref(layout.c), ctypes.byref(branches.c), q.data_ptr(),
                                         k_cache.data_ptr(), v_cache.data_ptr(), out.data_ptr(), _ptr(lse),
                                         ws_ptr, ws_bytes, _stream(stream))
    _check(st, "rg_multibranch_attention")
    return out, lse


def plan_branches(margin: torch.Tensor, top2: torch.Tensor, row_indptr: torch.Tensor, delta: float, *,
                  out: Optional[Dict[str, torch.Tensor]] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Risky positions and branches of each request's draft block
    (rg_plan_branches); margin fp32 / top2 int32 per draft row, row_indptr
    int32 [R+1] on the device."""
    _dev(margin, "margin", torch.float32)
    _dev(top2, "top2", torch.int32)
    _dev(row_indptr, "row_indptr", torch.int32)
    R = row_indptr.numel() - 1
    dev = margin.device
    if out is None:
        out = dict(n_risky=torch.empty(R, dtype=torch.int32, device=dev),
                   n_corr=torch.empty(R, dtype=torch.int32, device=dev),
                   corr_pos=torch.empty(R, 2, dtype=torch.int32, device=dev),
                   corr_tok=torch.empty(R, 2, dtype=torch.int32, device=dev),
                   continuation=torch.empty(R, dtype=torch.int32, device=dev))
    st = _lib().rg_plan_branches(_ptr(margin), _ptr(top2), row_indptr.data_ptr(), R, margin.numel(),
                                 ctypes.c_float(delta), out["n_risky"].data_ptr(), out["n_corr"].data_ptr(),
                                 out["corr_pos"].data_ptr(), out["corr_tok"].data_ptr(),
                                 out["continuation"].data_ptr(), _stream(stream))
    _check(st, "rg_plan_branches")
    return out


def match_branches(accept_len: torch.Tensor, next_token: torch.Tensor, block_len: torch.Tensor,
                   plan: Dict[str, torch.Tensor], cont_first: torch.Tensor, *,
                   out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Index of the branch each request's verification confirms, or -1
    (rg_match_branches); all int32 device tensors, `plan` from plan_branches."""
    for name, t in (("accept_len", accept_len), ("next_token", next_token), ("block_len", block_len),
                    ("cont_first", cont_first)):
        _dev(t, name, torch.int32)
    R = accept_len.numel()
    if out is None:
        out = torch.empty(R, dtype=torch.int32, device=accept_len.device)
    st = _lib().rg_match_branches(accept_len.data_ptr(), next_token.data_ptr(), block_len.data_ptr(),
                                  plan["n_corr"].data_ptr(), plan["corr_pos"].data_ptr(),
                                  plan["corr_tok"].data_ptr(), plan["continuation"].data_ptr(),
                                  cont_first.data_ptr(), R, out.data_ptr(), _stream(stream))
    _check(st, "rg_match_branches")
    return out


class _BlockPolicy:
    """An rg_block_policy with its host arrays kept alive."""

    def __init__(self, candidates, s_edges, cost, rho: float, value: torch.Tensor):
        self.candidates = np.ascontiguousarray(np.asarray(candidates), dtype=np.int32)
        self.s_edges = np.ascontiguousarray(np.asarray(s_edges, dtype=np.float32).reshape(-1))
        self.cost = np.ascontiguousarray(np.asarray(cost, dtype=np.float32).reshape(-1))
        _dev(value, "value", torch.float32)
        nb, ns = self.candidates.shape[0], self.s_edges.shape[0] + 1
        if tuple(value.shape) != (nb, ns, nb, 2):
            raise ValueError(f"value must be [{nb}, {ns}, {nb}, 2], got {tuple(value.shape)}")
        if self.cost.shape[0] != nb:
            raise ValueError("cost needs one entry per candidate")
        self.value = value
        self.c = BlockPolicy(nb, self.candidates.ctypes.data, ns,
                             self.s_edges.ctypes.data if ns > 1 else None, self.cost.ctypes.data,
                             float(rho), value.data_ptr())


def make_block_policy(candidates, s_edges, cost, rho: float, value: torch.Tensor) -> _BlockPolicy:
    """Policy of Eq. 3 at one load: candidate block sizes, s-bin edges, cost
    T_C(B) per candidate (host), rho_C, and the V_B table on the device as an
    fp32 tensor [NB, NS, NB, 2]."""
    return _BlockPolicy(candidates, s_edges, cost, rho, value)


def plan_block_sizes(policy: _BlockPolicy, accept_len: torch.Tensor, accept_entropy: torch.Tensor,
                     prev_block: torch.Tensor, entropy_hist: torch.Tensor, *, bucket: bool = True,
                     out: Optional[Dict[str, torch.Tensor]] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Next block size per request and the grouping by size
    (rg_plan_block_sizes); entropy_hist is updated in place."""
    _dev(accept_len, "accept_len", torch.int32)
    _dev(accept_entropy, "accept_entropy", torch.float32)
    _dev(prev_block, "prev_block", torch.int32)
    _dev(entropy_hist, "entropy_hist", torch.float32)
    R = accept_len.numel()
    for name, t in (("accept_entropy", accept_entropy), ("prev_block", prev_block), ("entropy_hist", entropy_hist)):
        if t.numel() != R:
            raise ValueError(f"{name} must have {R} entries")
    dev = accept_len.device
    nb = policy.candidates.shape[0]
    if out is None:
        out = dict(next_block=torch.empty(R, dtype=torch.int32, device=dev))
        if bucket:
            out["order"] = torch.empty(R, dtype=torch.int32, device=dev)
            out["bucket_offsets"] = torch.empty(nb + 1, dtype=torch.int32, device=dev)
    st = _lib().rg_plan_block_sizes(ctypes.byref(policy.c), _ptr(accept_len), _ptr(accept_entropy),
                                    _ptr(prev_block), _ptr(entropy_hist), R, _ptr(out["next_block"]),
                                    _ptr(out.get("order")), _ptr(out.get("bucket_offsets")), _stream(stream))
    _check(st, "rg_plan_block_sizes")
    return out


def verify_accept_workspace_bytes(num_requests: int, total_rows: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib().rg_verify_accept_workspace(num_requests, total_rows, vocab, ctypes.byref(n)),
           "rg_verify_accept_workspace")
    return int(n.value)


def draft_confidence_workspace_bytes(total_rows: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib().rg_draft_confidence_workspace(total_rows, vocab, ctypes.byref(n)),
           "rg_draft_confidence_workspace")
    return int(n.value)


def new_workspace(nbytes: int, device) -> torch.Tensor:
    """A zeroed workspace of at least `nbytes` bytes.  Attention workspaces must be
    zero before their first use (each call leaves them ready for the next); the
    others need no initialisation."""
    return torch.zeros(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def verify_accept(logits: torch.Tensor, row_indptr: torch.Tensor, draft_tokens: torch.Tensor, *,
                  workspace: Optional[torch.Tensor] = None, out: Optional[Dict[str, torch.Tensor]] = None,
                  want_entropy: bool = True, stream=None) -> Dict[str, torch.Tensor]:
    """Greedy verification (rg_verify_accept).  logits [rows, vocab] bf16
    (row stride may exceed vocab), row_indptr [R+1] int32, draft_tokens
    [rows] int32 -- all on the GPU."""
    if not logits.is_cuda or logits.dtype != torch.bfloat16 or logits.dim() != 2 or logits.stride(1) != 1:
        raise TypeError("logits must be a CUDA bf16 [rows, vocab] tensor with unit column stride")
    _dev(row_indptr, "row_indptr", torch.int32)
    rows, vocab = logits.shape
    R = row_indptr.shape[0] - 1
    if rows:
        _dev(draft_tokens, "draft_tokens", torch.int32)
    dev = logits.device
    o = dict(out or {})
    o.setdefault("row_argmax", torch.empty(rows, dtype=torch.int32, device=dev))
    o.setdefault("accept_len", torch.empty(R, dtype=torch.int32, device=dev))
    o.setdefault("next_token", torch.empty(R, dtype=torch.int32, device=dev))
    if want_entropy:
        o.setdefault("row_entropy", torch.empty(rows, dtype=torch.float32, device=dev))
        o.setdefault("accept_entropy", torch.empty(R, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = new_workspace(verify_accept_workspace_bytes(R, rows, vocab), dev)
    st = _lib().rg_verify_accept(
        logits.data_ptr() if rows else None, logits.stride(0) if rows else vocab, vocab, R, rows,
        row_indptr.data_ptr(), draft_tokens.data_ptr() if rows else None,
        o["row_argmax"].data_ptr() if rows else None, o["accept_len"].data_ptr(),
        o["next_token"].data_ptr(), _ptr(o.get("row_entropy")) if rows else None,
        _ptr(o.get("accept_entropy")), workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check(st, "rg_verify_accept")
    return o


def draft_confidence(logits: torch.Tensor, *, workspace: Optional[torch.Tensor] = None,
                     out: Optional[Dict[str, torch.Tensor]] = None, want_margin: bool = True,
                     want_entropy: bool = True, stream=None) -> Dict[str, torch.Tensor]:
    """Draft confidence (rg_draft_confidence) of logits [rows, vocab] bf16."""
    if not logits.is_cuda or logits.dtype != torch.bfloat16 or logits.dim() != 2 or logits.stride(1) != 1:
        raise TypeError("logits must be a CUDA bf16 [rows, vocab] tensor with unit column stride")
    rows, vocab = logits.shape
    dev = logits.device
    o = dict(out or {})
    for k, dt in (("top1", torch.int32), ("top2", torch.int32), ("p1", torch.float32), ("p2", torch.float32)):
        o.setdefault(k, torch.empty(rows, dtype=dt, device=dev))
    if want_margin:
        o.setdefault("margin", torch.empty(rows, dtype=torch.float32, device=dev))
    if want_entropy:
        o.setdefault("entropy", torch.empty(rows, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = new_workspace(draft_confidence_workspace_bytes(rows, vocab), dev)
    st = _lib().rg_draft_confidence(
        logits.data_ptr() if rows else None, logits.stride(0) if rows else vocab, vocab, rows,
        _ptr(o["top1"]), _ptr(o["top2"]), _ptr(o["p1"]), _ptr(o["p2"]), _ptr(o.get("margin")),
        _ptr(o.get("entropy")), workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check(st, "rg_draft_confidence")
    return o


def verify_and_confidence_workspace_bytes(num_requests: int, verify_rows: int, draft_rows: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib().rg_verify_and_confidence_workspace(num_requests, verify_rows, draft_rows, vocab, ctypes.byref(n)),
           "rg_verify_and_confidence_workspace")
    return int(n.value)


def verify_and_confidence(verify_logits: torch.Tensor, row_indptr: torch.Tensor, draft_tokens: torch.Tensor,
                          draft_logits: torch.Tensor, *, workspace: Optional[torch.Tensor] = None,
                          out_verify: Optional[Dict[str, torch.Tensor]] = None,
                          out_draft: Optional[Dict[str, torch.Tensor]] = None, noalloc: bool = False,
                          stream=None) -> Tuple[Dict[str, torch.Tensor], Dict[str, torch.Tensor]]:
    """Both logit passes of a round in one call (rg_verify_and_confidence):
    returns the outputs of verify_accept and of draft_confidence.  With
    ``noalloc`` the allocation-free variant runs instead
    (rg_verify_and_confidence_noalloc: the library's static scratch, no
    workspace; ``workspace`` is ignored)."""
    for t, name in ((verify_logits, "verify_logits"), (draft_logits, "draft_logits")):
        if not t.is_cuda or t.dtype != torch.bfloat16 or t.dim() != 2 or t.stride(1) != 1:
            raise TypeError(f"{name} must be a CUDA bf16 [rows, vocab] tensor with unit column stride")
    if verify_logits.shape[1] != draft_logits.shape[1]:
        raise ValueError("verify and draft logits must have the same vocabulary")
    _dev(row_indptr, "row_indptr", torch.int32)
    vrows, vocab = verify_logits.shape
    drows = draft_logits.shape[0]
    R = row_indptr.shape[0] - 1
    if vrows:
        _dev(draft_tokens, "draft_tokens", torch.int32)
    dev = verify_logits.device
    ov = dict(out_verify or {})
    ov.setdefault("row_argmax", torch.empty(vrows, dtype=torch.int32, device=dev))
    ov.setdefault("accept_len", torch.empty(R, dtype=torch.int32, device=dev))
    ov.setdefault("next_token", torch.empty(R, dtype=torch.int32, device=dev))
    ov.setdefault("row_entropy", torch.empty(vrows, dtype=torch.float32, device=dev))
    ov.setdefault("accept_entropy", torch.empty(R, dtype=torch.float32, device=dev))
    od = dict(out_draft or {})
    for k, dt in (("top1", torch.int32), ("top2", torch.int32), ("p1", torch.float32), ("p2", torch.float32),
                  ("margin", torch.float32), ("entropy", torch.float32)):
        od.setdefault(k, torch.empty(drows, dtype=dt, device=dev))
    args = (verify_logits.data_ptr() if vrows else None, verify_logits.stride(0) if vrows else vocab,
            draft_logits.data_ptr() if drows else None, draft_logits.stride(0) if drows else vocab, vocab, R, vrows,
            row_indptr.data_ptr(), draft_tokens.data_ptr() if vrows else None,
            ov["row_argmax"].data_ptr() if vrows else None, ov["accept_len"].data_ptr(), ov["next_token"].data_ptr(),
            _ptr(ov.get("row_entropy")) if vrows else None, _ptr(ov.get("accept_entropy")), drows,
            _ptr(od["top1"]) if drows else None, _ptr(od["top2"]) if drows else None,
            _ptr(od["p1"]) if drows else None, _ptr(od["p2"]) if drows else None,
            _ptr(od.get("margin")) if drows else None, _ptr(od.get("entropy")) if drows else None)
    if noalloc:
        _check(_lib().rg_verify_and_confidence_noalloc(*args, _stream(stream)), "rg_verify_and_confidence_noalloc")
        return ov, od
    if workspace is None:
        workspace = new_workspace(verify_and_confidence_workspace_bytes(R, vrows, drows, vocab), dev)
    st = _lib().rg_verify_and_confidence(*args, workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check(st, "rg_verify_and_confidence")
    return ov, od

