"""Python binding of the C ABI in ``include/zeta.h`` (argument marshalling only).

Each function carries the name of the C entry point it calls.  Tensors are
PyTorch tensors on a ROCm device; every step runs in the HIP kernels of
``libzeta.so`` on the current stream.  There is no fallback: if the library is
not built, the first call raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libzeta.so")
_lib = None

ZETA_OK, ZETA_ERR_INVALID_ARG, ZETA_ERR_UNSUPPORTED, ZETA_ERR_WORKSPACE, ZETA_ERR_HIP = range(5)
ZETA_F32, ZETA_BF16 = 0, 1
ZETA_ENCODE_STATIC_SCRATCH_BYTES = 1 << 20  # the allocation-free encode's per-GPU array (include/zeta.h)
# Attention scores (zeta_score_t): the method's Cauchy score and the variants.
SCORES = {"cauchy": 0, "dot": 1, "neg_euclid": 2, "inv_euclid": 3, "norm_dot": 4}
EXPORTED = (
    "zeta_morton_encode",
    "zeta_morton_encode_static",
    "zeta_sort_keys",
    "zeta_query_order",
    "zeta_select_topk",
    "zeta_topk_attn_fwd",
    "zeta_select_attend_fwd",
    "zeta_history_mean",
    "zeta_topk_attn_bwd",
    "zeta_select_attend_bwd",
    "zeta_exact_knn",
    "zeta_index_overlap",
    "zeta_workspace_size",
    "zeta_bwd_workspace_size",
    "zeta_select_attend_bwd_workspace_size",
    "zeta_status_string",
)


class ZetaError(RuntimeError):
    """A non-OK status returned by the library."""

    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {zeta_status_string(status)}")


def library_path() -> str:
    return _LIB_PATH


def load_library() -> ctypes.CDLL:
    """Load ``libzeta.so`` once and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run `python -m paper_2501_14577_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.zeta_morton_encode.argtypes = [vp, vp, i32, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp, sz, vp]
    L.zeta_morton_encode_static.argtypes = [vp, vp, i32, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp]
    L.zeta_sort_keys.argtypes = [vp, i64, i64, i32, vp, vp, vp, sz, vp]
    L.zeta_query_order.argtypes = [vp, i64, i64, i32, i32, i32, vp, vp, sz, vp]
    L.zeta_select_topk.argtypes = [vp, vp, vp, i64, i64, i32, i32, i32, vp, vp, vp, sz, vp]
    L.zeta_topk_attn_fwd.argtypes = [vp, vp, vp, i32, i64, i64, i64, i32, i32, i32, vp, vp, i32, f32, vp, vp, vp,
                                     vp]
    L.zeta_select_attend_fwd.argtypes = [vp, vp, vp, i32, i64, i64, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp,
                                         i32, f32, vp, vp, vp, vp, vp, sz, vp]
    L.zeta_history_mean.argtypes = [vp, vp, i32, i64, i64, i64, i32, i32, i32, vp, vp, vp, sz, vp]
    L.zeta_topk_attn_bwd.argtypes = [vp, vp, vp, i32, i64, i64, i64, i32, i32, i32, vp, vp, vp, f32, vp, vp, i32,
                                     vp, vp, vp, vp, vp, sz, vp]
    L.zeta_exact_knn.argtypes = [vp, vp, i32, i64, i64, i64, i32, i32, i32, vp, vp]
    L.zeta_index_overlap.argtypes = [vp, i32, vp, i32, i64, i64, vp, vp]
    L.zeta_workspace_size.argtypes = [i64, i64, i64, i32, i32, i32, i32]
    L.zeta_bwd_workspace_size.argtypes = [i64, i64, i64, i32, i32, i32, i32]
    L.zeta_select_attend_bwd.argtypes = [vp, vp, vp, i32, i64, i64, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp,
                                         vp, f32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.zeta_select_attend_bwd_workspace_size.argtypes = [i64, i64, i64, i32, i32, i32, i32]
    L.zeta_status_string.argtypes = [i32]
    for name in ("zeta_morton_encode", "zeta_morton_encode_static", "zeta_sort_keys", "zeta_query_order", "zeta_select_topk",
                 "zeta_topk_attn_fwd", "zeta_select_attend_fwd", "zeta_history_mean", "zeta_topk_attn_bwd",
                 "zeta_select_attend_bwd", "zeta_exact_knn", "zeta_index_overlap"):
        getattr(L, name).restype = ctypes.c_int
    L.zeta_workspace_size.restype = sz
    L.zeta_bwd_workspace_size.restype = sz
    L.zeta_select_attend_bwd_workspace_size.restype = sz
    L.zeta_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def zeta_status_string(status: int) -> str:
    return load_library().zeta_status_string(int(status)).decode()


def _check(fn: str, status: int) -> None:
    if status != ZETA_OK:
        raise ZetaError(fn, status)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return ZETA_F32
    if t.dtype == torch.bfloat16:
        return ZETA_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; expected float32 or bfloat16")


def _need_device(*ts: Optional[torch.Tensor]) -> None:
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("tensors must live on a ROCm GPU device")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def zeta_workspace_size(B: int, H: int, N: int, d_k: int, bits: int, topk: int, causal: bool) -> int:
    return int(load_library().zeta_workspace_size(B, H, N, d_k, bits, topk, int(bool(causal))))


def workspace_for(B, H, N, d_k, bits, topk, causal, device) -> torch.Tensor:
    n = max(zeta_workspace_size(B, H, N, d_k, bits, topk, causal), 256)
    return torch.empty(n, dtype=torch.uint8, device=device)


def zeta_bwd_workspace_size(B: int, H: int, N: int, d_k: int, d_v: int, topk: int, history_mean: bool) -> int:
    return int(load_library().zeta_bwd_workspace_size(B, H, N, d_k, d_v, topk, int(bool(history_mean))))


def bwd_workspace_for(B, H, N, d_k, d_v, topk, history_mean, device) -> torch.Tensor:
    n = max(zeta_bwd_workspace_size(B, H, N, d_k, d_v, topk, history_mean), 256)
    return torch.empty(n, dtype=torch.uint8, device=device)


def zeta_select_attend_bwd_workspace_size(B: int, H: int, N: int, d_v: int, topk: int, causal: bool,
                                          history_mean: bool = False) -> int:
    return int(load_library().zeta_select_attend_bwd_workspace_size(B, H, N, d_v, topk, int(bool(causal)),
                                                                      int(bool(history_mean))))


def select_attend_bwd_workspace_for(B, H, N, d_v, topk, causal, device, history_mean: bool = False) -> torch.Tensor:
    n = max(zeta_select_attend_bwd_workspace_size(B, H, N, d_v, topk, causal, history_mean), 256)
    return torch.empty(n, dtype=torch.uint8, device=device)


def zeta_morton_encode(q: torch.Tensor, k: torch.Tensor, bits: int, *,
                       range_lohi: Optional[torch.Tensor] = None,
                       range_out: Optional[torch.Tensor] = None,
                       q_codes: Optional[torch.Tensor] = None, k_codes: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Z-order codes of q and k ([B,H,N,d_k]) -> (q_codes, k_codes) uint32 [B,H,N]."""
    B, H, N, dk = q.shape
    if k.shape != q.shape or k.dtype != q.dtype:
        raise ValueError("q and k must share shape and dtype")
    if q_codes is None:
        q_codes = torch.empty((B, H, N), dtype=torch.uint32, device=q.device)
    if k_codes is None:
        k_codes = torch.empty((B, H, N), dtype=torch.uint32, device=q.device)
    if workspace is None and range_lohi is None:
        workspace = workspace_for(B, H, N, dk, bits, 1, False, q.device)
    _need_device(q, k, range_lohi, range_out, q_codes, k_codes, workspace)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().zeta_morton_encode(_ptr(q), _ptr(k), _dtype_code(q), B, H, N, dk, bits,
                                           _ptr(range_lohi), _ptr(range_out), _ptr(q_codes), _ptr(k_codes),
                                           _ptr(workspace), ws_bytes, _stream())
    _check("zeta_morton_encode", st)
    return q_codes, k_codes


def zeta_morton_encode_static(q: torch.Tensor, k: torch.Tensor, bits: int, *,
                              range_lohi: Optional[torch.Tensor] = None,
                              range_out: Optional[torch.Tensor] = None,
                              q_codes: Optional[torch.Tensor] = None,
                              k_codes: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """zeta_morton_encode without a workspace (the library's own per-GPU
    scratch holds the range partials; the C call allocates nothing)."""
    B, H, N, dk = q.shape
    if k.shape != q.shape or k.dtype != q.dtype:
        raise ValueError("q and k must share shape and dtype")
    if q_codes is None:
        q_codes = torch.empty((B, H, N), dtype=torch.uint32, device=q.device)
    if k_codes is None:
        k_codes = torch.empty((B, H, N), dtype=torch.uint32, device=q.device)
    _need_device(q, k, range_lohi, range_out, q_codes, k_codes)
    st = load_library().zeta_morton_encode_static(_ptr(q), _ptr(k), _dtype_code(q), B, H, N, dk, bits,
                                                  _ptr(range_lohi), _ptr(range_out), _ptr(q_codes), _ptr(k_codes),
                                                  _stream())
    _check("zeta_morton_encode_static", st)
    return q_codes, k_codes


def zeta_sort_keys(k_codes: torch.Tensor, code_bits: int, *, sorted_codes: Optional[torch.Tensor] = None,
                   perm: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Stable per-segment sort of uint32 codes [..., N] -> (sorted_codes, perm int32)."""
    N = k_codes.shape[-1]
    S = k_codes.numel() // N
    if sorted_codes is None:
        sorted_codes = torch.empty_like(k_codes)
    if perm is None:
        perm = torch.empty(k_codes.shape, dtype=torch.int32, device=k_codes.device)
    if workspace is None:
        workspace = workspace_for(S, 1, N, 1, code_bits, 1, False, k_codes.device)
    _need_device(k_codes, sorted_codes, perm, workspace)
    st = load_library().zeta_sort_keys(_ptr(k_codes), S, N, code_bits, _ptr(sorted_codes), _ptr(perm),
                                       _ptr(workspace), workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_sort_keys", st)
    return sorted_codes, perm


def zeta_query_order(q_order: Optional[torch.Tensor], N: int, S: int, topk: int, causal: bool, *,
                     chunk: int = 0, order_out: Optional[torch.Tensor] = None, device=None,
                     workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Regroup a processing order (int32 [..., N]; None: position order) by the
    list level each query searches (under the causal rule ``chunk``) -> int32
    order of the same shape."""
    dev = q_order.device if q_order is not None else device
    if order_out is None:
        shape = q_order.shape if q_order is not None else (S, N)
        order_out = torch.empty(shape, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = workspace_for(S, 1, N, 1, 1, topk, causal, dev)
    _need_device(q_order, order_out, workspace)
    st = load_library().zeta_query_order(_ptr(q_order), S, N, topk, int(bool(causal)), int(chunk), _ptr(order_out),
                                         _ptr(workspace), workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_query_order", st)
    return order_out


def _score_code(score) -> int:
    if isinstance(score, str):
        if score not in SCORES:
            raise ValueError(f"unknown score {score!r}; one of {sorted(SCORES)}")
        return SCORES[score]
    return int(score)


def zeta_select_topk(q_codes: torch.Tensor, sorted_codes: torch.Tensor, perm: torch.Tensor, topk: int,
                     causal: bool, *, chunk: int = 0, q_order: Optional[torch.Tensor] = None,
                     idx: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Candidate window of every query -> idx int32 [..., N, topk] (-1 padded).

    ``chunk`` > 0 selects the paper's chunked causal rule (pool: positions
    below floor(i / chunk) * chunk).  ``q_order`` (int32, shaped like
    ``q_codes``) is an optional processing order; it does not change the
    result."""
    N = q_codes.shape[-1]
    S = q_codes.numel() // N
    if idx is None:
        idx = torch.empty((*q_codes.shape, topk), dtype=torch.int32, device=q_codes.device)
    if workspace is None:
        workspace = workspace_for(S, 1, N, 1, 1, topk, causal, q_codes.device)
    _need_device(q_codes, sorted_codes, perm, q_order, idx, workspace)
    st = load_library().zeta_select_topk(_ptr(q_codes), _ptr(sorted_codes), _ptr(perm), S, N, topk,
                                         int(bool(causal)), int(chunk), _ptr(q_order), _ptr(idx), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_select_topk", st)
    return idx


def _means(mean_k, mean_v):
    if (mean_k is None) != (mean_v is None):
        raise ValueError("mean_k and mean_v are given together")
    for t in (mean_k, mean_v):
        if t is not None and t.dtype != torch.float32:
            raise ValueError("history means are float32")


def zeta_history_mean(k: torch.Tensor, v: torch.Tensor, causal: bool, *, mean_k: Optional[torch.Tensor] = None,
                      mean_v: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Mean key and mean value of each query's history -> (mean_k [B,H,N,d_k],
    mean_v [B,H,N,d_v]) float32: rows 0..i when causal, all rows otherwise."""
    B, H, N, dk = k.shape
    dv = v.shape[-1]
    f32 = dict(dtype=torch.float32, device=k.device)
    mean_k = torch.empty((B, H, N, dk), **f32) if mean_k is None else mean_k
    mean_v = torch.empty((B, H, N, dv), **f32) if mean_v is None else mean_v
    if workspace is None:
        workspace = workspace_for(B, H, N, dk, 1, 1, causal, k.device)
    _need_device(k, v, mean_k, mean_v, workspace)
    _means(mean_k, mean_v)
    if k.dtype != v.dtype:
        raise ValueError("k and v must share a dtype")
    st = load_library().zeta_history_mean(_ptr(k), _ptr(v), _dtype_code(k), B, H, N, dk, dv, int(bool(causal)),
                                          _ptr(mean_k), _ptr(mean_v), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_history_mean", st)
    return mean_k, mean_v


def zeta_topk_attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, idx: torch.Tensor, eps: float, *,
                       q_order: Optional[torch.Tensor] = None, score="cauchy",
                       mean_k: Optional[torch.Tensor] = None, mean_v: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Cauchy-softmax attention over idx (or a score variant, ``score`` a
    name of SCORES) -> out [B,H,N,d_v] in v's dtype; with mean_k and mean_v
    (``zeta_history_mean``) each window also holds the history-mean
    candidate."""
    B, H, N, dk = q.shape
    dv = v.shape[-1]
    topk = idx.shape[-1]
    if out is None:
        out = torch.empty((B, H, N, dv), dtype=v.dtype, device=v.device)
    _need_device(q, k, v, idx, q_order, mean_k, mean_v, out)
    _means(mean_k, mean_v)
    if not (q.dtype == k.dtype == v.dtype == out.dtype):
        raise ValueError("q, k, v and out must share a dtype")
    st = load_library().zeta_topk_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, H, N, dk, dv, topk,
                                           _ptr(idx), _ptr(q_order), _score_code(score), float(eps), _ptr(mean_k),
                                           _ptr(mean_v), _ptr(out), _stream())
    _check("zeta_topk_attn_fwd", st)
    return out


def zeta_topk_attn_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, idx: torch.Tensor, dout: torch.Tensor,
                       eps: float, *, q_order: Optional[torch.Tensor] = None, mean_k: Optional[torch.Tensor] = None,
                       mean_v: Optional[torch.Tensor] = None, causal: bool = True, dq: Optional[torch.Tensor] = None,
                       dk: Optional[torch.Tensor] = None, dv: Optional[torch.Tensor] = None,
                       deps: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """Gradients of the attention over idx -> (dq, dk, dv, deps), float32:
    dq, dk [B,H,N,d_k], dv [B,H,N,d_v], deps [1].  With mean_k and mean_v
    the history-mean candidate takes part, and ``causal`` says how its
    history was formed."""
    B, H, N, dkk = q.shape
    dvv = v.shape[-1]
    topk = idx.shape[-1]
    f32 = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty((B, H, N, dkk), **f32) if dq is None else dq
    dk = torch.empty((B, H, N, dkk), **f32) if dk is None else dk
    dv = torch.empty((B, H, N, dvv), **f32) if dv is None else dv
    deps = torch.empty((1,), **f32) if deps is None else deps
    if workspace is None:
        workspace = bwd_workspace_for(B, H, N, dkk, dvv, topk, mean_k is not None, q.device)
    _need_device(q, k, v, idx, dout, q_order, mean_k, mean_v, dq, dk, dv, deps, workspace)
    _means(mean_k, mean_v)
    if not (q.dtype == k.dtype == v.dtype == dout.dtype):
        raise ValueError("q, k, v and dout must share a dtype")
    if any(t.dtype != torch.float32 for t in (dq, dk, dv, deps)):
        raise ValueError("gradients are float32")
    st = load_library().zeta_topk_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, H, N, dkk, dvv, topk,
                                           _ptr(idx), _ptr(q_order), _ptr(dout), float(eps), _ptr(mean_k),
                                           _ptr(mean_v), int(bool(causal)), _ptr(dq), _ptr(dk),
                                           _ptr(dv), _ptr(deps), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_topk_attn_bwd", st)
    return dq, dk, dv, deps


def zeta_select_attend_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, q_codes: torch.Tensor,
                           sorted_codes: torch.Tensor, perm: torch.Tensor, topk: int, causal: bool, eps: float, *,
                           chunk: int = 0, score="cauchy",
                           q_order: Optional[torch.Tensor] = None, mean_k: Optional[torch.Tensor] = None,
                           mean_v: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                           idx_out: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Select and attend in one pass -> out [B,H,N,d_v]; ``idx_out`` (int32
    [B,H,N,topk]) optionally receives the windows."""
    B, H, N, dk = q.shape
    dv = v.shape[-1]
    if out is None:
        out = torch.empty((B, H, N, dv), dtype=v.dtype, device=v.device)
    if workspace is None:
        workspace = workspace_for(B, H, N, dk, 1, topk, causal, q.device)
    _need_device(q, k, v, q_codes, sorted_codes, perm, q_order, mean_k, mean_v, out, idx_out, workspace)
    _means(mean_k, mean_v)
    if not (q.dtype == k.dtype == v.dtype == out.dtype):
        raise ValueError("q, k, v and out must share a dtype")
    st = load_library().zeta_select_attend_fwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, H, N, dk, dv, topk,
                                               int(bool(causal)), int(chunk), _ptr(q_codes), _ptr(sorted_codes),
                                               _ptr(perm), _ptr(q_order), _score_code(score), float(eps),
                                               _ptr(mean_k), _ptr(mean_v), _ptr(out),
                                               _ptr(idx_out), _ptr(workspace),
                                               workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_select_attend_fwd", st)
    return out


def zeta_select_attend_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, q_codes: torch.Tensor,
                           sorted_codes: torch.Tensor, perm: torch.Tensor, topk: int, causal: bool, eps: float,
                           dout: torch.Tensor, *, chunk: int = 0, q_order: Optional[torch.Tensor] = None,
                           mean_k: Optional[torch.Tensor] = None, mean_v: Optional[torch.Tensor] = None,
                           dq: Optional[torch.Tensor] = None, dk: Optional[torch.Tensor] = None,
                           dv: Optional[torch.Tensor] = None, deps: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None):
    """Gradients of zeta_select_attend_fwd's attention (bfloat16, d_k = 3,
    Cauchy score) -> (dq, dk, dv, deps), float32: dq, dk [B,H,N,3],
    dv [B,H,N,d_v], deps [1].  With mean_k and mean_v the history-mean
    candidate takes part, and ``causal`` also says how its history was
    formed."""
    B, H, N, dkk = q.shape
    dvv = v.shape[-1]
    f32 = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty((B, H, N, dkk), **f32) if dq is None else dq
    dk = torch.empty((B, H, N, dkk), **f32) if dk is None else dk
    dv = torch.empty((B, H, N, dvv), **f32) if dv is None else dv
    deps = torch.empty((1,), **f32) if deps is None else deps
    if workspace is None:
        workspace = select_attend_bwd_workspace_for(B, H, N, dvv, topk, causal, q.device, mean_k is not None)
    _need_device(q, k, v, q_codes, sorted_codes, perm, q_order, dout, mean_k, mean_v, dq, dk, dv, deps, workspace)
    _means(mean_k, mean_v)
    if not (q.dtype == k.dtype == v.dtype == dout.dtype):
        raise ValueError("q, k, v and dout must share a dtype")
    if any(t.dtype != torch.float32 for t in (dq, dk, dv, deps)):
        raise ValueError("gradients are float32")
    st = load_library().zeta_select_attend_bwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, H, N, dkk, dvv, topk,
                                               int(bool(causal)), int(chunk), _ptr(q_codes), _ptr(sorted_codes),
                                               _ptr(perm), _ptr(q_order), _ptr(dout), float(eps), _ptr(mean_k),
                                               _ptr(mean_v), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(deps), _ptr(workspace),
                                               workspace.numel() * workspace.element_size(), _stream())
    _check("zeta_select_attend_bwd", st)
    return dq, dk, dv, deps


def zeta_exact_knn(q: torch.Tensor, k: torch.Tensor, kn: int, causal: bool, *,
                   knn_idx: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The kn keys nearest to each query in Euclidean distance within its
    pool, by (distance, position) -> int32 [B,H,N,kn] (-1 padded)."""
    B, H, N, dk = q.shape
    if knn_idx is None:
        knn_idx = torch.empty((B, H, N, kn), dtype=torch.int32, device=q.device)
    _need_device(q, k, knn_idx)
    if k.shape != q.shape or k.dtype != q.dtype:
        raise ValueError("q and k must share shape and dtype")
    st = load_library().zeta_exact_knn(_ptr(q), _ptr(k), _dtype_code(q), B, H, N, dk, kn, int(bool(causal)),
                                       _ptr(knn_idx), _stream())
    _check("zeta_exact_knn", st)
    return knn_idx


def zeta_index_overlap(idx_a: torch.Tensor, idx_b: torch.Tensor, N: int, *,
                       counts: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Per row, the number of positions rows of idx_a [..., ka] and idx_b
    [..., kb] share -> int32 [...]."""
    ka, kb = idx_a.shape[-1], idx_b.shape[-1]
    rows = idx_a.numel() // ka
    if idx_b.numel() // kb != rows:
        raise ValueError("idx_a and idx_b must have the same rows")
    if counts is None:
        counts = torch.empty(idx_a.shape[:-1], dtype=torch.int32, device=idx_a.device)
    _need_device(idx_a, idx_b, counts)
    st = load_library().zeta_index_overlap(_ptr(idx_a), ka, _ptr(idx_b), kb, rows, N, _ptr(counts), _stream())
    _check("zeta_index_overlap", st)
    return counts


def locality_counts(q: torch.Tensor, k: torch.Tensor, bits: int, kn: int = 64, causal: bool = False):
    """The counts behind Section 4.4's locality measure, all on the GPU:
    encode, sort and select each query's Z-order window of kn keys, the exact
    kn nearest keys (``zeta_exact_knn``) and, per query, how many keys the two
    share (``zeta_index_overlap``).  Returns (shared [B,H,N] int32, nearest
    [B,H,N,kn] int32, -1 padded); the measure is shared.sum() over the number
    of valid nearest entries."""
    B, H, N, dk = q.shape
    ws = workspace_for(B, H, N, dk, bits, kn, causal, q.device)
    qc, kc = zeta_morton_encode(q, k, bits, workspace=ws)
    sc, perm = zeta_sort_keys(kc, dk * bits, workspace=ws)
    win = zeta_select_topk(qc, sc, perm, kn, causal, workspace=ws)
    nn = zeta_exact_knn(q, k, kn, causal)
    return zeta_index_overlap(win, nn, N), nn


def forward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, topk: int, eps: float, causal: bool = True,
            bits: int = 10, *, workspace: Optional[torch.Tensor] = None, buffers: Optional[dict] = None,
            zorder: bool = True, fused: bool = False, history: bool = False, chunk: int = 0, score="cauchy",
            return_intermediates: bool = False):
    """The whole forward: encode, sort, select, attend (four calls, one stream).

    The query codes are sorted together with the key codes (one call over
    2*B*H segments); their Z-order, regrouped by list level, drives select
    and attend (``zorder``).  ``fused`` runs select and attend as one pass.
    The result is the same either way.  ``history`` adds the history-mean
    candidate to every window; ``chunk`` picks the paper's chunked causal
    rule and ``score`` a score variant.  ``buffers`` (from ``alloc_buffers``)
    holds preallocated outputs so that repeated calls allocate nothing.
    """
    B, H, N, dk = q.shape
    b = buffers if buffers is not None else alloc_buffers(B, H, N, v.shape[-1], topk, v.dtype, q.device)
    if workspace is None:
        workspace = workspace_for(B, H, N, dk, bits, topk, causal, q.device)
    qc, kc = zeta_morton_encode(q, k, bits, q_codes=b["codes"][0], k_codes=b["codes"][1], workspace=workspace)
    if zorder:
        sc2, perm2 = zeta_sort_keys(b["codes"], dk * bits, sorted_codes=b["sorted_codes2"], perm=b["perm2"],
                                    workspace=workspace)
        sc, perm = sc2[1], perm2[1]
        order = zeta_query_order(perm2[0], N, B * H, topk, causal, chunk=chunk, order_out=b["order"],
                                 workspace=workspace)
    else:
        sc, perm = zeta_sort_keys(kc, dk * bits, sorted_codes=b["sorted_codes2"][1], perm=b["perm2"][1],
                                  workspace=workspace)
        order = None
    mk = mv = None
    if history:
        mk, mv = zeta_history_mean(k, v, causal, workspace=workspace)
    if fused:
        idx = b["idx"] if return_intermediates else None
        out = zeta_select_attend_fwd(q, k, v, qc, sc, perm, topk, causal, eps, chunk=chunk, score=score, q_order=order,
                                     mean_k=mk, mean_v=mv, out=b["out"], idx_out=idx, workspace=workspace)
    else:
        idx = zeta_select_topk(qc, sc, perm, topk, causal, chunk=chunk, q_order=order, idx=b["idx"],
                               workspace=workspace)
        out = zeta_topk_attn_fwd(q, k, v, idx, eps, q_order=order, score=score, mean_k=mk, mean_v=mv, out=b["out"])
    if return_intermediates:
        return dict(q_codes=qc, k_codes=kc, sorted_codes=sc, perm=perm, q_order=order, idx=idx, mean_k=mk,
                    mean_v=mv, out=out)
    return out


def alloc_buffers(B: int, H: int, N: int, dv: int, topk: int, dtype: torch.dtype, device) -> dict:
    """Output buffers for ``forward(..., buffers=...)``.  Query and key codes
    share one [2, B, H, N] tensor so that one sort call orders both."""
    return dict(
        codes=torch.empty((2, B, H, N), dtype=torch.uint32, device=device),
        sorted_codes2=torch.empty((2, B, H, N), dtype=torch.uint32, device=device),
        perm2=torch.empty((2, B, H, N), dtype=torch.int32, device=device),
        order=torch.empty((B, H, N), dtype=torch.int32, device=device),
        idx=torch.empty((B, H, N, topk), dtype=torch.int32, device=device),
        out=torch.empty((B, H, N, dv), dtype=dtype, device=device),
    )
