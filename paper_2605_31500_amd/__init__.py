"""Fused graph-transformer attention over a CSR graph for AMD MI355X (gfx950).

Python binding of the C ABI declared in ``include/gt_attn.h``.  Every function
here only marshals arguments (torch tensors -> device pointers, sizes and the
current HIP stream) and calls ``libgtattn.so``; all arithmetic runs in the HIP
kernels.  PyTorch provides device memory and streams.  There is no fallback:
if the library is missing or the call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgtattn.so")

GT_SUCCESS = 0
GT_ERROR_INVALID_VALUE = 1
GT_ERROR_NOT_SUPPORTED = 2
GT_ERROR_OUT_OF_MEMORY = 3
GT_ERROR_HIP = 4
GT_DTYPE_F32 = 0
GT_DTYPE_BF16 = 1

EXPORTED_SYMBOLS = (
    "gt_attn_fwd", "gt_attn_fwd_bf16", "gt_attn_fwd_ex", "gt_attn_fwd_noalloc", "gt_gatv2_fwd", "gt_attn_bwd",
    "gt_segment_reduce", "gt_dot_aggr", "gt_csr_validate", "gt_status_string",
    "gt_last_error_message", "gt_profile_enable", "gt_profile_collect", "gt_workspace_release",
    "gt_workspace_pool_stats",
)


class GtTuning(ctypes.Structure):
    _fields_ = [("light_max_deg", ctypes.c_int32), ("heavy_min_deg", ctypes.c_int32),
                ("chunk_edges", ctypes.c_int32), ("grid_blocks", ctypes.c_int32),
                ("dense_tiles", ctypes.c_int32), ("bf16_weights", ctypes.c_int32)]


class GtError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("gt_attn status %d: %s" % (status, message))
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libgtattn.so (torch is imported first so the library binds to the
    HIP runtime torch already loaded, making torch streams valid for it)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libgtattn.so is not built; run __graft_entry__.build() or "
                           "python -m paper_2605_31500_amd._build")
    L = ctypes.CDLL(path)
    P, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    sig = [P, P, P, P, P, P, i64, i64, i32, i32, f32, P]
    L.gt_attn_fwd.argtypes = sig
    L.gt_attn_fwd_bf16.argtypes = sig
    L.gt_attn_fwd_ex.argtypes = [ctypes.c_int] + sig[:6] + [P] + sig[6:-1] + [ctypes.POINTER(GtTuning), P]
    L.gt_attn_fwd_noalloc.argtypes = L.gt_attn_fwd_ex.argtypes
    L.gt_gatv2_fwd.argtypes = [ctypes.c_int, P, P, P, P, P, f32, P, P, i64, i64, i32, i32,
                               ctypes.POINTER(GtTuning), P]
    L.gt_segment_reduce.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P, P, i64, i64, i32,
                                    ctypes.POINTER(GtTuning), P]
    L.gt_dot_aggr.argtypes = [P, P, P, P, i64, i64, i32, i32, i32, P]
    L.gt_attn_bwd.argtypes = [ctypes.c_int, P, P, P, P, P, P, P, P, P, P, P, P, P, i64, i64, i32, i32,
                              f32, P]
    L.gt_csr_validate.argtypes = [P, P, i64, i64, ctypes.POINTER(i32), P]
    L.gt_status_string.argtypes = [ctypes.c_int]
    L.gt_status_string.restype = ctypes.c_char_p
    L.gt_last_error_message.argtypes = []
    L.gt_last_error_message.restype = ctypes.c_char_p
    L.gt_profile_enable.argtypes = [i32]
    L.gt_profile_collect.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]
    L.gt_workspace_release.argtypes = []
    L.gt_workspace_pool_stats.argtypes = [i32, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
    for name in ("gt_attn_fwd", "gt_attn_fwd_bf16", "gt_attn_fwd_ex", "gt_attn_fwd_noalloc", "gt_gatv2_fwd",
                 "gt_attn_bwd",
                 "gt_segment_reduce", "gt_dot_aggr", "gt_csr_validate",
                 "gt_profile_enable", "gt_profile_collect", "gt_workspace_release",
                 "gt_workspace_pool_stats"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int) -> None:
    if status != GT_SUCCESS:
        L = load_library()
        raise GtError(status, "%s: %s" % (L.gt_status_string(status).decode(),
                                         L.gt_last_error_message().decode()))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device, stream):
    """The HIP stream to launch on; the library launches on the current device,
    so the tensors must live there."""
    if device.index is not None and device.index != torch.cuda.current_device():
        raise ValueError("tensors are on %s but the current device is cuda:%d; call under "
                         "torch.cuda.device(%s)" % (device, torch.cuda.current_device(), device))
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check_tensors(rowptr, colidx, Q, K, V, out, dtypes):
    for name, t in (("rowptr", rowptr), ("colidx", colidx), ("Q", Q), ("K", K), ("V", V),
                    ("out", out)):
        if not isinstance(t, torch.Tensor):
            raise TypeError(name + " must be a torch.Tensor")
        if not t.is_cuda:
            raise ValueError(name + " must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(name + " must be contiguous")
    if any(t.device != Q.device for t in (rowptr, colidx, K, V, out)):
        raise ValueError("all tensors must be on one device")
    if rowptr.dtype != torch.int64 or colidx.dtype != torch.int32:
        raise TypeError("rowptr must be int64 and colidx int32")
    if Q.dim() != 3 or K.shape != Q.shape or V.shape != Q.shape or out.shape != Q.shape:
        raise ValueError("Q, K, V, out must share one [N, H, D] shape")
    for t in (Q, K, V, out):
        if t.dtype not in dtypes:
            raise TypeError("feature dtype %s not in %s" % (t.dtype, dtypes))
    if rowptr.numel() != Q.shape[0] + 1:
        raise ValueError("rowptr must have N+1 entries")


def gt_attn_fwd(rowptr, colidx, Q, K, V, out, scale, stream=None) -> None:
    """fp32 features; writes out.  See include/gt_attn.h."""
    _check_tensors(rowptr, colidx, Q, K, V, out, (torch.float32,))
    N, H, D = Q.shape
    _check(load_library().gt_attn_fwd(_ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K), _ptr(V),
                                      _ptr(out), N, colidx.numel(), H, D, float(scale),
                                      _stream(Q.device, stream)))


def gt_attn_fwd_bf16(rowptr, colidx, Q, K, V, out, scale, stream=None) -> None:
    """bf16 features (torch.bfloat16, or int16/uint16 holding bf16 bits); writes out."""
    _check_tensors(rowptr, colidx, Q, K, V, out, (torch.bfloat16, torch.int16, torch.uint16))
    N, H, D = Q.shape
    _check(load_library().gt_attn_fwd_bf16(_ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K), _ptr(V),
                                           _ptr(out), N, colidx.numel(), H, D, float(scale),
                                           _stream(Q.device, stream)))


def gt_attn_fwd_ex(rowptr, colidx, Q, K, V, out, scale, tuning=None, stream=None, lse=None) -> None:
    """Either dtype (taken from Q); tuning: dict or GtTuning of partition overrides;
    lse: optional float32 [N, H] device tensor receiving ln(sum_e exp(s_e)) per row."""
    if Q.dtype == torch.float32:
        dtype, allowed = GT_DTYPE_F32, (torch.float32,)
    else:
        dtype, allowed = GT_DTYPE_BF16, (torch.bfloat16, torch.int16, torch.uint16)
    _check_tensors(rowptr, colidx, Q, K, V, out, allowed)
    N, H, D = Q.shape
    if isinstance(tuning, dict):
        tuning = GtTuning(**tuning)
    tp = ctypes.byref(tuning) if tuning is not None else None
    if lse is not None:
        if not (lse.is_cuda and lse.device == out.device and lse.is_contiguous()
                and lse.dtype == torch.float32 and tuple(lse.shape) == (N, H)):
            raise ValueError("lse must be a contiguous float32 [N, H] device tensor")
    _check(load_library().gt_attn_fwd_ex(dtype, _ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K),
                                         _ptr(V), _ptr(out), _ptr(lse), N, colidx.numel(), H, D,
                                         float(scale), tp, _stream(Q.device, stream)))


def gt_attn_fwd_noalloc(rowptr, colidx, Q, K, V, out, scale, tuning=None, stream=None, lse=None) -> None:
    """As gt_attn_fwd_ex, through the allocation-free entry point (workspace in
    the library's 256 MiB per-device scratch array; overlapping calls on one
    device race)."""
    if Q.dtype == torch.float32:
        dtype, allowed = GT_DTYPE_F32, (torch.float32,)
    else:
        dtype, allowed = GT_DTYPE_BF16, (torch.bfloat16, torch.int16, torch.uint16)
    _check_tensors(rowptr, colidx, Q, K, V, out, allowed)
    N, H, D = Q.shape
    if isinstance(tuning, dict):
        tuning = GtTuning(**tuning)
    tp = ctypes.byref(tuning) if tuning is not None else None
    if lse is not None:
        if not (lse.is_cuda and lse.device == out.device and lse.is_contiguous()
                and lse.dtype == torch.float32 and tuple(lse.shape) == (N, H)):
            raise ValueError("lse must be a contiguous float32 [N, H] device tensor")
    _check(load_library().gt_attn_fwd_noalloc(dtype, _ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K),
                                              _ptr(V), _ptr(out), _ptr(lse), N, colidx.numel(), H, D,
                                              float(scale), tp, _stream(Q.device, stream)))


def gt_gatv2_fwd(rowptr, colidx, L, R, att, slope, out, tuning=None, stream=None, lse=None) -> None:
    """GATv2 forward: out[i] = sum_e softmax_e(<att, LeakyReLU(L[i] + R[j_e])>) R[j_e]
    per head.  L, R, out: [N, H, D] (dtype from L); att: float32 [H, D] device
    tensor; slope: LeakyReLU negative slope; lse as in gt_attn_fwd_ex."""
    if L.dtype == torch.float32:
        dtype, allowed = GT_DTYPE_F32, (torch.float32,)
    else:
        dtype, allowed = GT_DTYPE_BF16, (torch.bfloat16, torch.int16, torch.uint16)
    _check_tensors(rowptr, colidx, L, R, R, out, allowed)
    N, H, D = L.shape
    if not (isinstance(att, torch.Tensor) and att.device == L.device and att.is_contiguous()
            and att.dtype == torch.float32 and tuple(att.shape) == (H, D)):
        raise ValueError("att must be a contiguous float32 [H, D] device tensor")
    if isinstance(tuning, dict):
        tuning = GtTuning(**tuning)
    tp = ctypes.byref(tuning) if tuning is not None else None
    if lse is not None:
        if not (lse.is_cuda and lse.device == out.device and lse.is_contiguous()
                and lse.dtype == torch.float32 and tuple(lse.shape) == (N, H)):
            raise ValueError("lse must be a contiguous float32 [N, H] device tensor")
    _check(load_library().gt_gatv2_fwd(dtype, _ptr(rowptr), _ptr(colidx), _ptr(L), _ptr(R),
                                       _ptr(att), float(slope), _ptr(out), _ptr(lse), N,
                                       colidx.numel(), H, D, tp, _stream(L.device, stream)))


DOT_MAPPINGS = {"feature": 0, "neighbor": 1}


def gt_dot_aggr(rowptr, colidx, X, out, mapping="feature", load_bytes=16, stream=None) -> None:
    """Locality-study microbenchmark: out[i] = sum over row i's entries of <X[i], X[j]>.
    X: float32 [N, F] device tensor; out: float32 [N]."""
    for name, t in (("rowptr", rowptr), ("colidx", colidx), ("X", X), ("out", out)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
            raise ValueError(name + " must be a contiguous device tensor")
    if any(t.device != X.device for t in (rowptr, colidx, out)):
        raise ValueError("all tensors must be on one device")
    if rowptr.dtype != torch.int64 or colidx.dtype != torch.int32:
        raise TypeError("rowptr must be int64 and colidx int32")
    if X.dtype != torch.float32 or out.dtype != torch.float32 or X.dim() != 2:
        raise TypeError("X must be float32 [N, F] and out float32 [N]")
    N, F = X.shape
    if out.numel() != N or rowptr.numel() != N + 1:
        raise ValueError("out must have N entries and rowptr N+1")
    _check(load_library().gt_dot_aggr(_ptr(rowptr), _ptr(colidx), _ptr(X), _ptr(out), N,
                                      colidx.numel(), F, DOT_MAPPINGS[mapping], int(load_bytes),
                                      _stream(X.device, stream)))


GT_REDUCE_OPS = {"min": 0, "max": 1}


def gt_segment_reduce(rowptr, colidx, X, out, arg=None, op="min", tuning=None, stream=None) -> None:
    """Segment min/max over each row's sources: out[i, f] and the source arg[i, f]
    that attains it (see include/gt_attn.h).  X, out: [N, F] (dtype from X);
    arg: int32 [N, F] device tensor or None."""
    if X.dtype == torch.float32:
        dtype, allowed = GT_DTYPE_F32, (torch.float32,)
    else:
        dtype, allowed = GT_DTYPE_BF16, (torch.bfloat16, torch.int16, torch.uint16)
    for name, t in (("rowptr", rowptr), ("colidx", colidx), ("X", X), ("out", out)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
            raise ValueError(name + " must be a contiguous device tensor")
    if any(t.device != X.device for t in (rowptr, colidx, out) + (() if arg is None else (arg,))):
        raise ValueError("all tensors must be on one device")
    if rowptr.dtype != torch.int64 or colidx.dtype != torch.int32:
        raise TypeError("rowptr must be int64 and colidx int32")
    if X.dim() != 2 or out.shape != X.shape or X.dtype not in allowed or out.dtype != X.dtype:
        raise ValueError("X and out must share one [N, F] shape and dtype")
    N, F = X.shape
    if rowptr.numel() != N + 1:
        raise ValueError("rowptr must have N+1 entries")
    if arg is not None and not (arg.is_cuda and arg.is_contiguous() and arg.dtype == torch.int32
                                and tuple(arg.shape) == (N, F)):
        raise ValueError("arg must be a contiguous int32 [N, F] device tensor")
    if isinstance(tuning, dict):
        tuning = GtTuning(**tuning)
    tp = ctypes.byref(tuning) if tuning is not None else None
    _check(load_library().gt_segment_reduce(dtype, GT_REDUCE_OPS[op], _ptr(rowptr), _ptr(colidx),
                                            _ptr(X), _ptr(out), _ptr(arg), N, colidx.numel(), F,
                                            tp, _stream(X.device, stream)))


def gt_attn_bwd(rowptr, colidx, rowptr_t, colidx_t, Q, K, V, out, dout, lse, dQ, dK, dV, scale,
                stream=None) -> None:
    """Gradients of sum(out * dout); see include/gt_attn.h.  rowptr_t/colidx_t
    is the transposed structure (sources as rows)."""
    if Q.dtype == torch.float32:
        dtype, allowed = GT_DTYPE_F32, (torch.float32,)
    else:
        dtype, allowed = GT_DTYPE_BF16, (torch.bfloat16, torch.int16, torch.uint16)
    _check_tensors(rowptr, colidx, Q, K, V, out, allowed)
    _check_tensors(rowptr_t, colidx_t, dout, dQ, dK, dV, allowed)
    N, H, D = Q.shape
    if colidx_t.numel() != colidx.numel():
        raise ValueError("the transposed structure must have as many entries as the CSR")
    if dout.device != Q.device:
        raise ValueError("all tensors must be on one device")
    if not (lse.is_cuda and lse.device == Q.device and lse.is_contiguous()
            and lse.dtype == torch.float32 and tuple(lse.shape) == (N, H)):
        raise ValueError("lse must be a contiguous float32 [N, H] device tensor")
    _check(load_library().gt_attn_bwd(dtype, _ptr(rowptr), _ptr(colidx), _ptr(rowptr_t),
                                      _ptr(colidx_t), _ptr(Q), _ptr(K), _ptr(V), _ptr(out),
                                      _ptr(dout), _ptr(lse), _ptr(dQ), _ptr(dK), _ptr(dV), N,
                                      colidx.numel(), H, D, float(scale),
                                      _stream(Q.device, stream)))


def attention(rowptr, colidx, Q, K, V, scale=None, tuning=None, out=None, stream=None,
              return_lse=False):
    """Convenience: allocates ``out`` like Q (and ``lse`` when asked) and
    dispatches on Q's dtype."""
    if out is None:
        out = torch.empty_like(Q)
    if scale is None:
        scale = Q.shape[-1] ** -0.5
    lse = torch.empty(Q.shape[:2], dtype=torch.float32, device=Q.device) if return_lse else None
    gt_attn_fwd_ex(rowptr, colidx, Q, K, V, out, scale, tuning=tuning, stream=stream, lse=lse)
    return (out, lse) if return_lse else out


def from_numpy(a):
    """numpy array -> contiguous tensor on the current device; uint16 arrays
    (bf16 bit patterns) become torch.bfloat16 with the same bits."""
    import numpy as np
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def to_numpy_f32(t):
    """Device tensor -> float32 numpy array (bf16 widened exactly)."""
    import numpy as np
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return (bits.astype(np.uint32) << 16).view(np.float32)
    return t.cpu().numpy()


def gt_csr_validate(rowptr, colidx, stream=None) -> bool:
    """Device-side CSR structure check (synchronous)."""
    for name, t in (("rowptr", rowptr), ("colidx", colidx)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
            raise ValueError(name + " must be a contiguous device tensor")
    if colidx.device != rowptr.device:
        raise ValueError("all tensors must be on one device")
    if rowptr.dtype != torch.int64 or colidx.dtype != torch.int32:
        raise TypeError("rowptr must be int64 and colidx int32")
    if rowptr.numel() < 1:
        raise ValueError("rowptr must have N+1 >= 1 entries")
    valid = ctypes.c_int32(0)
    _check(load_library().gt_csr_validate(_ptr(rowptr), _ptr(colidx), rowptr.numel() - 1,
                                          colidx.numel(), ctypes.byref(valid),
                                          _stream(rowptr.device, stream)))
    return bool(valid.value)


def gt_profile_enable(enable: bool = True) -> None:
    _check(load_library().gt_profile_enable(1 if enable else 0))


def gt_profile_collect():
    """Returns ([partition_ms, attention_ms, merge_ms] summed over calls, calls)."""
    ms = (ctypes.c_double * 3)()
    calls = ctypes.c_int64(0)
    _check(load_library().gt_profile_collect(ms, ctypes.byref(calls)))
    return [ms[0], ms[1], ms[2]], calls.value


def gt_workspace_pool_stats(device=None):
    """(reserved_bytes, used_bytes) of the library's workspace pool on a device
    (default: the current one)."""
    dev = torch.cuda.current_device() if device is None else int(device)
    r, u = ctypes.c_uint64(0), ctypes.c_uint64(0)
    _check(load_library().gt_workspace_pool_stats(dev, ctypes.byref(r), ctypes.byref(u)))
    return r.value, u.value


def gt_workspace_release() -> None:
    """Return the unused memory of the library's workspace pools to the devices."""
    _check(load_library().gt_workspace_release())
