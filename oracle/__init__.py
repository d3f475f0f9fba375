"""CPU oracle for the CSR operators of the paper: graph-transformer attention
(forward and backward) and GATv2 attention in float64, and the segment min/max
reduction with its selected sources.

TEST INFRASTRUCTURE: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product path
(the HIP library and its binding) never imports or calls it, and this package
never imports the product path.

The arithmetic lives in ``gt_oracle.c`` (plain two-pass softmax per row and
head, paper Section 2.2 family (iii); plain per-feature scans for family
(ii)).  This file only compiles it and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gt_oracle.c")
_SO = os.path.join(_HERE, "libgt_oracle.so")
_lib = None


def build() -> str:
    """Compile gt_oracle.c (always recompiles).  IEEE semantics: no fast-math."""
    tmp = _SO + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp,
                    "-lm"], check=True)
    os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        L.gt_oracle_fwd.argtypes = [ctypes.c_int, P, P, P, P, P, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_float, P,
                                    ctypes.c_int64, P, P, P]
        L.gt_oracle_fwd.restype = ctypes.c_int
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        L.gt_oracle_bwd_dq.argtypes = [ctypes.c_int, P, P, P, P, P, P, i64, i64, i32, i32,
                                       ctypes.c_float, P, i64, P, P]
        L.gt_oracle_bwd_dq.restype = ctypes.c_int
        L.gt_oracle_bwd_dkv.argtypes = [ctypes.c_int, P, P, P, P, P, P, P, P, i64, i64, i32, i32,
                                        ctypes.c_float, P, i64, P, P, P, P]
        L.gt_oracle_bwd_dkv.restype = ctypes.c_int
        L.gt_oracle_gatv2_fwd.argtypes = [ctypes.c_int, P, P, P, P, P, i64, i64, i32, i32,
                                          ctypes.c_float, P, i64, P, P, P]
        L.gt_oracle_gatv2_fwd.restype = ctypes.c_int
        L.gt_oracle_segment_reduce.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, i64, i64, i32,
                                               P, i64, P, P]
        L.gt_oracle_segment_reduce.restype = ctypes.c_int
        L.gt_oracle_dot_aggr.argtypes = [P, P, P, i64, i64, i32, P, i64, P, P]
        L.gt_oracle_dot_aggr.restype = ctypes.c_int
        L.gt_oracle_threads.argtypes = []
        L.gt_oracle_threads.restype = ctypes.c_int
        L.gt_oracle_set_threads.argtypes = [ctypes.c_int]
        L.gt_oracle_set_threads.restype = None
        _lib = L
    return _lib


def threads() -> int:
    return int(_load().gt_oracle_threads())


def set_threads(n: int) -> None:
    """OpenMP threads of later oracle calls in this process (n >= 1)."""
    _load().gt_oracle_set_threads(int(n))


def _ptr(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def gt_attn_fwd(rowptr, colidx, Q, K, V, scale, rows=None, want_absagg=True, want_lse=True):
    """Reference forward.  Q/K/V: [N,H,D] float32, or uint16 bf16 bit patterns.

    Returns (out, absagg, lse) as float64 arrays shaped [R,H,D], [R,H,D], [R,H]
    for the requested rows (all rows when ``rows`` is None); absagg/lse are
    None when not requested.
    """
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    Q, K, V = (np.ascontiguousarray(x) for x in (Q, K, V))
    if not (Q.dtype == K.dtype == V.dtype) or Q.dtype not in (np.float32, np.uint16):
        raise TypeError("Q, K, V must all be float32 or all uint16 (bf16 bits)")
    if Q.ndim != 3 or K.shape != Q.shape or V.shape != Q.shape:
        raise ValueError("Q, K, V must share one [N, H, D] shape")
    N, H, D = Q.shape
    if rowptr.shape != (N + 1,):
        raise ValueError("rowptr must have N+1 entries")
    dtype = 0 if Q.dtype == np.float32 else 1
    if rows is None:
        rows_arr, nrows = None, N
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        nrows = rows_arr.size
    out = np.empty((nrows, H, D), dtype=np.float64)
    absagg = np.empty_like(out) if want_absagg else None
    lse = np.empty((nrows, H), dtype=np.float64) if want_lse else None
    rc = _load().gt_oracle_fwd(dtype, _ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K), _ptr(V), N,
                               colidx.size, H, D, ctypes.c_float(float(scale)), _ptr(rows_arr),
                               nrows, _ptr(out), _ptr(absagg), _ptr(lse))
    if rc == 1:
        raise ValueError("oracle: invalid arguments")
    if rc == 2:
        raise ValueError("oracle: invalid CSR structure")
    return out, absagg, lse


def _features(Q, K, V, extra=()):
    arrs = [np.ascontiguousarray(x) for x in (Q, K, V) + tuple(extra)]
    if any(a.dtype != arrs[0].dtype for a in arrs) or arrs[0].dtype not in (np.float32, np.uint16):
        raise TypeError("features must all be float32 or all uint16 (bf16 bits)")
    if any(a.shape != arrs[0].shape for a in arrs) or arrs[0].ndim != 3:
        raise ValueError("features must share one [N, H, D] shape")
    return arrs, (0 if arrs[0].dtype == np.float32 else 1)


def gt_attn_bwd_dq(rowptr, colidx, Q, K, V, dO, scale, rows=None):
    """dQ and its error scale (float64 [R, H, D] each) for the requested rows."""
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    (Q, K, V, dO), dtype = _features(Q, K, V, (dO,))
    N, H, D = Q.shape
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    nrows = N if rows is None else rows_arr.size
    dQ = np.empty((nrows, H, D))
    sdQ = np.empty_like(dQ)
    rc = _load().gt_oracle_bwd_dq(dtype, _ptr(rowptr), _ptr(colidx), _ptr(Q), _ptr(K), _ptr(V),
                                  _ptr(dO), N, colidx.size, H, D, ctypes.c_float(float(scale)),
                                  _ptr(rows_arr), nrows, _ptr(dQ), _ptr(sdQ))
    if rc:
        raise ValueError("oracle: invalid arguments or CSR (code %d)" % rc)
    return dQ, sdQ


def gt_attn_bwd_dkv(rowptr, colidx, rowptr_t, colidx_t, Q, K, V, dO, scale, cols=None):
    """dK, dV and their error scales (float64 [C, H, D] each) for the requested
    source ids; rowptr_t/colidx_t is the transposed CSR (sources as rows)."""
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    rowptr_t = np.ascontiguousarray(rowptr_t, dtype=np.int64)
    colidx_t = np.ascontiguousarray(colidx_t, dtype=np.int32)
    (Q, K, V, dO), dtype = _features(Q, K, V, (dO,))
    N, H, D = Q.shape
    cols_arr = None if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
    ncols = N if cols is None else cols_arr.size
    dK = np.empty((ncols, H, D))
    dV, sdK, sdV = np.empty_like(dK), np.empty_like(dK), np.empty_like(dK)
    rc = _load().gt_oracle_bwd_dkv(dtype, _ptr(rowptr), _ptr(colidx), _ptr(rowptr_t),
                                   _ptr(colidx_t), _ptr(Q), _ptr(K), _ptr(V), _ptr(dO), N,
                                   colidx.size, H, D, ctypes.c_float(float(scale)), _ptr(cols_arr),
                                   ncols, _ptr(dK), _ptr(dV), _ptr(sdK), _ptr(sdV))
    if rc:
        raise ValueError("oracle: invalid arguments or CSR (code %d)" % rc)
    return dK, dV, sdK, sdV


def gatv2_fwd(rowptr, colidx, Lf, Rf, att, slope, rows=None, want_absagg=True, want_lse=True):
    """GATv2 reference forward.  Lf, Rf: [N,H,D] float32 or uint16 bf16 bits;
    att: [H,D] float32; slope: LeakyReLU negative slope.  Returns (out, absagg, lse)."""
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    arrs, dtype = _features(Lf, Rf, Rf)
    Lf, Rf = arrs[0], arrs[1]
    att = np.ascontiguousarray(att, dtype=np.float32)
    N, H, D = Lf.shape
    if att.shape != (H, D):
        raise ValueError("att must be [H, D]")
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    nrows = N if rows is None else rows_arr.size
    out = np.empty((nrows, H, D))
    absagg = np.empty_like(out) if want_absagg else None
    lse = np.empty((nrows, H)) if want_lse else None
    rc = _load().gt_oracle_gatv2_fwd(dtype, _ptr(rowptr), _ptr(colidx), _ptr(Lf), _ptr(Rf),
                                     _ptr(att), N, colidx.size, H, D, ctypes.c_float(float(slope)),
                                     _ptr(rows_arr), nrows, _ptr(out), _ptr(absagg), _ptr(lse))
    if rc:
        raise ValueError("oracle: invalid arguments or CSR (code %d)" % rc)
    return out, absagg, lse


REDUCE_OPS = {"min": 0, "max": 1}


def segment_reduce(rowptr, colidx, X, op="min", rows=None):
    """Min or max of each row's source features (paper Section 2.2, family (ii)),
    with the source that attains it.  X: [N, F] float32 or uint16 bf16 bits.
    Returns (out float32 [nrows, F], arg int32 [nrows, F]); an empty row gives
    0 and -1.  Ties go to the smallest source id; -0 orders below +0."""
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    X = np.ascontiguousarray(X)
    if X.dtype == np.float32:
        dtype = 0
    elif X.dtype == np.uint16:
        dtype = 1
    else:
        raise TypeError("X must be float32 or uint16 (bf16 bits)")
    if X.ndim != 2:
        raise ValueError("X must be [N, F]")
    N, F = X.shape
    if rowptr.size != N + 1:
        raise ValueError("rowptr must have N+1 entries")
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    nrows = N if rows is None else rows_arr.size
    out = np.empty((nrows, F), dtype=np.float32)
    arg = np.empty((nrows, F), dtype=np.int32)
    rc = _load().gt_oracle_segment_reduce(dtype, REDUCE_OPS[op], _ptr(rowptr), _ptr(colidx),
                                          _ptr(X), N, colidx.size, F, _ptr(rows_arr), nrows,
                                          _ptr(out), _ptr(arg))
    if rc:
        raise ValueError("oracle: invalid arguments or CSR (code %d)" % rc)
    return out, arg


def dot_aggr(rowptr, colidx, X, rows=None):
    """Locality-study microbenchmark: s[i] = sum over row i's entries of <X[i], X[j]>.
    X: [N, F] float32.  Returns (s, abs) float64 [nrows]; abs is the sum of the
    absolute products (rounding-error scale)."""
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    colidx = np.ascontiguousarray(colidx, dtype=np.int32)
    X = np.ascontiguousarray(X, dtype=np.float32)
    if X.ndim != 2:
        raise ValueError("X must be [N, F]")
    N, F = X.shape
    if rowptr.size != N + 1:
        raise ValueError("rowptr must have N+1 entries")
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    nrows = N if rows is None else rows_arr.size
    out = np.empty(nrows)
    absout = np.empty(nrows)
    rc = _load().gt_oracle_dot_aggr(_ptr(rowptr), _ptr(colidx), _ptr(X), N, colidx.size, F,
                                    _ptr(rows_arr), nrows, _ptr(out), _ptr(absout))
    if rc:
        raise ValueError("oracle: invalid arguments or CSR (code %d)" % rc)
    return out, absout
