"""Seeded synthetic graphs and features for CSR graph attention.

This module holds input generation only (no attention arithmetic).  The CPU
oracle and the GPU path both take their inputs from here and from nowhere
else.  Graphs are CSR with destination rows: ``rowptr`` int64[N+1] and
``colidx`` int32[E] listing the in-neighbours (sources) of each row, self-loops
included where a recipe says so.  Features are ``[N, H, D]`` row-major, fp32 or
bf16 (stored as uint16 bit patterns, rounded to nearest even from fp32).

The five named workloads stand in for the paper's datasets (Appendix C,
dataset statistics table), which are not available here; their recipes are
the shapes those datasets have (node count, edge count, degree skew, local
density), not the datasets themselves.

Randomness: Philox4x32-10 keyed by (seed, stream), implemented in
``synth.c``; every value is a pure function of its counter.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_SO = os.path.join(_HERE, "libsynth.so")

STREAM_GRAPH = 1
STREAM_Q = 2
STREAM_K = 3
STREAM_V = 4
STREAM_DEG = 5
STREAM_PERM = 6
STREAM_ROUND = 7
STREAM_EXTRA = 8

_lib = None


def build() -> str:
    """Compile synth.c into libsynth.so (always recompiles)."""
    tmp = _SO + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", "-O3", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", _SRC,
                    "-o", tmp, "-lm"], check=True)
    os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_SO):
        build()
    L = ctypes.CDLL(_SO)
    P = ctypes.c_void_p
    i64, u64, u32, dbl, ci = ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_double, ctypes.c_int
    L.synth_philox4x32_10.argtypes = [P, P, P]
    L.synth_philox4x32_10.restype = None
    L.synth_normal.argtypes = [u64, u32, dbl, i64, P, P]
    L.synth_normal.restype = None
    L.synth_uniform01.argtypes = [u64, u32, i64, P]
    L.synth_uniform01.restype = None
    L.synth_distinct_sources.argtypes = [u64, u32, i64, P, P, ci]
    L.synth_distinct_sources.restype = ci
    L.synth_rmat.argtypes = [u64, u32, ci, dbl, dbl, dbl, i64, i64, P, P]
    L.synth_rmat.restype = i64
    L.synth_csr_from_pairs.argtypes = [i64, i64, P, P, ci, P, P]
    L.synth_csr_from_pairs.restype = None
    L.synth_sbm.argtypes = [u64, u32, i64, i64, i64, P, P]
    L.synth_sbm.restype = None
    _lib = L
    return L


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


# ------------------------------------------------------------------ primitives

def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    lib().synth_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def normal(seed: int, stream: int, shape, std: float = 1.0, dtype: str = "f32") -> np.ndarray:
    """Gaussian array; dtype 'f32' -> float32, 'bf16' -> uint16 bf16 bits (RNE)."""
    n = int(np.prod(shape))
    if dtype == "f32":
        out = np.empty(shape, dtype=np.float32)
        lib().synth_normal(seed, stream, std, n, _p(out), None)
    elif dtype == "bf16":
        out = np.empty(shape, dtype=np.uint16)
        lib().synth_normal(seed, stream, std, n, None, _p(out))
    else:
        raise ValueError(dtype)
    return out


def uniform01(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    lib().synth_uniform01(seed, stream, n, _p(out))
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------- graphs

def csr_from_degrees(seed: int, N: int, deg: np.ndarray, self_loops: bool = True,
                     stream: int = STREAM_GRAPH):
    """Row i gets deg[i] distinct uniform sources from [0,N) minus i, plus itself."""
    deg = np.asarray(deg, dtype=np.int64)
    lens = deg + (1 if self_loops else 0)
    rowptr = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(lens, out=rowptr[1:])
    colidx = np.empty(int(rowptr[-1]), dtype=np.int32)
    rc = lib().synth_distinct_sources(seed, stream, N, _p(rowptr), _p(colidx), 1 if self_loops else 0)
    if rc != 0:
        raise ValueError("a row asks for more distinct sources than the graph has")
    return rowptr, colidx


def er_graph(seed: int, N: int, k: int):
    """Every node: k distinct uniform in-neighbours plus its self-loop."""
    return csr_from_degrees(seed, N, np.full(N, k, dtype=np.int64))


def shifted_zipf_degrees(seed: int, N: int, exponent: float, kmax: int, shift: float) -> np.ndarray:
    """d ~ P(k) proportional to (k + shift)^-exponent on k = 1..kmax (inverse CDF)."""
    k = np.arange(1, kmax + 1, dtype=np.float64)
    pmf = (k + shift) ** (-exponent)
    cdf = np.cumsum(pmf)
    cdf /= cdf[-1]
    u = uniform01(seed, STREAM_DEG, N)
    return (np.searchsorted(cdf, u, side="left") + 1).astype(np.int64)


def chung_lu_graph(seed: int, N: int, exponent: float = 2.1, kmax: int = 13000, shift: float = 0.532):
    deg = np.minimum(shifted_zipf_degrees(seed, N, exponent, kmax, shift), N - 1)
    return csr_from_degrees(seed, N, deg)


def rmat_graph(seed: int, scale: int, a: float, b: float, c: float, avg_deg: int):
    """R-MAT pairs (src bits = row of the R-MAT matrix), distinct, no self pairs,
    exactly (avg_deg - 1) * N of them, node ids randomly permuted, then a
    self-loop per node; CSR rows are destinations."""
    N = 1 << scale
    target = (avg_deg - 1) * N
    src = np.empty(target, dtype=np.int32)
    dst = np.empty(target, dtype=np.int32)
    used = lib().synth_rmat(seed, STREAM_GRAPH, scale, a, b, c, target, 4 * target, _p(src), _p(dst))
    if used < 0:
        raise RuntimeError("R-MAT sample budget exhausted")
    perm = np.argsort(uniform01(seed, STREAM_PERM, N), kind="stable").astype(np.int32)
    src = perm[src]
    dst = perm[dst]
    rowptr = np.empty(N + 1, dtype=np.int64)
    colidx = np.empty(target + N, dtype=np.int32)
    lib().synth_csr_from_pairs(N, target, _p(dst), _p(src), 1, _p(rowptr), _p(colidx))
    return rowptr, colidx


def sbm_graph(seed: int, N: int, block: int, n_out: int):
    """Contiguous blocks of `block` ids; intra-block pairs w.p. 1/2; n_out
    distinct uniform sources outside the block; self-loop.  Every block must
    leave at least n_out ids outside it (the draw of distinct sources would
    not end otherwise)."""
    if block < 1 or n_out < 0 or (n_out > 0 and N - min(block, N) < n_out):
        raise ValueError("sbm_graph: %d ids outside a block of %d cannot give %d distinct sources"
                         % (N - min(block, N), block, n_out))
    rowptr = np.empty(N + 1, dtype=np.int64)
    lib().synth_sbm(seed, STREAM_GRAPH, N, block, n_out, _p(rowptr), None)
    colidx = np.empty(int(rowptr[-1]), dtype=np.int32)
    lib().synth_sbm(seed, STREAM_GRAPH, N, block, n_out, _p(rowptr), _p(colidx))
    return rowptr, colidx


def lognormal_degrees(seed: int, N: int, mu: float, sigma: float, dmax: int, total: int) -> np.ndarray:
    """clip(round(exp(mu + sigma z)), 1, dmax), then rescaled to sum ~ total by
    stochastic rounding (each degree stays >= 1)."""
    z = normal(seed, STREAM_DEG, (N,), 1.0, "f32").astype(np.float64)
    d = np.clip(np.rint(np.exp(mu + sigma * z)), 1, dmax)
    x = d * (total / d.sum())
    fl = np.floor(x)
    u = uniform01(seed, STREAM_ROUND, N)
    d = fl + (u < (x - fl))
    return np.maximum(d, 1).astype(np.int64)


def lognormal_graph(seed: int, N: int, mu: float = 2.5, sigma: float = 1.5, dmax: int = 200000,
                    total: int = 30_000_000):
    deg = np.minimum(lognormal_degrees(seed, N, mu, sigma, dmax, total), N - 1)
    return csr_from_degrees(seed, N, deg)


def check_csr(rowptr: np.ndarray, colidx: np.ndarray, N: int) -> None:
    """Structural CSR invariants (raises AssertionError)."""
    assert rowptr.dtype == np.int64 and colidx.dtype == np.int32
    assert rowptr.shape == (N + 1,)
    assert rowptr[0] == 0 and rowptr[-1] == colidx.size
    assert np.all(np.diff(rowptr) >= 0)
    if colidx.size:
        assert colidx.min() >= 0 and colidx.max() < N


# ------------------------------------------------------------------- workloads

@dataclasses.dataclass
class Workload:
    name: str
    N: int
    E: int
    H: int
    D: int
    dtype: str          # 'f32' or 'bf16'
    scale: np.float32
    rowptr: np.ndarray
    colidx: np.ndarray
    Q: np.ndarray
    K: np.ndarray
    V: np.ndarray

    def describe(self) -> dict:
        return {"workload": self.name, "N": self.N, "E": self.E, "H": self.H, "D": self.D,
                "dtype": self.dtype}


def features(seed: int, N: int, H: int, D: int, dtype: str, std: float = 1.0):
    return tuple(normal(seed, s, (N, H, D), std, dtype) for s in (STREAM_Q, STREAM_K, STREAM_V))


def make_workload(name: str, rowptr, colidx, H: int, D: int, dtype: str, seed: int = 0,
                  std: float = 1.0, scale: float | None = None) -> Workload:
    N = rowptr.size - 1
    Q, K, V = features(seed, N, H, D, dtype, std)
    sc = np.float32(1.0 / math.sqrt(D)) if scale is None else np.float32(scale)
    return Workload(name, N, int(colidx.size), H, D, dtype, sc, rowptr, colidx, Q, K, V)


# The named workloads (index = position in the table of workload shapes).
# 0-4 are the five shapes the path is specified on; 5 is workload 2's graph
# (R-MAT scale 21) with fp32 features, the largest power-law graph in the
# paper's own CSR precision: its K and V (2.1 GB) far exceed the 256 MB
# Infinity Cache, so gathers are served by HBM.
CONFIG_NAMES = {
    0: "er-2k-h1d32-f32",
    1: "chunglu-arxiv-169k-h4d32-f32",
    2: "rmat-s21-h4d32-bf16",
    3: "sbm-1m-b64-h2d64-bf16",
    4: "lognormal-hub-1m-h8d64-bf16",
    5: "rmat-s21-h4d32-f32",
}

# graph recipe of each workload (workloads 2 and 5 share one graph)
GRAPH_OF = {0: "er-2k", 1: "chunglu-169k", 2: "rmat-s21", 3: "sbm-1m-b64", 4: "lognormal-1m", 5: "rmat-s21"}


def graph(name: str, seed: int = 0):
    """(rowptr, colidx) of a named graph recipe (see GRAPH_OF)."""
    if name == "er-2k":
        return er_graph(seed, 2000, 8)
    if name == "chunglu-169k":
        return chung_lu_graph(seed, 169_343)
    if name == "rmat-s21":
        return rmat_graph(seed, 21, 0.57, 0.19, 0.19, 24)
    if name == "sbm-1m-b64":
        return sbm_graph(seed, 1 << 20, 64, 4)
    if name == "lognormal-1m":
        return lognormal_graph(seed, 1_000_000)
    raise ValueError(name)


def config_from_graph(idx: int, rowptr, colidx, seed: int = 0) -> Workload:
    """Workload idx on its graph (as returned by graph(GRAPH_OF[idx], seed))."""
    name = CONFIG_NAMES[idx]
    if idx == 0:
        return make_workload(name, rowptr, colidx, 1, 32, "f32", seed)
    if idx == 1:
        return make_workload(name, rowptr, colidx, 4, 32, "f32", seed)
    if idx == 2:
        return make_workload(name, rowptr, colidx, 4, 32, "bf16", seed)
    if idx == 3:
        return make_workload(name, rowptr, colidx, 2, 64, "bf16", seed)
    if idx == 4:
        return make_workload(name, rowptr, colidx, 8, 64, "bf16", seed, std=0.5)
    if idx == 5:
        return make_workload(name, rowptr, colidx, 4, 32, "f32", seed)
    raise ValueError(idx)


def config(idx: int, seed: int = 0) -> Workload:
    """Full-size workload idx (0..5)."""
    if idx not in CONFIG_NAMES:
        raise ValueError(idx)
    return config_from_graph(idx, *graph(GRAPH_OF[idx], seed), seed=seed)


def ragged_graph(seed: int, N: int, max_deg: int, empty_frac: float = 0.1, hubs=None,
                 self_loops: bool = False, dup_frac: float = 0.0, shuffle: bool = False):
    """Small irregular CSR for edge-case tests.

    Degrees uniform in [0, max_deg]; a fraction `empty_frac` of rows forced
    empty; `hubs` maps row -> degree (must be <= N-1).  Sources are distinct
    and exclude the row itself (plus the self-loop when `self_loops`).  With
    dup_frac > 0 each entry after the first of a row is replaced, with that
    probability, by the entry before it (repeated entries).  With shuffle the
    entries of each row are put in a random order.
    """
    u = uniform01(seed, STREAM_EXTRA, 3 * N)
    deg = np.minimum(np.floor(u[:N] * (max_deg + 1)).astype(np.int64), N - 1)
    deg[u[N:2 * N] < empty_frac] = 0
    for r, d in (hubs or {}).items():
        deg[r] = d
    rowptr, colidx = csr_from_degrees(seed, N, deg, self_loops=self_loops)
    E = colidx.size
    if E and dup_frac > 0:
        ue = uniform01(seed, STREAM_EXTRA + 1, E)
        starts = np.zeros(E, dtype=bool)
        starts[rowptr[:-1][np.diff(rowptr) > 0]] = True
        rep = (ue < dup_frac) & ~starts
        # copy forward sequentially so runs of repeats chain correctly
        idx = np.arange(E)
        src_pos = np.where(rep, idx - 1, idx)
        for _ in range(int(max_deg) + 2):
            nxt = src_pos[src_pos]
            if np.array_equal(nxt, src_pos):
                break
            src_pos = nxt
        colidx = colidx[src_pos].copy()
    if E and shuffle:
        us = uniform01(seed, STREAM_EXTRA + 2, E)
        row_of = np.repeat(np.arange(N), np.diff(rowptr))
        order = np.lexsort((us, row_of))
        colidx = colidx[order].copy()
    return rowptr, colidx


def transpose_csr(rowptr: np.ndarray, colidx: np.ndarray, N: int):
    """Transposed structure: row j lists every destination i whose row holds j
    (one entry per CSR entry, destinations in increasing order)."""
    rows = np.repeat(np.arange(N, dtype=np.int32), np.diff(rowptr))
    order = np.argsort(colidx, kind="stable")
    colidx_t = np.ascontiguousarray(rows[order])
    rowptr_t = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(np.bincount(colidx, minlength=N), out=rowptr_t[1:])
    return rowptr_t, colidx_t


# ------------------------------------------------------------ node orderings
# Relabelings for the locality study: new node k is old node perm[k].

def permute_graph(rowptr: np.ndarray, colidx: np.ndarray, perm: np.ndarray):
    """CSR of the relabeled graph: row k is old row perm[k] with every source
    mapped to its new id; each row keeps its entry order.  Features follow
    with X[perm]."""
    N = rowptr.size - 1
    perm = np.ascontiguousarray(perm, dtype=np.int64)
    if perm.size != N or not np.array_equal(np.sort(perm), np.arange(N)):
        raise ValueError("perm must be a permutation of 0..N-1")
    inv = np.empty(N, dtype=np.int64)
    inv[perm] = np.arange(N)
    deg = np.diff(rowptr)[perm]
    new_rowptr = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(deg, out=new_rowptr[1:])
    # gather the old rows in the new order, then map their sources
    starts = rowptr[:-1][perm]
    idx = np.repeat(starts - new_rowptr[:-1], deg) + np.arange(new_rowptr[-1])
    new_colidx = inv[colidx[idx]].astype(np.int32)
    return new_rowptr, new_colidx


def random_order(seed: int, N: int) -> np.ndarray:
    """A uniformly random relabeling (argsort of seeded uniforms)."""
    return np.argsort(uniform01(seed, STREAM_PERM, N), kind="stable")


def rcm_order(rowptr: np.ndarray, colidx: np.ndarray) -> np.ndarray:
    """Reverse Cuthill-McKee order of the symmetrized graph (scipy): a
    bandwidth-reducing relabeling that places neighbourhoods at nearby ids,
    standing in for partition-based reorderings such as METIS."""
    import scipy.sparse as sp
    from scipy.sparse.csgraph import reverse_cuthill_mckee
    N = rowptr.size - 1
    A = sp.csr_matrix((np.ones(colidx.size, dtype=np.int8), colidx, rowptr), shape=(N, N))
    S = (A + A.T).tocsr()
    return np.asarray(reverse_cuthill_mckee(S, symmetric_mode=True), dtype=np.int64)
