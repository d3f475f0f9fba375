"""Shared test helpers: the parity metric and the worked-example loader.

The parity metric compares a result x with the float64 reference r using the
scale sum_j alpha_ij |v_j| (``absagg``) that bounds the rounding error of any
floating-point evaluation of a convex combination (Higham, Accuracy and
Stability of Numerical Algorithms, ch. 4):

    err = max_e |x_e - r_e| / max(|r_e|, absagg_e, tiny)

Where no cancellation happens absagg_e == |r_e| and this is the ordinary
relative error.
"""
from __future__ import annotations

import functools
import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def gate_error(x, ref, absagg) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    denom = np.maximum(np.maximum(np.abs(ref), np.asarray(absagg, dtype=np.float64)), 1e-30)
    if x.size == 0:
        return 0.0
    return float(np.max(np.abs(x - ref) / denom))


def score_rounding_bound(rowptr, colidx, Q, K, scale) -> np.ndarray:
    """Per (row, head): the largest bound on the absolute rounding error of a
    computed score of the row, D * 2^-24 * scale * sum_d |q_d k_d| (the
    standard bound for a D-term fp32 dot product, plus the scaling).  Q, K:
    float32 or bf16 bits.  Rows without entries get 0."""
    N, H, D = Q.shape
    widen = lambda x: bf16_bits_to_f32(x) if x.dtype == np.uint16 else x
    q, k = np.abs(widen(Q).astype(np.float64)), np.abs(widen(K).astype(np.float64))
    deg = np.diff(rowptr)
    dst = np.repeat(np.arange(N), deg)
    per_entry = np.einsum("ehd,ehd->eh", q[dst], k[colidx]) * D * 2.0 ** -24 * scale
    bound = np.zeros((N, H))
    nz = deg > 0
    if per_entry.size:
        bound[nz] = np.maximum.reduceat(per_entry, rowptr[:-1][nz], axis=0)
    return bound


def bf16_bits_to_f32(bits) -> np.ndarray:
    return (np.asarray(bits).astype(np.uint32) << 16).view(np.float32)


def load_worked_example(name: str = "worked_example.txt") -> dict:
    rows = {}
    Q, K, V = {}, {}, {}
    OUT, ABS, LSE = {}, {}, {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tag, rest = line.split(None, 1)
            if tag in ("N", "H", "D"):
                rows[tag] = int(rest)
            elif tag == "scale":
                assert rest.strip() == "ln2"
                rows["scale"] = np.float32(math.log(2.0))
            elif tag == "rowptr":
                rows["rowptr"] = np.array([int(t) for t in rest.split()], dtype=np.int64)
            elif tag == "colidx":
                rows["colidx"] = np.array([int(t) for t in rest.split()], dtype=np.int32)
            elif tag in ("Q", "K", "V", "OUT", "ABS", "LSE"):
                idx, vals = rest.split(None, 1)
                heads = [h.split() for h in vals.split("|")]
                tgt = {"Q": Q, "K": K, "V": V, "OUT": OUT, "ABS": ABS, "LSE": LSE}[tag]
                tgt[int(idx)] = heads
    N, H, D = rows["N"], rows["H"], rows["D"]

    def arr(d, conv, dtype):
        a = np.zeros((N, H, D) if d is not LSE else (N, H), dtype=dtype)
        for i, heads in d.items():
            for h, vals in enumerate(heads):
                if d is LSE:
                    a[i, h] = conv(vals[0])
                else:
                    a[i, h, :] = [conv(v) for v in vals]
        return a

    def lnconv(s):
        if s == "-inf":
            return -math.inf
        assert s.startswith("ln(") and s.endswith(")")
        return math.log(float(Fraction(s[3:-1])))

    rows["Q"] = arr(Q, float, np.float32)
    rows["K"] = arr(K, float, np.float32)
    rows["V"] = arr(V, float, np.float32)
    rows["OUT"] = arr(OUT, lambda s: float(Fraction(s)), np.float64)
    rows["ABS"] = arr(ABS, lambda s: float(Fraction(s)), np.float64)
    rows["LSE"] = arr(LSE, lnconv, np.float64)
    return rows


# ------------------------------------------------------- workloads, row blocks

@functools.lru_cache(maxsize=None)
def _graph(name: str):
    import synth
    return synth.graph(name)


@functools.lru_cache(maxsize=None)
def workload(idx: int):
    """synth.config(idx), built once per test session (workloads 2 and 5 share
    one generated graph).  Callers must not modify the arrays."""
    import synth
    return synth.config_from_graph(idx, *_graph(synth.GRAPH_OF[idx]))


def row_blocks(N: int, elems_per_row: int, budget: int = 1 << 25):
    """Consecutive (lo, hi) row ranges covering [0, N), about `budget` output
    elements each: the oracle runs block by block, so that its float64 outputs
    stay a few hundred MB whatever the graph size."""
    step = max(1, budget // max(1, elems_per_row))
    for lo in range(0, N, step):
        yield lo, min(N, lo + step)


def fwd_gate_error_all_rows(w, got) -> float:
    """Gate error of a forward output (float32 [N, H, D]) against the oracle on
    every row of workload-like `w` (rowptr, colidx, Q, K, V, scale, N, H, D)."""
    import oracle
    err = 0.0
    for lo, hi in row_blocks(w.N, w.H * w.D):
        ref, absagg, _ = oracle.gt_attn_fwd(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale,
                                           rows=np.arange(lo, hi, dtype=np.int64), want_lse=False)
        err = max(err, gate_error(got[lo:hi], ref, absagg))
    return err


# ------------------------------------------------------------ device helpers

def to_device(a):
    """numpy -> torch CUDA tensor; uint16 arrays (bf16 bits) become torch.bfloat16."""
    import paper_2605_31500_amd as gt
    return gt.from_numpy(a)


def to_host_f32(t) -> np.ndarray:
    """torch CUDA tensor -> float32 numpy (bf16 widened exactly)."""
    import paper_2605_31500_amd as gt
    return gt.to_numpy_f32(t)


def run_gpu(rowptr, colidx, Q, K, V, scale, tuning=None, stream=None):
    """One call of the HIP path through the C ABI; returns float32 host output."""
    import torch
    import paper_2605_31500_amd as gt
    dt = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dt[2])
    gt.gt_attn_fwd_ex(*dt, out, scale, tuning=tuning, stream=stream)
    torch.cuda.synchronize()
    return to_host_f32(out)


def run_gpu_bare(rowptr, colidx, Q, K, V, scale, stream=None):
    """One call of the contract entry point of the feature dtype, gt_attn_fwd
    (fp32) or gt_attn_fwd_bf16, through the C ABI; float32 host output."""
    import torch
    import paper_2605_31500_amd as gt
    dt = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dt[2])
    fn = gt.gt_attn_fwd if Q.dtype == np.float32 else gt.gt_attn_fwd_bf16
    fn(*dt, out, scale, stream=stream)
    torch.cuda.synchronize()
    return to_host_f32(out)


def sample_rows(rowptr: np.ndarray, n_random: int, n_top: int, seed: int = 0) -> np.ndarray:
    """Rows to check at full size: the n_top highest-degree rows, n_random rows
    drawn uniformly (seeded), the first and last rows, and one row of each
    degree 0, 1 and 2 when present."""
    import synth
    N = rowptr.size - 1
    deg = np.diff(rowptr)
    top = np.argsort(deg, kind="stable")[-n_top:]
    rnd = np.floor(synth.uniform01(seed, synth.STREAM_EXTRA + 7, n_random) * N).astype(np.int64)
    extra = [0, N - 1]
    for d in (0, 1, 2):
        hit = np.flatnonzero(deg == d)
        if hit.size:
            extra.append(int(hit[0]))
    return np.unique(np.concatenate([top, rnd, np.array(extra, dtype=np.int64)]))


def run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, scale, tuning=None):
    """Forward (with lse) then backward through the C ABI; float32 host results
    (out, lse, dQ, dK, dV)."""
    import torch
    import paper_2605_31500_amd as gt
    import synth
    N, H, D = Q.shape
    rpt, cit = synth.transpose_csr(rowptr, colidx, N)
    rp, ci, rpt_d, cit_d, q, k, v, do = (to_device(x) for x in (rowptr, colidx, rpt, cit, Q, K, V, dO))
    out = torch.empty_like(q)
    lse = torch.empty((N, H), dtype=torch.float32, device=q.device)
    gt.gt_attn_fwd_ex(rp, ci, q, k, v, out, scale, tuning=tuning, lse=lse)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    gt.gt_attn_bwd(rp, ci, rpt_d, cit_d, q, k, v, out, do, lse, dq, dk, dv, scale)
    torch.cuda.synchronize()
    return (to_host_f32(out), lse.cpu().numpy(), to_host_f32(dq), to_host_f32(dk), to_host_f32(dv))
