"""GPU parity of the fused GATv2 forward (paper Section 2.2, GATv2 logits
a^T LeakyReLU(l_i + r_j) and values r_j; Appendix D.2, fused GATv2 forward)
against the float64 oracle on the same seeded inputs, through the C ABI.

Gate as for the graph-transformer forward: max_e |x - r| / max(|r|, absagg)
<= 1e-5 for fp32 features, <= 2e-2 for bf16 features; lse within 1e-5 of the
oracle relative to max(1, |lse|).  The score is a D-term fp32 sum of
products of the attention vector with LeakyReLU values of magnitude O(1), the
same rounding profile as the scaled dot product of the other forward.

Inputs: L and R are the workload's first two feature tensors (N(0,1) entries),
the attention vector is N(0, 1/D) per entry (a Glorot-scale initialisation, so
scores are O(1)); one case uses N(0, 1) for peaked softmax weights."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import (TOL_BF16, TOL_F32, bf16_bits_to_f32, gate_error, row_blocks,
                           to_device, to_host_f32, workload)

pytestmark = pytest.mark.gpu

SHAPES = [(h, d) for h in (1, 2, 4, 8) for d in (32, 64, 128, 256)]
BF16_ONLY = [(1, 512), (2, 512), (4, 512)]  # a 512-element fp32 head exceeds 64 lanes of 16 B
CASES = [(h, d, t) for (h, d) in SHAPES for t in ("f32", "bf16")] + [(h, d, "bf16") for (h, d) in BF16_ONLY]
FORCED_SPLIT = {"light_max_deg": 2, "heavy_min_deg": 6, "chunk_edges": 64, "grid_blocks": 0}
SLOPE = 0.2


def tol(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


def attention_vector(seed, H, D, std=None):
    return synth.normal(seed, synth.STREAM_EXTRA + 9, (H, D),
                        1.0 / math.sqrt(D) if std is None else std, "f32")


def run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, slope, tuning=None):
    import torch
    import paper_2605_31500_amd as gt
    rp, ci, l, r, a = (to_device(x) for x in (rowptr, colidx, Lf, Rf, att))
    out = torch.empty_like(l)
    lse = torch.empty(l.shape[:2], dtype=torch.float32, device=l.device)
    gt.gt_gatv2_fwd(rp, ci, l, r, a, slope, out, tuning=tuning, lse=lse)
    torch.cuda.synchronize()
    return to_host_f32(out), lse.cpu().numpy()


def check_lse(lse, ref, atol=1e-5):
    fin = np.isfinite(ref)
    assert np.array_equal(np.isneginf(lse), ~fin)
    assert np.all(np.abs(lse[fin] - ref[fin]) <= atol * np.maximum(1.0, np.abs(ref[fin])))


def check(rowptr, colidx, Lf, Rf, att, slope, dtype, tuning=None, rows=None):
    got, lse = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, slope, tuning=tuning)
    ref, absagg, ref_lse = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, slope, rows=rows)
    if rows is not None:
        got, lse = got[rows], lse[rows]
    assert np.all(np.isfinite(got))
    err = gate_error(got, ref, absagg)
    assert err <= tol(dtype), "gate error %.3g > %.3g" % (err, tol(dtype))
    check_lse(lse, ref_lse)
    return got


@pytest.mark.parametrize("split", [False, True], ids=["default", "forced_split"])
@pytest.mark.parametrize("H,D,dtype", CASES)
def test_gatv2_ragged_small(H, D, dtype, split):
    N = 300
    seed = 7000 + H * 1000 + D
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=24, empty_frac=0.1,
                                        hubs={7: 299, 100: 150, 299: 70}, self_loops=True,
                                        dup_frac=0.05, shuffle=True)
    Lf, Rf, _ = synth.features(seed, N, H, D, dtype)
    check(rowptr, colidx, Lf, Rf, attention_vector(seed, H, D), SLOPE, dtype,
          tuning=FORCED_SPLIT if split else None)


@pytest.mark.parametrize("slope", [0.0, 1.0, -0.5, 3.0])
def test_gatv2_slopes_and_peaked_scores(slope):
    # slope 0 is ReLU, 1 the identity (the l_i term then cancels in the
    # softmax), negative and > 1 slopes are legal values of the parameter
    N, H, D = 400, 4, 32
    rowptr, colidx = synth.ragged_graph(11, N, max_deg=40, empty_frac=0.05, hubs={3: 399},
                                        dup_frac=0.1, shuffle=True)
    Lf, Rf, _ = synth.features(11, N, H, D, "f32")
    check(rowptr, colidx, Lf, Rf, attention_vector(11, H, D, std=1.0), slope, "f32",
          tuning=FORCED_SPLIT)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gatv2_zero_attention_is_neighbour_mean(dtype):
    # a = 0 makes every score 0: the output is the plain mean of the gathered
    # R rows (an empty row gives 0), independent of the oracle
    N, H, D = 500, 2, 64
    rowptr, colidx = synth.ragged_graph(12, N, max_deg=30, empty_frac=0.1, hubs={9: 499},
                                        dup_frac=0.1, shuffle=True)
    Lf, Rf, _ = synth.features(12, N, H, D, dtype)
    got, lse = run_gpu_gatv2(rowptr, colidx, Lf, Rf, np.zeros((H, D), np.float32), SLOPE)
    R64 = (Rf if dtype == "f32" else bf16_bits_to_f32(Rf)).astype(np.float64)
    deg = np.diff(rowptr)
    want = np.zeros((N, H, D))
    absm = np.zeros((N, H, D))
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        if J.size:
            want[i] = R64[J].mean(axis=0)
            absm[i] = np.abs(R64[J]).mean(axis=0)
    assert gate_error(got, want, absm) <= tol(dtype)
    with np.errstate(divide="ignore"):
        ref_lse = np.repeat(np.log(deg.astype(np.float64))[:, None], H, axis=1)
    check_lse(lse, ref_lse)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gatv2_single_entry_rows_are_exact(dtype):
    # one entry per row: the weight is exactly 1, so out[i] == R[colidx[i]]
    N, H, D = 1000, 8, 32
    rowptr, colidx = synth.csr_from_degrees(13, N, np.ones(N, dtype=np.int64), self_loops=False)
    Lf, Rf, _ = synth.features(13, N, H, D, dtype)
    got, _ = run_gpu_gatv2(rowptr, colidx, Lf, Rf, attention_vector(13, H, D), SLOPE)
    want = (Rf if dtype == "f32" else bf16_bits_to_f32(Rf))[colidx]
    assert np.array_equal(got, want)


def test_gatv2_deterministic():
    N, H, D = 2000, 2, 64
    rowptr, colidx = synth.ragged_graph(14, N, max_deg=50, empty_frac=0.05,
                                        hubs={1: 1999, 2: 1500}, dup_frac=0.05, shuffle=True)
    Lf, Rf, _ = synth.features(14, N, H, D, "f32")
    att = attention_vector(14, H, D)
    a, la = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, SLOPE, tuning=FORCED_SPLIT)
    b, lb = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, SLOPE, tuning=FORCED_SPLIT)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4, 5])
def test_gatv2_full_config_all_rows(idx):
    w = workload(idx)
    print("config", idx, w.name, "N", w.N, "E", w.E, flush=True)
    att = attention_vector(idx, w.H, w.D)
    got, lse = run_gpu_gatv2(w.rowptr, w.colidx, w.Q, w.K, att, SLOPE)
    assert np.all(np.isfinite(got))
    err = 0.0
    for lo, hi in row_blocks(w.N, w.H * w.D):
        ref, absagg, ref_lse = oracle.gatv2_fwd(w.rowptr, w.colidx, w.Q, w.K, att, SLOPE,
                                                rows=np.arange(lo, hi, dtype=np.int64))
        err = max(err, gate_error(got[lo:hi], ref, absagg))
        check_lse(lse[lo:hi], ref_lse)
    print("gate error %.3g" % err, flush=True)
    assert err <= tol(w.dtype), "gate error %.3g > %.3g" % (err, tol(w.dtype))
