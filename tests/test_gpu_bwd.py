"""GPU parity of the logsumexp output and of the backward pass (Appendix D.2
of the paper: weights recomputed from the stored row statistic) against the
float64 oracle.  Gradient gate: max |x - r| / max(|r|, S) with S the same sums
over absolute values of every factor (returned by the oracle); 1e-5 for fp32,
2e-2 for bf16."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import (TOL_BF16, TOL_F32, gate_error, row_blocks, run_gpu_fwd_bwd,
                           score_rounding_bound, workload)

pytestmark = pytest.mark.gpu

SHAPES = [(h, d) for h in (1, 2, 4, 8) for d in (32, 64, 128, 256)]
BF16_ONLY = [(1, 512), (2, 512), (4, 512)]  # a 512-element fp32 head exceeds 64 lanes of 16 B
CASES = [(h, d, t) for (h, d) in SHAPES for t in ("f32", "bf16")] + [(h, d, "bf16") for (h, d) in BF16_ONLY]
FORCED_SPLIT = {"light_max_deg": 2, "heavy_min_deg": 6, "chunk_edges": 64, "grid_blocks": 0}


def tol(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


def check_lse(lse, ref, atol):
    fin = np.isfinite(ref)
    assert np.array_equal(np.isneginf(lse), ~fin)
    assert np.all(np.abs(lse[fin] - ref[fin]) <= atol * np.maximum(1.0, np.abs(ref[fin])))


def check_grads(rowptr, colidx, Q, K, V, dO, scale, got, dtype, rows=None, cols=None):
    _, _, dq, dk, dv = got
    N = Q.shape[0]
    rpt, cit = synth.transpose_csr(rowptr, colidx, N)
    rq, sq = oracle.gt_attn_bwd_dq(rowptr, colidx, Q, K, V, dO, scale, rows=rows)
    rk, rv, sk, sv = oracle.gt_attn_bwd_dkv(rowptr, colidx, rpt, cit, Q, K, V, dO, scale, cols=cols)
    if rows is not None:
        dq = dq[rows]
    if cols is not None:
        dk, dv = dk[cols], dv[cols]
    for name, x, r, sc in (("dQ", dq, rq, sq), ("dK", dk, rk, sk), ("dV", dv, rv, sv)):
        assert np.all(np.isfinite(x)), name
        err = gate_error(x, r, sc)
        assert err <= tol(dtype), "%s gate error %.3g" % (name, err)


@pytest.mark.parametrize("split", [False, True], ids=["default", "forced_split"])
@pytest.mark.parametrize("H,D,dtype", CASES)
def test_lse_and_backward_small(H, D, dtype, split):
    N = 300
    seed = 7000 + H * 100 + D
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=24, empty_frac=0.1,
                                        hubs={7: 299, 100: 150, 299: 70}, self_loops=True,
                                        dup_frac=0.05, shuffle=True)
    Q, K, V = synth.features(seed, N, H, D, dtype)
    dO, _, _ = synth.features(seed + 1, N, H, D, dtype)
    scale = np.float32(1 / math.sqrt(D))
    got = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, scale,
                          tuning=FORCED_SPLIT if split else None)
    _, _, ref_lse = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_absagg=False)
    check_lse(got[1], ref_lse, 1e-5)
    check_grads(rowptr, colidx, Q, K, V, dO, scale, got, dtype)


def per_node_error(x, r, scale):
    """max over the feature axis of |x - r| / max(|r|, S): [nodes, H]."""
    return np.max(np.abs(x - r) / np.maximum(np.maximum(np.abs(r), scale), 1e-30), axis=2)


@pytest.mark.parametrize("split", [False, True], ids=["default", "forced_split"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_peaked_scores(dtype, split):
    """Scores spread over hundreds of units (most weights underflow, one or two
    entries carry a row).  A recomputed weight exp(s_e - lse_i) is off by at
    most the rounding errors of s_e and of lse_i, and Delta_i = <out_i, dout_i>
    inherits the error of out_i, each at most the row's worst score error e_i
    (tests.helpers.score_rounding_bound).  So dQ of row i is held to 3 e_i, and
    dK, dV of node j to 3 max e_i over the rows i that hold j, plus the gate."""
    N, H, D = 3000, 4, 32
    scale = 6.0
    rowptr, colidx = synth.ragged_graph(41, N, max_deg=40, hubs={3: 2999, 9: 1800})
    Q, K, V = synth.features(41, N, H, D, dtype)
    dO, _, _ = synth.features(42, N, H, D, dtype)
    out, lse, dq, dk, dv = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, np.float32(scale),
                                           tuning=FORCED_SPLIT if split else None)
    gate = tol(dtype)
    e_row = score_rounding_bound(rowptr, colidx, Q, K, scale)
    e_col = np.zeros_like(e_row)
    np.maximum.at(e_col, colidx, e_row[np.repeat(np.arange(N), np.diff(rowptr))])
    _, _, ref_lse = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_absagg=False)
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isneginf(lse), ~fin)
    assert np.all(np.abs(lse[fin] - ref_lse[fin]) <= e_row[fin] + 1e-5 * np.maximum(1.0, np.abs(ref_lse[fin])))
    rpt, cit = synth.transpose_csr(rowptr, colidx, N)
    rq, sq = oracle.gt_attn_bwd_dq(rowptr, colidx, Q, K, V, dO, scale)
    rk, rv, sk, sv = oracle.gt_attn_bwd_dkv(rowptr, colidx, rpt, cit, Q, K, V, dO, scale)
    for name, x, r, sc, e in (("dQ", dq, rq, sq, e_row), ("dK", dk, rk, sk, e_col), ("dV", dv, rv, sv, e_col)):
        assert np.all(np.isfinite(x)), name
        err = per_node_error(x, r, sc)
        bound = 3.0 * e + gate
        assert np.all(err <= bound), "%s worst ratio %.3g" % (name, np.max(err / bound))


def test_backward_deterministic():
    N, H, D = 5000, 4, 32
    rowptr, colidx = synth.ragged_graph(31, N, max_deg=30, hubs={1: 4999, 2: 3000})
    Q, K, V = synth.features(31, N, H, D, "f32")
    dO, _, _ = synth.features(32, N, H, D, "f32")
    a = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, np.float32(0.2))
    b = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, np.float32(0.2))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_entry_rows_zero_query_key_gradients(dtype):
    N, H, D = 3000, 4, 32
    rowptr, colidx = synth.csr_from_degrees(33, N, np.ones(N, dtype=np.int64), self_loops=False)
    Q, K, V = synth.features(33, N, H, D, dtype)
    dO, _, _ = synth.features(34, N, H, D, dtype)
    got = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, np.float32(0.3))
    assert np.all(got[2] == 0) and np.all(got[3] == 0)
    check_grads(rowptr, colidx, Q, K, V, dO, np.float32(0.3), got, dtype)


def test_lse_tile_mode():
    w_rp, w_ci = synth.sbm_graph(35, 64 * 20 + 9, 64, 4)
    N = w_rp.size - 1
    Q, K, V = synth.features(35, N, 2, 64, "bf16")
    dO, _, _ = synth.features(36, N, 2, 64, "bf16")
    got = run_gpu_fwd_bwd(w_rp, w_ci, Q, K, V, dO, np.float32(0.125), tuning={"dense_tiles": 256})
    _, _, ref_lse = oracle.gt_attn_fwd(w_rp, w_ci, Q, K, V, np.float32(0.125), want_absagg=False)
    check_lse(got[1], ref_lse, 1e-5)  # the tile normaliser sums the fp32 weights


def check_grads_all(w, dO, got):
    """lse on every row, dQ on every row and dK, dV on every column, the oracle
    taken in row (column) blocks."""
    out, lse, dq, dk, dv = got
    rpt, cit = synth.transpose_csr(w.rowptr, w.colidx, w.N)
    for name, x in (("dQ", dq), ("dK", dk), ("dV", dv)):
        assert np.all(np.isfinite(x)), name
    errs = {"dQ": 0.0, "dK": 0.0, "dV": 0.0}
    for lo, hi in row_blocks(w.N, 2 * w.H * w.D):
        idx = np.arange(lo, hi, dtype=np.int64)
        _, _, ref_lse = oracle.gt_attn_fwd(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, rows=idx,
                                           want_absagg=False)
        check_lse(lse[lo:hi], ref_lse, 1e-5)
        rq, sq = oracle.gt_attn_bwd_dq(w.rowptr, w.colidx, w.Q, w.K, w.V, dO, w.scale, rows=idx)
        errs["dQ"] = max(errs["dQ"], gate_error(dq[lo:hi], rq, sq))
        rk, rv, sk, sv = oracle.gt_attn_bwd_dkv(w.rowptr, w.colidx, rpt, cit, w.Q, w.K, w.V, dO, w.scale,
                                                cols=idx)
        errs["dK"] = max(errs["dK"], gate_error(dk[lo:hi], rk, sk))
        errs["dV"] = max(errs["dV"], gate_error(dv[lo:hi], rv, sv))
    print("gate errors", {k: "%.3g" % v for k, v in errs.items()}, flush=True)
    for name, err in errs.items():
        assert err <= tol(w.dtype), "%s gate error %.3g" % (name, err)


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_full_config_all_rows_and_columns(idx):
    w = workload(idx)
    print("config", idx, w.name, "N", w.N, "E", w.E, flush=True)
    dO, _, _ = synth.features(37 if idx == 1 else 38, w.N, w.H, w.D, w.dtype)
    got = run_gpu_fwd_bwd(w.rowptr, w.colidx, w.Q, w.K, w.V, dO, w.scale)
    check_grads_all(w, dO, got)
