"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded inputs.  Gate: max_e |x - r| / max(|r|, absagg) <= 1e-5 for
fp32 features and <= 2e-2 for bf16 features (fp32 accumulation, bf16 output)."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import (TOL_BF16, TOL_F32, fwd_gate_error_all_rows, gate_error,
                           load_worked_example, run_gpu, run_gpu_bare, workload)

pytestmark = pytest.mark.gpu

SHAPES = [(h, d) for h in (1, 2, 4, 8) for d in (32, 64, 128, 256)]
BF16_ONLY = [(1, 512), (2, 512), (4, 512)]  # a 512-element fp32 head exceeds 64 lanes of 16 B
CASES = [(h, d, t) for (h, d) in SHAPES for t in ("f32", "bf16")] + [(h, d, "bf16") for (h, d) in BF16_ONLY]
FORCED_SPLIT = {"light_max_deg": 2, "heavy_min_deg": 6, "chunk_edges": 64, "grid_blocks": 0}


def tol(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


def check(w_or_arrays, dtype, tuning=None, rows=None):
    rowptr, colidx, Q, K, V, scale = w_or_arrays
    got = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tuning)
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, rows=rows, want_lse=False)
    if rows is not None:
        got = got[rows]
    err = gate_error(got, ref, absagg)
    assert np.all(np.isfinite(got))
    assert err <= tol(dtype), "gate error %.3g > %.3g" % (err, tol(dtype))
    return err, got, ref


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_worked_example(dtype):
    ex = load_worked_example()
    # zero-pad the head dimension 2 -> 32 (a compiled shape): dots are unchanged
    # and the padded output columns must come out as exactly 0
    pad = lambda x: np.ascontiguousarray(np.pad(x, ((0, 0), (0, 0), (0, 30))))
    Q, K, V = (pad(ex[k]) for k in ("Q", "K", "V"))
    if dtype == "bf16":  # small integers: exact in bf16
        Q, K, V = ((x.view(np.uint32) >> 16).astype(np.uint16) for x in (Q, K, V))
    got = run_gpu(ex["rowptr"], ex["colidx"], Q, K, V, ex["scale"])
    # fp32 evaluation: ~1e-7; bf16 output adds its round-to-nearest step,
    # at most half an ulp = 2^-8 relative
    bound = 1e-6 if dtype == "f32" else 2.0 ** -8 + 1e-6
    assert gate_error(got[:, :, :2], ex["OUT"], ex["ABS"]) <= bound
    assert np.all(got[:, :, 2:] == 0)
    assert np.array_equal(got[1, :, :2], ex["V"][1])  # single-entry row is exact


@pytest.mark.parametrize("split", [False, True], ids=["default", "forced_split"])
@pytest.mark.parametrize("H,D,dtype", CASES)
def test_ragged_small(H, D, dtype, split):
    N = 300
    rowptr, colidx = synth.ragged_graph(H * 1000 + D, N, max_deg=24, empty_frac=0.1,
                                        hubs={7: 299, 100: 150, 299: 70}, self_loops=True,
                                        dup_frac=0.05, shuffle=True)
    Q, K, V = synth.features(H * 1000 + D, N, H, D, dtype)
    check((rowptr, colidx, Q, K, V, np.float32(1 / math.sqrt(D))), dtype,
          tuning=FORCED_SPLIT if split else None)


BF16_CASES = [(h, d) for (h, d, t) in CASES if t == "bf16"]


@pytest.mark.parametrize("split", [False, True], ids=["default", "forced_split"])
@pytest.mark.parametrize("H,D", BF16_CASES)
def test_ragged_small_weight_precision(H, D, split):
    """bf16 features: by default the softmax weights stay fp32 for P*V, so the
    error left is the bf16 rounding of the output (unit roundoff 2^-8) plus
    fp32 arithmetic, well inside the bf16 gate; the bf16_weights option rounds
    each weight to bf16 as well, which adds up to 2^-8 of the absolute sum."""
    N = 300
    rowptr, colidx = synth.ragged_graph(H * 1000 + D + 5, N, max_deg=24, empty_frac=0.1,
                                        hubs={7: 299, 100: 150, 299: 70}, self_loops=True,
                                        dup_frac=0.05, shuffle=True)
    Q, K, V = synth.features(H * 1000 + D + 5, N, H, D, "bf16")
    scale = np.float32(1 / math.sqrt(D))
    base = FORCED_SPLIT if split else {}
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
    got = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=base or None)
    assert gate_error(got, ref, absagg) <= 2.0 ** -8 + 1e-5
    rounded = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=dict(base, bf16_weights=1))
    assert gate_error(rounded, ref, absagg) <= 2.0 ** -8 + 2.0 ** -8 + 1e-5


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4, 5])
def test_full_config_all_rows(idx):
    """Every row of each full-size workload, through the contract entry point
    of its feature dtype (gt_attn_fwd for fp32, gt_attn_fwd_bf16 for bf16) in
    the launch configuration the benchmark times."""
    w = workload(idx)
    print("config", idx, w.name, "N", w.N, "E", w.E, flush=True)
    got = run_gpu_bare(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale)
    assert np.all(np.isfinite(got))
    err = fwd_gate_error_all_rows(w, got)
    print("gate error %.3g" % err, flush=True)
    assert err <= tol(w.dtype), "gate error %.3g > %.3g" % (err, tol(w.dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bare_entry_equals_generic_entry(dtype):
    """gt_attn_fwd / gt_attn_fwd_bf16 and gt_attn_fwd_ex without tuning are the
    same computation: bit-identical outputs."""
    N, H, D = 3000, 4, 32
    rowptr, colidx = synth.ragged_graph(77, N, max_deg=70, empty_frac=0.05,
                                        hubs={5: 2999, 17: 1500, 800: 300}, self_loops=True)
    Q, K, V = synth.features(77, N, H, D, dtype)
    a = run_gpu_bare(rowptr, colidx, Q, K, V, np.float32(0.2))
    b = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2))
    assert np.array_equal(a, b)
