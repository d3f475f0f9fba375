"""Randomised parity: small graphs of several kinds (ragged rows with hubs,
repeated and unsorted entries, empty rows; 64-id block models that tile)
crossed with random shapes, dtypes and partition settings (light bound, front
threshold, chunk length, grid size, dense-tile threshold, weight precision),
each against the float64 oracle: the graph-transformer forward and the GATv2
forward (output and lse, and a second call bit for bit), the segment min/max
(bit-exact) and the backward (lse and the three gradients).  The cases are drawn from fixed seeds, so every run checks the
same ones."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.helpers import TOL_BF16, TOL_F32, gate_error, to_device, to_host_f32
from tests.test_gpu_gatv2 import attention_vector, run_gpu_gatv2
from tests.test_gpu_reduce import features as reduce_features, oracle_bits, run_gpu_reduce

pytestmark = pytest.mark.gpu

SHAPES_F32 = [(h, d) for h in (1, 2, 4, 8) for d in (32, 64, 128, 256)]
SHAPES_BF16 = SHAPES_F32 + [(1, 512), (2, 512), (4, 512)]
TILE_SHAPES = [(1, 32), (1, 64), (1, 128), (2, 32), (2, 64), (4, 32)]
N_CASES = 160


def draw_case(seed):
    rng = np.random.default_rng(1000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    dtype = pick(["f32", "bf16"])
    kind = pick(["ragged", "ragged", "blocks"])
    if kind == "blocks" and dtype == "bf16":
        H, D = pick(TILE_SHAPES)
    else:
        H, D = pick(SHAPES_F32 if dtype == "f32" else SHAPES_BF16)
    N = int(rng.integers(1, 3000))
    if kind == "blocks":
        N = max(N, 130)
        graph = dict(kind=kind, N=N, n_out=int(rng.integers(0, 9)))
    else:
        n_hubs = int(rng.integers(0, 4)) if N >= 2 else 0
        hubs = {int(r): int(rng.integers(1, N)) for r in rng.integers(0, N, size=n_hubs)}
        graph = dict(kind=kind, N=N, max_deg=int(pick([1, 3, 20, 90, 300])),
                     empty_frac=float(pick([0.0, 0.1, 0.5])), hubs=hubs,
                     self_loops=bool(rng.integers(2)), dup_frac=float(pick([0.0, 0.05, 0.3])),
                     shuffle=bool(rng.integers(2)))
    tuning = dict(light_max_deg=int(pick([0, 0, 1, 2, 7, 16, 64, 100])),
                  heavy_min_deg=int(pick([0, 0, 2, 9, 64, 300])),
                  chunk_edges=int(pick([0, 0, 1, 64, 100, 1000])),
                  grid_blocks=int(pick([0, 0, 1, 8, 13, 1000])),
                  dense_tiles=int(pick([0, 0, -1, 1, 50, 256])),
                  bf16_weights=int(pick([0, 0, 1])))
    return dict(seed=seed, dtype=dtype, H=H, D=D, graph=graph, tuning=tuning,
                want_lse=bool(rng.integers(2)), std=float(pick([0.5, 1.0])))


def make_graph(seed, g):
    if g["kind"] == "blocks":
        N = g["N"]
        n_out = min(g["n_out"], N - 64)
        return synth.sbm_graph(seed, N, 64, n_out)
    return synth.ragged_graph(seed, g["N"], g["max_deg"], empty_frac=g["empty_frac"], hubs=g["hubs"],
                              self_loops=g["self_loops"], dup_frac=g["dup_frac"], shuffle=g["shuffle"])


def run(rowptr, colidx, Q, K, V, scale, tuning, want_lse):
    import paper_2605_31500_amd as gt
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dev[2])
    lse = torch.empty(Q.shape[:2], dtype=torch.float32, device=out.device) if want_lse else None
    gt.gt_attn_fwd_ex(*dev, out, scale, tuning=tuning, lse=lse)
    torch.cuda.synchronize()
    return to_host_f32(out), (lse.cpu().numpy() if want_lse else None)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_case(seed):
    c = draw_case(seed)
    rowptr, colidx = make_graph(2000 + seed, c["graph"])
    N = rowptr.size - 1
    Q, K, V = synth.features(3000 + seed, N, c["H"], c["D"], c["dtype"], std=c["std"])
    scale = np.float32(1 / math.sqrt(c["D"]))
    got, lse = run(rowptr, colidx, Q, K, V, scale, c["tuning"], c["want_lse"])
    ref, absagg, ref_lse = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale)
    tol = TOL_F32 if c["dtype"] == "f32" else TOL_BF16
    assert np.all(np.isfinite(got)), c
    err = gate_error(got, ref, absagg)
    assert err <= tol, "gate error %.3g > %.3g for %s" % (err, tol, c)
    if c["want_lse"]:
        fin = np.isfinite(ref_lse)
        assert np.array_equal(np.isneginf(lse), ~fin), c
        assert np.all(np.abs(lse[fin] - ref_lse[fin]) <= 1e-5 * np.maximum(1.0, np.abs(ref_lse[fin]))), c
    again, _ = run(rowptr, colidx, Q, K, V, scale, c["tuning"], False)
    assert np.array_equal(got, again), c


def check_lse(lse, ref_lse, c):
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isneginf(lse), ~fin), c
    assert np.all(np.abs(lse[fin] - ref_lse[fin]) <= 1e-5 * np.maximum(1.0, np.abs(ref_lse[fin]))), c


@pytest.mark.parametrize("seed", range(N_CASES // 2))
def test_random_case_gatv2(seed):
    c = draw_case(10_000 + seed)
    rowptr, colidx = make_graph(4000 + seed, c["graph"])
    N = rowptr.size - 1
    Lf, Rf, _ = synth.features(5000 + seed, N, c["H"], c["D"], c["dtype"], std=c["std"])
    att = attention_vector(5000 + seed, c["H"], c["D"])
    slope = float([0.2, 0.0, 1.0, -0.5][seed % 4])
    got, lse = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, slope, tuning=c["tuning"])
    ref, absagg, ref_lse = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, slope)
    tol = TOL_F32 if c["dtype"] == "f32" else TOL_BF16
    assert np.all(np.isfinite(got)), c
    err = gate_error(got, ref, absagg)
    assert err <= tol, "gate error %.3g > %.3g for %s" % (err, tol, c)
    check_lse(lse, ref_lse, c)
    again, _ = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, slope, tuning=c["tuning"])
    assert np.array_equal(got, again), c


@pytest.mark.parametrize("seed", range(N_CASES // 2))
def test_random_case_segment_reduce(seed):
    c = draw_case(20_000 + seed)
    rowptr, colidx = make_graph(6000 + seed, c["graph"])
    N = rowptr.size - 1
    F = c["H"] * c["D"]
    if c["dtype"] == "f32" and F > 1024:
        F = 1024
    X = reduce_features(7000 + seed, N, F, c["dtype"])
    op = "min" if seed % 2 == 0 else "max"
    tuning = {k: v for k, v in c["tuning"].items() if k in ("light_max_deg", "heavy_min_deg", "chunk_edges",
                                                             "grid_blocks")}
    bits, arg = run_gpu_reduce(rowptr, colidx, X, op, tuning=tuning)
    ref, ref_arg = oracle.segment_reduce(rowptr, colidx, X, op)
    assert np.array_equal(bits, oracle_bits(ref, c["dtype"])), c
    assert np.array_equal(arg, ref_arg), c


@pytest.mark.parametrize("seed", range(N_CASES // 4))
def test_random_case_backward(seed):
    """The backward on the same random graphs and shapes (its partition uses
    the defaults; the forward that produces out and lse takes the case's
    settings), each gradient against the oracle's under the gate."""
    from tests.helpers import run_gpu_fwd_bwd
    from tests.test_gpu_bwd import check_grads, check_lse
    c = draw_case(30_000 + seed)
    rowptr, colidx = make_graph(11_000 + seed, c["graph"])
    N = rowptr.size - 1
    Q, K, V = synth.features(12_000 + seed, N, c["H"], c["D"], c["dtype"], std=c["std"])
    dO, _, _ = synth.features(13_000 + seed, N, c["H"], c["D"], c["dtype"])
    scale = np.float32(1 / math.sqrt(c["D"]))
    got = run_gpu_fwd_bwd(rowptr, colidx, Q, K, V, dO, scale, tuning=c["tuning"])
    _, _, ref_lse = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale)
    check_lse(got[1], ref_lse, 1e-5)
    check_grads(rowptr, colidx, Q, K, V, dO, scale, got, c["dtype"])
