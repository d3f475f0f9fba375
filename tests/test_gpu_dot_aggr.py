"""GPU parity of the locality-study microbenchmark (dot-aggr, both mappings,
scalar and 16-byte loads) against the float64 oracle, through the C ABI.

Bound, derived from the arithmetic: each lane sums its products with fp32
FMAs in sequence, then the wave adds the 64 lane sums in a 6-level tree, so
the error is at most (n + 7) u sum|x_i,f x_j,f| with u = 2^-24 and n the
longest per-lane chain: deg * max(EPL, F/64) terms (feature-parallel, EPL =
floats per load) or ceil(deg/64) * F terms (neighbour-parallel)."""
import numpy as np
import pytest

import oracle
import synth
from tests.helpers import to_device, workload

pytestmark = pytest.mark.gpu

VARIANTS = [(m, vb) for m in ("feature", "neighbor") for vb in (4, 16)]
FS = [32, 64, 128, 256, 512]


def run_gpu_dot(rowptr, colidx, X, mapping, load_bytes):
    import torch
    import paper_2605_31500_amd as gt
    rp, ci, x = (to_device(a) for a in (rowptr, colidx, X))
    out = torch.empty(x.shape[0], dtype=torch.float32, device=x.device)
    gt.gt_dot_aggr(rp, ci, x, out, mapping=mapping, load_bytes=load_bytes)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def bound(deg, F, mapping, load_bytes, absval):
    epl = load_bytes // 4
    if mapping == "feature":
        n = deg * max(epl, F // 64)
    else:
        n = np.ceil(deg / 64.0) * F
    return 1.05 * (n + 7) * 2.0 ** -24 * absval + 1e-30


def check(rowptr, colidx, X, mapping, load_bytes, rows=None):
    got = run_gpu_dot(rowptr, colidx, X, mapping, load_bytes)
    ref, absval = oracle.dot_aggr(rowptr, colidx, X, rows=rows)
    deg = np.diff(rowptr)
    if rows is not None:
        got, deg = got[rows], deg[rows]
    err = np.abs(got - ref)
    lim = bound(deg, X.shape[1], mapping, load_bytes, absval)
    assert np.all(err <= lim), "worst err/bound %.3g" % float(np.max(err / lim))
    assert np.all(got[deg == 0] == 0)
    return float(np.max(err / np.maximum(absval, 1e-30)))


@pytest.mark.parametrize("F", FS)
@pytest.mark.parametrize("mapping,load_bytes", VARIANTS)
def test_dot_aggr_ragged(mapping, load_bytes, F):
    N = 700
    rowptr, colidx = synth.ragged_graph(30 + F, N, max_deg=90, empty_frac=0.1,
                                        hubs={3: 699, 4: 400, 5: 130}, self_loops=True,
                                        dup_frac=0.1, shuffle=True)
    X = synth.normal(30 + F, synth.STREAM_Q, (N, F), 1.0, "f32")
    check(rowptr, colidx, X, mapping, load_bytes)


@pytest.mark.parametrize("mapping,load_bytes", VARIANTS)
def test_dot_aggr_integer_inputs_are_exact(mapping, load_bytes):
    # small integers: every partial sum is an exact integer below 2^24
    N, F = 600, 128
    rowptr, colidx = synth.ragged_graph(40, N, max_deg=70, empty_frac=0.1, hubs={1: 599})
    u = synth.uniform01(40, synth.STREAM_V, N * F).reshape(N, F)
    X = (np.floor(u * 5) - 2).astype(np.float32)
    got = run_gpu_dot(rowptr, colidx, X, mapping, load_bytes)
    ref, _ = oracle.dot_aggr(rowptr, colidx, X)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("order", ["original", "random", "rcm"])
@pytest.mark.parametrize("mapping,load_bytes", VARIANTS)
def test_dot_aggr_study_graph(mapping, load_bytes, order):
    # the power-law bench graph at F = 128 under the study's three orders
    w = workload(1)
    X = synth.normal(1, synth.STREAM_Q, (w.N, 128), 1.0, "f32")
    rowptr, colidx = w.rowptr, w.colidx
    if order != "original":
        perm = synth.random_order(1, w.N) if order == "random" else synth.rcm_order(rowptr, colidx)
        rowptr, colidx = synth.permute_graph(rowptr, colidx, perm)
        X = np.ascontiguousarray(X[perm])
    check(rowptr, colidx, X, mapping, load_bytes)
