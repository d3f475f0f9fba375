"""Non-finite inputs.  A row's output is a function of its own query and of
the keys and values of the sources its CSR entries name (Section 2.2, the
attention family), so Inf or NaN in the rows of other nodes must not reach it.
The dense-tile path multiplies whole 64-column windows, where a weight of 0
times such a value would be NaN: a window whose value tile holds one is
streamed entry by entry instead.  Where a row does name such a source, its
output is non-finite exactly where the float64 oracle's is.

Graphs: 64-id block models (every window dense enough to tile) with a partial
last window, one hub row (split into chunks and merged) and one medium row."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import TOL_BF16, TOL_F32, gate_error, run_gpu
from tests.test_gpu_gatv2 import attention_vector, run_gpu_gatv2

pytestmark = pytest.mark.gpu

CSR_ONLY = {"dense_tiles": -1}
N = 64 * 10 + 21
HUB, MEDIUM = 100, 300
# node -> (K row, V row): "nan", "+inf", "-inf" or None (finite)
BAD = {64 + 5: ("nan", None),             # window 1: a key only, so its tile still runs
       64 * 3 + 17: (None, "+inf"),
       64 * 5 + 63: ("-inf", "nan"),
       64 * 6: (None, "-inf"),
       N - 1: (None, "nan")}              # the partial last window
BAD_V_WINDOWS = sorted({i // 64 for i, (_, v) in BAD.items() if v})
CASES = [("bf16", 2, 64), ("bf16", 4, 32), ("bf16", 1, 128), ("bf16", 8, 64), ("f32", 4, 32)]
BF16_BITS = {"nan": 0x7FC0, "+inf": 0x7F80, "-inf": 0xFF80}
F32_VALUES = {"nan": np.nan, "+inf": np.inf, "-inf": -np.inf}


def rows_of(seed, referenced):
    rp, ci = synth.sbm_graph(seed, N, 64, 4)
    rows = [list(ci[rp[i]:rp[i + 1]]) for i in range(N)]
    u = synth.uniform01(seed, synth.STREAM_EXTRA + 5, 4000)
    rows[HUB] = sorted(set(int(x) for x in np.floor(u[:3000] * N)))
    rows[MEDIUM] = sorted(set(int(x) for x in np.floor(u[3000:3100] * N)))
    if not referenced:
        rows = [[j for j in r if j not in BAD] for r in rows]
    else:
        # every bad node is named by some row (the SBM rows of its window do)
        assert all(any(b in r for r in rows) for b in BAD)
    rowptr = np.zeros(N + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    return rowptr, np.concatenate([np.asarray(r, dtype=np.int32) for r in rows])


def poison(X, which, dtype):
    X = X.copy()
    for i, kinds in BAD.items():
        kind = kinds[which]
        if kind:
            X[i] = BF16_BITS[kind] if dtype == "bf16" else F32_VALUES[kind]
    return X


def inputs(seed, referenced, dtype, H, D):
    rowptr, colidx = rows_of(seed, referenced)
    Q, K, V = synth.features(seed, N, H, D, dtype)
    return rowptr, colidx, Q, poison(K, 0, dtype), poison(V, 1, dtype)


def tile_shape(dtype, H, D):
    return dtype == "bf16" and H * D <= 128 and D % 32 == 0


@pytest.mark.parametrize("dtype,H,D", CASES)
def test_unreferenced_non_finite_rows_do_not_leak(dtype, H, D):
    seed = 9100 + H * 10 + D
    rowptr, colidx, Q, K, V = inputs(seed, False, dtype, H, D)
    scale = np.float32(1 / math.sqrt(D))
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
    assert np.all(np.isfinite(ref))
    for tuning in (None, {"chunk_edges": 64}):
        got = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tuning)
        assert np.all(np.isfinite(got)), "non-finite rows: %s" % np.unique(np.nonzero(~np.isfinite(got))[0])[:20]
        assert gate_error(got, ref, absagg) <= tol
    if tile_shape(dtype, H, D):
        # windows with a non-finite value were streamed (bit for bit the CSR
        # path's output); the others, the key-only window 1 included, tiled
        csr = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=CSR_ONLY)
        for w in range(N // 64 + 1):
            rows = slice(64 * w, min(64 * w + 64, N))
            if w in BAD_V_WINDOWS:
                assert np.array_equal(got[rows], csr[rows]), "window %d" % w
            elif w in (0, 1, 2):
                assert not np.array_equal(got[rows], csr[rows]), "window %d" % w


@pytest.mark.parametrize("dtype,H,D", CASES)
def test_referenced_non_finite_values_match_the_oracle_pattern(dtype, H, D):
    seed = 9200 + H * 10 + D
    rowptr, colidx, Q, K, V = inputs(seed, True, dtype, H, D)
    scale = np.float32(1 / math.sqrt(D))
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
    fin = np.isfinite(ref)
    assert not np.all(fin) and np.any(fin)
    for tuning in (None, {"chunk_edges": 64}, CSR_ONLY):
        got = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tuning)
        assert np.array_equal(np.isfinite(got), fin)
        assert gate_error(got[fin], ref[fin], absagg[fin]) <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gatv2_unreferenced_non_finite_rows_do_not_leak(dtype):
    H, D = 4, 32
    seed = 9300
    rowptr, colidx = rows_of(seed, False)
    Lf, Rf, _ = synth.features(seed, N, H, D, dtype)
    Rf = poison(poison(Rf, 0, dtype), 1, dtype)
    att = attention_vector(seed, H, D)
    ref, absagg, _ = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, 0.2)
    for tuning in (None, {"chunk_edges": 64}):
        got, _ = run_gpu_gatv2(rowptr, colidx, Lf, Rf, att, 0.2, tuning=tuning)
        assert np.all(np.isfinite(got))
        assert gate_error(got, ref, absagg) <= (TOL_F32 if dtype == "f32" else TOL_BF16)
