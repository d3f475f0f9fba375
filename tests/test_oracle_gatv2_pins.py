"""Pins of the float64 GATv2 oracle (paper Section 2.2: e_ij = a^T
LeakyReLU(W_l h_i + W_r h_j), values W_r h_j; Appendix D.2, fused GATv2
forward).  A dense masked evaluation written independently, closed forms
(zero attention vector, single entries, slope 1 where the row term cancels)
and invariants."""
import numpy as np
import pytest

import oracle
import synth
from tests.helpers import bf16_bits_to_f32


def lrelu(x, slope):
    return np.where(x > 0, x, slope * x)


def dense_gatv2(rowptr, colidx, Lf, Rf, att, slope):
    N, H, D = Lf.shape
    C = np.zeros((N, N))
    for i in range(N):
        for e in range(rowptr[i], rowptr[i + 1]):
            C[i, colidx[e]] += 1.0
    out = np.zeros((N, H, D))
    for h in range(H):
        L = Lf[:, h, :].astype(np.float64)
        R = Rf[:, h, :].astype(np.float64)
        S = np.einsum("ijd,d->ij", lrelu(L[:, None, :] + R[None, :, :], float(slope)),
                      att[h].astype(np.float64))
        S = np.where(C > 0, S, -np.inf)
        mx = S.max(axis=1, keepdims=True)
        W = np.where(C > 0, C * np.exp(S - np.where(np.isfinite(mx), mx, 0.0)), 0.0)
        Z = W.sum(axis=1, keepdims=True)
        out[:, h, :] = np.where(Z > 0, (W @ R) / np.where(Z > 0, Z, 1), 0)
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", [0, 1])
def test_dense_masked(dtype, seed):
    N, H, D = 33, 2, 8
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=9, empty_frac=0.15, hubs={4: 32},
                                        self_loops=True, dup_frac=0.2, shuffle=True)
    Lf, Rf, _ = synth.features(seed, N, H, D, dtype)
    att = synth.normal(seed, synth.STREAM_EXTRA + 9, (H, D), 1.0, "f32")
    out, absagg, lse = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, 0.2)
    f = (lambda a: a) if dtype == "f32" else bf16_bits_to_f32
    ref = dense_gatv2(rowptr, colidx, f(Lf), f(Rf), att, np.float32(0.2))
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    assert np.all(absagg >= np.abs(out) - 1e-12)


def test_zero_attention_vector_gives_mean():
    N, H, D = 40, 2, 8
    rowptr, colidx = synth.ragged_graph(2, N, max_deg=10, empty_frac=0.1, dup_frac=0.1)
    Lf, Rf, _ = synth.features(2, N, H, D, "f32")
    out, _, _ = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, np.zeros((H, D), np.float32), 0.2)
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        want = Rf[J].astype(np.float64).mean(axis=0) if J.size else np.zeros((H, D))
        np.testing.assert_allclose(out[i], want, rtol=1e-13, atol=1e-14)


def test_single_entry_rows_exact():
    N, H, D = 30, 4, 8
    rowptr, colidx = synth.csr_from_degrees(3, N, np.ones(N, dtype=np.int64), self_loops=False)
    Lf, Rf, _ = synth.features(3, N, H, D, "f32")
    att = synth.normal(3, synth.STREAM_EXTRA + 9, (H, D), 1.0, "f32")
    out, _, lse = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, 0.2)
    assert np.array_equal(out, Rf[colidx].astype(np.float64))


def test_slope_one_row_term_cancels():
    """With slope 1 the score is a.l_i + a.r_j; the row term cancels in the
    softmax, so the weights are proportional to exp(a.r_j)."""
    N, H, D = 35, 2, 8
    rowptr, colidx = synth.ragged_graph(4, N, max_deg=8, empty_frac=0.1, self_loops=True)
    Lf, Rf, _ = synth.features(4, N, H, D, "f32")
    att = synth.normal(4, synth.STREAM_EXTRA + 9, (H, D), 1.0, "f32")
    out, _, _ = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, 1.0)
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        for h in range(H):
            if J.size == 0:
                assert np.all(out[i, h] == 0)
                continue
            z = Rf[J, h, :].astype(np.float64) @ att[h].astype(np.float64)
            w = np.exp(z - z.max())
            want = (w[:, None] * Rf[J, h, :].astype(np.float64)).sum(0) / w.sum()
            np.testing.assert_allclose(out[i, h], want, rtol=1e-12, atol=1e-13)


def test_permutation_invariance():
    N, H, D = 50, 2, 8
    rowptr, colidx = synth.ragged_graph(5, N, max_deg=20, self_loops=True, dup_frac=0.1)
    _, shuffled = synth.ragged_graph(5, N, max_deg=20, self_loops=True, dup_frac=0.1, shuffle=True)
    Lf, Rf, _ = synth.features(5, N, H, D, "f32")
    att = synth.normal(5, synth.STREAM_EXTRA + 9, (H, D), 1.0, "f32")
    a, _, la = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, 0.2)
    b, _, lb = oracle.gatv2_fwd(rowptr, shuffled, Lf, Rf, att, 0.2)
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(la, lb, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("case", range(40))
def test_dense_form_on_random_small_graphs(case):
    """Forty seeded random cases (1..30 rows, any H and D, empty rows, repeats,
    self-loops, unsorted rows, slopes from -1 to 3, attention vectors of
    several scales) against the dense masked form."""
    rng = np.random.default_rng(8000 + case)
    N = int(rng.integers(1, 31))
    H, D = int(rng.integers(1, 4)), int(rng.integers(1, 13))
    dtype = "f32" if case % 2 == 0 else "bf16"
    rowptr, colidx = synth.ragged_graph(8100 + case, N, max_deg=int(rng.integers(0, 10)),
                                        empty_frac=float(rng.choice([0.0, 0.3])), self_loops=bool(case % 3 == 0),
                                        dup_frac=float(rng.choice([0.0, 0.3])), shuffle=bool(case % 4 == 1))
    Lf, Rf, _ = synth.features(8200 + case, N, H, D, dtype)
    att = synth.normal(8300 + case, synth.STREAM_EXTRA + 9, (H, D), float(rng.choice([0.3, 1.0, 3.0])), "f32")
    slope = float(rng.choice([0.2, 0.0, 1.0, -1.0, 3.0]))
    out, absagg, _ = oracle.gatv2_fwd(rowptr, colidx, Lf, Rf, att, slope)
    f = (lambda a: a) if dtype == "f32" else bf16_bits_to_f32
    ref = dense_gatv2(rowptr, colidx, f(Lf), f(Rf), att, np.float32(slope))
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-10)
    assert np.all(absagg >= np.abs(out) - 1e-12)
