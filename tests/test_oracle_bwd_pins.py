"""Pins of the float64 oracle backward (gradients of the graph-transformer
attention; the paper's backward recomputes the weights from the stored row
statistic, Appendix D.2).  The main pin is independent of the backward code:
central finite differences of the (separately pinned) oracle forward of the
loss sum(out * dO).  Closed forms and consistency checks complete it."""
import math

import numpy as np
import pytest

import oracle
import synth


def loss(rowptr, colidx, Q, K, V, dO, scale):
    out, _, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_absagg=False,
                                   want_lse=False)
    return float(np.sum(out * dO.astype(np.float64)))


def fd_grad(rowptr, colidx, Q, K, V, dO, scale, which, h=2.0 ** -9):
    arrs = [Q.copy(), K.copy(), V.copy()]
    x = arrs[which]
    g = np.zeros(x.shape)
    for idx in np.ndindex(*x.shape):
        x0 = x[idx]
        xp, xm = np.float32(x0 + h), np.float32(x0 - h)
        x[idx] = xp
        fp = loss(rowptr, colidx, *arrs, dO, scale)
        x[idx] = xm
        fm = loss(rowptr, colidx, *arrs, dO, scale)
        x[idx] = x0
        g[idx] = (fp - fm) / (float(xp) - float(xm))
    return g


def all_grads(rowptr, colidx, Q, K, V, dO, scale):
    N = Q.shape[0]
    rpt, cit = synth.transpose_csr(rowptr, colidx, N)
    dQ, sdQ = oracle.gt_attn_bwd_dq(rowptr, colidx, Q, K, V, dO, scale)
    dK, dV, sdK, sdV = oracle.gt_attn_bwd_dkv(rowptr, colidx, rpt, cit, Q, K, V, dO, scale)
    return dQ, dK, dV, sdQ, sdK, sdV


@pytest.mark.parametrize("seed", [0, 1])
def test_finite_differences(seed):
    N, H, D = 9, 2, 4
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=5, empty_frac=0.15, self_loops=True,
                                        dup_frac=0.25, shuffle=True)
    Q, K, V = synth.features(seed, N, H, D, "f32")
    dO, _, _ = synth.features(seed + 100, N, H, D, "f32")
    scale = np.float32(0.7)
    dQ, dK, dV, _, _, _ = all_grads(rowptr, colidx, Q, K, V, dO, scale)
    for which, g in ((0, dQ), (1, dK), (2, dV)):
        fd = fd_grad(rowptr, colidx, Q, K, V, dO, scale, which)
        np.testing.assert_allclose(g, fd, rtol=2e-5, atol=2e-6 * max(1.0, np.abs(fd).max()))


def test_zero_query_value_gradient():
    N, H, D = 30, 2, 8
    rowptr, colidx = synth.ragged_graph(2, N, max_deg=8, empty_frac=0.1, dup_frac=0.2)
    _, K, V = synth.features(2, N, H, D, "f32")
    dO, _, _ = synth.features(3, N, H, D, "f32")
    Q = np.zeros_like(K)
    _, _, dV, _, _, _ = all_grads(rowptr, colidx, Q, K, V, dO, np.float32(0.5))
    want = np.zeros((N, H, D))
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        for j in J:  # uniform weights 1/deg, once per entry
            want[j] += dO[i].astype(np.float64) / J.size
    np.testing.assert_allclose(dV, want, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_entry_rows(dtype):
    N, H, D = 25, 3, 8
    rowptr, colidx = synth.csr_from_degrees(4, N, np.ones(N, dtype=np.int64), self_loops=False)
    Q, K, V = synth.features(4, N, H, D, dtype)
    dO, _, _ = synth.features(5, N, H, D, dtype)
    dQ, dK, dV, _, _, _ = all_grads(rowptr, colidx, Q, K, V, dO, np.float32(0.3))
    assert np.all(dQ == 0) and np.all(dK == 0)
    f = (lambda a: a) if dtype == "f32" else synth.bf16_to_f32
    want = np.zeros((N, H, D))
    for i in range(N):
        want[colidx[i]] += f(dO[i]).astype(np.float64)
    np.testing.assert_array_equal(dV, want)


def test_subsets_match_full_and_scales_bound():
    N, H, D = 40, 2, 8
    rowptr, colidx = synth.ragged_graph(6, N, max_deg=12, hubs={3: 39}, dup_frac=0.1)
    Q, K, V = synth.features(6, N, H, D, "f32")
    dO, _, _ = synth.features(7, N, H, D, "f32")
    scale = np.float32(0.35)
    dQ, dK, dV, sdQ, sdK, sdV = all_grads(rowptr, colidx, Q, K, V, dO, scale)
    rows = np.array([3, 0, 39, 17], dtype=np.int64)
    sq, _ = oracle.gt_attn_bwd_dq(rowptr, colidx, Q, K, V, dO, scale, rows=rows)
    assert np.array_equal(sq, dQ[rows])
    rpt, cit = synth.transpose_csr(rowptr, colidx, N)
    sk, sv, _, _ = oracle.gt_attn_bwd_dkv(rowptr, colidx, rpt, cit, Q, K, V, dO, scale, cols=rows)
    assert np.array_equal(sk, dK[rows]) and np.array_equal(sv, dV[rows])
    for g, sg in ((dQ, sdQ), (dK, sdK), (dV, sdV)):
        assert np.all(sg >= np.abs(g) * (1 - 1e-12))
