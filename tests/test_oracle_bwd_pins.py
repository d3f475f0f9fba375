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


def dense_grads(rowptr, colidx, Qf, Kf, Vf, dOf, scale):
    """Gradients of sum(out * dO) from the dense masked form by matrix calculus,
    written independently of the oracle: per head, P = row-normalised
    C * exp(S) with S = scale Q K^T and C the entry multiplicities;
    dV = P^T dO, dS = P * (dO V^T - rowsum(P * dO V^T)), dQ = scale dS K,
    dK = scale dS^T Q."""
    N, H, D = Qf.shape
    C = np.zeros((N, N))
    for i in range(N):
        for e in range(rowptr[i], rowptr[i + 1]):
            C[i, colidx[e]] += 1.0
    dQ, dK, dV = np.zeros((N, H, D)), np.zeros((N, H, D)), np.zeros((N, H, D))
    for h in range(H):
        q, k, v, do = (x[:, h, :].astype(np.float64) for x in (Qf, Kf, Vf, dOf))
        S = float(scale) * (q @ k.T)
        S = np.where(C > 0, S, -np.inf)
        mx = S.max(axis=1, keepdims=True)
        W = np.where(C > 0, C * np.exp(S - np.where(np.isfinite(mx), mx, 0.0)), 0.0)
        Z = W.sum(axis=1, keepdims=True)
        P = W / np.where(Z > 0, Z, 1.0)
        dV[:, h, :] = P.T @ do
        dP = do @ v.T
        dS = P * (dP - (P * dP).sum(axis=1, keepdims=True))
        dQ[:, h, :] = float(scale) * (dS @ k)
        dK[:, h, :] = float(scale) * (dS.T @ q)
    return dQ, dK, dV


@pytest.mark.parametrize("case", range(30))
def test_dense_gradients_on_random_small_graphs(case):
    """Thirty seeded random cases (1..30 rows, any H and D, empty rows, repeats,
    self-loops, unsorted rows, fp32 and bf16) against the dense gradients."""
    rng = np.random.default_rng(10_000 + case)
    N = int(rng.integers(1, 31))
    H, D = int(rng.integers(1, 4)), int(rng.integers(1, 13))
    dtype = "f32" if case % 2 == 0 else "bf16"
    rowptr, colidx = synth.ragged_graph(10_100 + case, N, max_deg=int(rng.integers(0, 10)),
                                        empty_frac=float(rng.choice([0.0, 0.3])), self_loops=bool(case % 3 == 0),
                                        dup_frac=float(rng.choice([0.0, 0.3])), shuffle=bool(case % 4 == 1))
    Q, K, V = synth.features(10_200 + case, N, H, D, dtype)
    dO, _, _ = synth.features(10_300 + case, N, H, D, dtype)
    scale = np.float32(rng.choice([1 / math.sqrt(D), -0.5, 2.0]))
    dQ, dK, dV, _, _, _ = all_grads(rowptr, colidx, Q, K, V, dO, scale)
    f = (lambda a: a) if dtype == "f32" else (lambda b: (np.asarray(b).astype(np.uint32) << 16).view(np.float32))
    rQ, rK, rV = dense_grads(rowptr, colidx, f(Q), f(K), f(V), f(dO), scale)
    for got, want in ((dQ, rQ), (dK, rK), (dV, rV)):
        np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-10 * max(1.0, np.abs(want).max()))
