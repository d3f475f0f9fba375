"""Pins of the locality-study microbenchmark oracle (dot-aggr: per row, the
sum over its entries of <x_i, x_j>) and of the node relabelings the study
applies (synth.permute_graph, random_order, rcm_order)."""
import numpy as np
import pytest

import oracle
import synth


def graph(seed, N=120):
    return synth.ragged_graph(seed, N, max_deg=14, empty_frac=0.1, hubs={4: N - 1},
                              self_loops=True, dup_frac=0.2, shuffle=True)


@pytest.mark.parametrize("F", [1, 7, 32])
def test_dense_form(F):
    N = 90
    rowptr, colidx = graph(1, N)
    X = synth.normal(1, synth.STREAM_Q, (N, F), 1.0, "f32")
    C = np.zeros((N, N))
    for i in range(N):
        for j in colidx[rowptr[i]:rowptr[i + 1]]:
            C[i, j] += 1
    X64 = X.astype(np.float64)
    want = (C * (X64 @ X64.T)).sum(axis=1)
    s, a = oracle.dot_aggr(rowptr, colidx, X)
    np.testing.assert_allclose(s, want, rtol=1e-12, atol=1e-12)
    assert np.all(a >= np.abs(s) - 1e-12)


def test_ones_give_degree_times_width():
    N, F = 100, 16
    rowptr, colidx = graph(2, N)
    s, a = oracle.dot_aggr(rowptr, colidx, np.ones((N, F), np.float32))
    assert np.array_equal(s, np.diff(rowptr) * float(F)) and np.array_equal(a, s)


def test_one_hot_counts_same_class_entries():
    N, F = 80, 5
    rowptr, colidx = graph(3, N)
    cls = np.arange(N) % F
    X = np.eye(F, dtype=np.float32)[cls]
    s, _ = oracle.dot_aggr(rowptr, colidx, X)
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        assert s[i] == np.sum(cls[J] == cls[i])


@pytest.mark.parametrize("order", ["random", "rcm"])
def test_relabeling_permutes_the_result(order):
    N, F = 150, 8
    rowptr, colidx = graph(4, N)
    X = synth.normal(4, synth.STREAM_K, (N, F), 1.0, "f32")
    perm = synth.random_order(4, N) if order == "random" else synth.rcm_order(rowptr, colidx)
    rp2, ci2 = synth.permute_graph(rowptr, colidx, perm)
    synth.check_csr(rp2, ci2, N)
    assert np.array_equal(np.diff(rp2), np.diff(rowptr)[perm])
    s, _ = oracle.dot_aggr(rowptr, colidx, X)
    s2, _ = oracle.dot_aggr(rp2, ci2, np.ascontiguousarray(X[perm]))
    assert np.array_equal(s2, s[perm])  # same products, same order: bit-identical
    # the relabeled edges are the old edges under the new names
    old = {(int(perm[k]), int(perm[j])) for k in range(N) for j in ci2[rp2[k]:rp2[k + 1]]}
    ref = {(i, int(j)) for i in range(N) for j in colidx[rowptr[i]:rowptr[i + 1]]}
    assert old == ref


def test_rcm_reduces_bandwidth_of_a_shuffled_band():
    # a band graph (|i - j| <= 3) under a random relabeling has bandwidth ~N;
    # RCM must bring it back near the band
    N = 400
    rows = [[j for j in range(max(0, i - 3), min(N, i + 4))] for i in range(N)]
    rowptr = np.zeros(N + 1, np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    colidx = np.array([j for r in rows for j in r], np.int32)
    rp, ci = synth.permute_graph(rowptr, colidx, synth.random_order(5, N))
    rp2, ci2 = synth.permute_graph(rp, ci, synth.rcm_order(rp, ci))
    bw = lambda rp_, ci_: int(np.max(np.abs(np.repeat(np.arange(N), np.diff(rp_)) - ci_)))
    assert bw(rp, ci) > 200 and bw(rp2, ci2) <= 6
