"""Pins of the float64 oracle to facts fixed by the paper and by mathematics.

The paper prints no numeric worked example for the attention operator, so
every pin here is constructed: a hand-derived example with exact answers, the
dense masked softmax(Q K^T) V textbook form, closed forms (zero query gives the
neighbour mean, one entry returns its value, two entries follow the logistic
function), invariants (order of entries, constant V, linearity in V,
independent heads) and a stability limit.  Definition followed: Section 2.2,
attention-based family (iii), graph-transformer logits q_i . k_j / sqrt(D).
"""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import bf16_bits_to_f32, load_worked_example


def run(rowptr, colidx, Q, K, V, scale, rows=None):
    return oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, rows=rows)


def dense_reference(rowptr, colidx, Qf, Kf, Vf, scale):
    """softmax over the masked dense score matrix, written independently:
    C[i,j] counts how often j appears in row i; out = (C * exp(S - rowmax)) V / rowsum."""
    N, H, D = Qf.shape
    C = np.zeros((N, N))
    for i in range(N):
        for e in range(rowptr[i], rowptr[i + 1]):
            C[i, colidx[e]] += 1.0
    out = np.zeros((N, H, D))
    for h in range(H):
        S = float(scale) * (Qf[:, h, :].astype(np.float64) @ Kf[:, h, :].astype(np.float64).T)
        S = np.where(C > 0, S, -np.inf)
        mx = S.max(axis=1, keepdims=True)
        W = np.where(C > 0, C * np.exp(S - np.where(np.isfinite(mx), mx, 0.0)), 0.0)
        Z = W.sum(axis=1, keepdims=True)
        out[:, h, :] = np.where(Z > 0, (W @ Vf[:, h, :].astype(np.float64)) / np.where(Z > 0, Z, 1), 0)
    return out


def test_worked_example_by_hand():
    ex = load_worked_example()
    out, absagg, lse = run(ex["rowptr"], ex["colidx"], ex["Q"], ex["K"], ex["V"], ex["scale"])
    np.testing.assert_allclose(out, ex["OUT"], rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(absagg, ex["ABS"], rtol=1e-6, atol=1e-7)
    fin = np.isfinite(ex["LSE"])
    np.testing.assert_allclose(lse[fin], ex["LSE"][fin], rtol=1e-6, atol=1e-7)
    assert np.all(np.isneginf(lse[~fin]))
    # the single-entry row returns its neighbour's value bit for bit
    assert np.array_equal(out[1], ex["V"][1].astype(np.float64))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dense_masked_softmax(dtype, seed):
    N, H, D = 41, 3, 8
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=9, empty_frac=0.15, hubs={5: 40},
                                        self_loops=True, dup_frac=0.2, shuffle=True)
    Q, K, V = synth.features(seed, N, H, D, dtype)
    out, absagg, lse = run(rowptr, colidx, Q, K, V, np.float32(1 / math.sqrt(D)))
    f = (lambda a: a) if dtype == "f32" else bf16_bits_to_f32
    ref = dense_reference(rowptr, colidx, f(Q), f(K), f(V), np.float32(1 / math.sqrt(D)))
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_dense_catches_transposed_roles():
    """Q is the destination side, K the gathered side: swapping them must differ."""
    N, H, D = 20, 1, 8
    rowptr, colidx = synth.ragged_graph(3, N, max_deg=6, self_loops=True)
    Q, K, V = synth.features(3, N, H, D, "f32")
    out, _, _ = run(rowptr, colidx, Q, K, V, np.float32(0.5))
    swapped = dense_reference(rowptr, colidx, K, Q, V, np.float32(0.5))
    assert np.max(np.abs(out - swapped)) > 1e-3


def test_zero_query_gives_neighbour_mean():
    N, H, D = 50, 2, 16
    rowptr, colidx = synth.ragged_graph(4, N, max_deg=12, empty_frac=0.1, dup_frac=0.1)
    _, K, V = synth.features(4, N, H, D, "f32")
    Q = np.zeros_like(K)
    out, _, _ = run(rowptr, colidx, Q, K, V, np.float32(0.25))
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        want = V[J].astype(np.float64).mean(axis=0) if J.size else np.zeros((H, D))
        np.testing.assert_allclose(out[i], want, rtol=1e-13, atol=1e-14)
    # scale = 0 is the same closed form with any Q
    Q2, _, _ = synth.features(5, N, H, D, "f32")
    out2, _, _ = run(rowptr, colidx, Q2, K, V, np.float32(0.0))
    np.testing.assert_allclose(out2, out, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_entry_row_is_exact(dtype):
    N, H, D = 30, 4, 32
    deg = np.ones(N, dtype=np.int64)
    rowptr, colidx = synth.csr_from_degrees(6, N, deg, self_loops=False)
    Q, K, V = synth.features(6, N, H, D, dtype, std=3.0)
    out, absagg, lse = run(rowptr, colidx, Q, K, V, np.float32(0.17))
    f = (lambda a: a) if dtype == "f32" else bf16_bits_to_f32
    assert np.array_equal(out, f(V)[colidx].astype(np.float64))
    assert np.array_equal(absagg, np.abs(f(V)[colidx]).astype(np.float64))


def test_permutation_invariance():
    N, H, D = 60, 2, 8
    rowptr, colidx = synth.ragged_graph(7, N, max_deg=25, self_loops=True, dup_frac=0.1)
    _, shuffled = synth.ragged_graph(7, N, max_deg=25, self_loops=True, dup_frac=0.1, shuffle=True)
    assert not np.array_equal(colidx, shuffled)
    Q, K, V = synth.features(7, N, H, D, "f32")
    a, _, la = run(rowptr, colidx, Q, K, V, np.float32(0.3))
    b, _, lb = run(rowptr, shuffled, Q, K, V, np.float32(0.3))
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(la, lb, rtol=1e-13, atol=1e-13)


def test_two_entries_logistic():
    N, H, D = 40, 2, 8
    rowptr, colidx = synth.csr_from_degrees(8, N, np.full(N, 2), self_loops=False)
    Q, K, V = synth.features(8, N, H, D, "f32")
    scale = np.float32(0.4)
    out, _, lse = run(rowptr, colidx, Q, K, V, scale)
    for i in range(N):
        j1, j2 = colidx[rowptr[i]:rowptr[i + 1]]
        for h in range(H):
            s1 = float(scale) * float(np.dot(Q[i, h].astype(np.float64), K[j1, h].astype(np.float64)))
            s2 = float(scale) * float(np.dot(Q[i, h].astype(np.float64), K[j2, h].astype(np.float64)))
            a1 = 1.0 / (1.0 + math.exp(s2 - s1))
            a2 = 1.0 / (1.0 + math.exp(s1 - s2))
            want = a1 * V[j1, h].astype(np.float64) + a2 * V[j2, h].astype(np.float64)
            np.testing.assert_allclose(out[i, h], want, rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(lse[i, h], max(s1, s2) + math.log1p(math.exp(-abs(s1 - s2))),
                                       rtol=1e-13, atol=1e-13)


def test_constant_values_and_convex_bounds():
    N, H, D = 50, 2, 8
    rowptr, colidx = synth.ragged_graph(9, N, max_deg=15, self_loops=True, dup_frac=0.1)
    Q, K, V = synth.features(9, N, H, D, "f32", std=2.0)
    Vc = np.full_like(V, np.float32(-1.25))
    out, _, _ = run(rowptr, colidx, Q, K, Vc, np.float32(0.5))
    np.testing.assert_allclose(out, -1.25, rtol=1e-14)
    out, absagg, _ = run(rowptr, colidx, Q, K, V, np.float32(0.5))
    for i in range(N):
        J = colidx[rowptr[i]:rowptr[i + 1]]
        lo = V[J].min(axis=0)
        hi = V[J].max(axis=0)
        assert np.all(out[i] >= lo - 1e-12) and np.all(out[i] <= hi + 1e-12)
    assert np.all(absagg >= np.abs(out) - 1e-12)
    Vp = np.abs(V)
    outp, absp, _ = run(rowptr, colidx, Q, K, Vp, np.float32(0.5))
    np.testing.assert_allclose(absp, outp, rtol=1e-14)


def test_linearity_in_v_and_head_independence():
    N, H, D = 45, 3, 8
    rowptr, colidx = synth.ragged_graph(10, N, max_deg=10, self_loops=True)
    Q, K, V1 = synth.features(10, N, H, D, "f32")
    _, _, V2 = synth.features(11, N, H, D, "f32")
    a, b = 0.75, -2.0
    Vmix = (a * V1.astype(np.float64) + b * V2.astype(np.float64)).astype(np.float32)
    # Vmix is rounded to float32; compare with the rounding accounted for
    o1, _, _ = run(rowptr, colidx, Q, K, V1, np.float32(0.35))
    o2, _, _ = run(rowptr, colidx, Q, K, V2, np.float32(0.35))
    om, _, _ = run(rowptr, colidx, Q, K, Vmix, np.float32(0.35))
    np.testing.assert_allclose(om, a * o1 + b * o2, rtol=0, atol=1e-6)
    for h in range(H):
        oh, _, _ = run(rowptr, colidx, np.ascontiguousarray(Q[:, h:h + 1]),
                       np.ascontiguousarray(K[:, h:h + 1]), np.ascontiguousarray(V1[:, h:h + 1]),
                       np.float32(0.35))
        assert np.array_equal(oh[:, 0], o1[:, h])


def test_dominant_score_is_stable():
    N, H, D = 16, 1, 8
    rowptr, colidx = synth.csr_from_degrees(12, N, np.full(N, 6), self_loops=True)
    Q, K, V = synth.features(12, N, H, D, "f32")
    # make the last entry of every row dominate by aligning its key with the query
    for i in range(N):
        jstar = colidx[rowptr[i + 1] - 1]
        K[jstar] = 0
    for i in range(N):
        jstar = colidx[rowptr[i + 1] - 1]
        K[jstar] += Q[i]
    scale = np.float32(1e4)  # scores up to ~1e5: exp would overflow without the max shift
    out, _, lse = run(rowptr, colidx, Q, K, V, scale)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))


def test_dominant_score_limit():
    N, H, D = 3, 1, 4
    rowptr = np.array([0, 3, 4, 5], dtype=np.int64)
    colidx = np.array([0, 1, 2, 1, 2], dtype=np.int32)
    Q = np.zeros((N, H, D), np.float32)
    K = np.zeros((N, H, D), np.float32)
    V, _, _ = synth.features(13, N, H, D, "f32")
    Q[0, 0, 0] = 1.0
    K[1, 0, 0] = 1.0
    out, _, lse = run(rowptr, colidx, Q, K, V, np.float32(1e6))
    np.testing.assert_array_equal(out[0], V[1].astype(np.float64))
    assert lse[0, 0] == pytest.approx(1e6)


def test_empty_rows():
    rowptr = np.array([0, 0, 2, 2], dtype=np.int64)
    colidx = np.array([0, 2], dtype=np.int32)
    Q, K, V = synth.features(14, 3, 2, 4, "f32")
    out, absagg, lse = run(rowptr, colidx, Q, K, V, np.float32(0.5))
    assert np.all(out[0] == 0) and np.all(out[2] == 0) and np.all(absagg[0] == 0)
    assert np.all(np.isneginf(lse[0])) and np.all(np.isneginf(lse[2]))
    assert np.all(np.isfinite(lse[1]))


def test_repeated_entry_counts_twice():
    rowptr = np.array([0, 3, 4, 5], dtype=np.int64)
    colidx = np.array([1, 2, 1, 1, 2], dtype=np.int32)
    Q, K, V = synth.features(15, 3, 1, 4, "f32")
    out, _, _ = run(rowptr, colidx, Q, K, V, np.float32(0.5))
    s1 = 0.5 * float(np.dot(Q[0, 0].astype(np.float64), K[1, 0].astype(np.float64)))
    s2 = 0.5 * float(np.dot(Q[0, 0].astype(np.float64), K[2, 0].astype(np.float64)))
    w1, w2 = 2 * math.exp(s1), math.exp(s2)
    want = (w1 * V[1, 0].astype(np.float64) + w2 * V[2, 0].astype(np.float64)) / (w1 + w2)
    np.testing.assert_allclose(out[0, 0], want, rtol=1e-13)


def test_row_subset_matches_full():
    w = synth.config(0)
    full, fa, fl = run(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale)
    rows = np.array([5, 0, 1999, 77, 5], dtype=np.int64)
    sub, sa, sl = run(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, rows=rows)
    assert np.array_equal(sub, full[rows]) and np.array_equal(sl, fl[rows])


def test_rejects_invalid_csr():
    rowptr = np.array([0, 2, 3], dtype=np.int64)
    colidx = np.array([0, 5, 1], dtype=np.int32)  # 5 is out of range
    Q, K, V = synth.features(16, 2, 1, 4, "f32")
    with pytest.raises(ValueError):
        run(rowptr, colidx, Q, K, V, np.float32(1.0))
    with pytest.raises(ValueError):
        run(np.array([0, 2, 2], dtype=np.int64), np.array([0, 1, 1], dtype=np.int32), Q, K, V,
            np.float32(1.0))


def dense_lse(rowptr, colidx, Qf, Kf, scale):
    """ln sum over the row's entries (with multiplicity) of exp(score), from the
    dense masked score matrix; -inf for an empty row."""
    N, H, D = Qf.shape
    C = np.zeros((N, N))
    for i in range(N):
        for e in range(rowptr[i], rowptr[i + 1]):
            C[i, colidx[e]] += 1.0
    out = np.full((N, H), -np.inf)
    for h in range(H):
        S = float(scale) * (Qf[:, h, :].astype(np.float64) @ Kf[:, h, :].astype(np.float64).T)
        for i in range(N):
            m = C[i] > 0
            if m.any():
                s = S[i, m]
                mx = s.max()
                out[i, h] = mx + math.log(float((C[i, m] * np.exp(s - mx)).sum()))
    return out


@pytest.mark.parametrize("case", range(60))
def test_dense_form_on_random_small_graphs(case):
    """Sixty seeded random cases of every size the oracle takes (1..40 rows, any
    H and D, empty rows, repeats, self-loops, unsorted rows, hubs, scales from
    negative to large), each against the dense masked form and its log-sum-exp."""
    rng = np.random.default_rng(5000 + case)
    N = int(rng.integers(1, 41))
    H, D = int(rng.integers(1, 4)), int(rng.integers(1, 17))
    dtype = "f32" if case % 2 == 0 else "bf16"
    hubs = {int(rng.integers(0, N)): int(rng.integers(1, N))} if N >= 2 and case % 3 == 0 else None
    rowptr, colidx = synth.ragged_graph(6000 + case, N, max_deg=int(rng.integers(0, 12)),
                                        empty_frac=float(rng.choice([0.0, 0.2, 0.6])), hubs=hubs,
                                        self_loops=bool(case % 4 == 1), dup_frac=float(rng.choice([0.0, 0.3])),
                                        shuffle=bool(case % 5 == 2))
    Q, K, V = synth.features(7000 + case, N, H, D, dtype, std=float(rng.choice([0.5, 1.0, 3.0])))
    scale = np.float32(rng.choice([1 / math.sqrt(D), 0.0, -0.7, 4.0]))
    out, absagg, lse = run(rowptr, colidx, Q, K, V, scale)
    f = (lambda a: a) if dtype == "f32" else bf16_bits_to_f32
    ref = dense_reference(rowptr, colidx, f(Q), f(K), f(V), scale)
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-10)
    ref_lse = dense_lse(rowptr, colidx, f(Q), f(K), scale)
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isneginf(lse), ~fin)
    np.testing.assert_allclose(lse[fin], ref_lse[fin], rtol=1e-12, atol=1e-10)
    assert np.all(absagg >= np.abs(out) - 1e-12)
