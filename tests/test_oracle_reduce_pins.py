"""Pins of the segment min/max oracle (paper Section 2.2, reduction family
(ii); Appendix, degree-aware reduction-based aggregation and its
order-preserving (key, index) packing).

Independent checks: a pure-Python brute force over (value, source) tuples on
inputs where the float order is the real order (no zeros, NaNs or
infinities), heavy ties from small integers (ties go to the smallest source
id), and the special values whose order the key rule fixes: -0 below +0,
infinities at the ends, a NaN with the sign bit clear above +inf and one with
the sign bit set below -inf."""
import math
import struct

import numpy as np
import pytest

import oracle
import synth


def f32(bits):
    return struct.unpack("<f", struct.pack("<I", bits))[0]


def bits_of(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def brute(rowptr, colidx, Xf, op):
    """Python tuple order: (value, source) for min; (-value, source) for max."""
    N, F = Xf.shape
    out = np.zeros((N, F), np.float32)
    arg = np.full((N, F), -1, np.int32)
    for i in range(N):
        J = [int(j) for j in colidx[rowptr[i]:rowptr[i + 1]]]
        if not J:
            continue
        for f in range(F):
            if op == "min":
                v, j = min((float(Xf[j, f]), j) for j in J)
            else:
                nv, j = min((-float(Xf[j, f]), j) for j in J)
                v = -nv
            out[i, f], arg[i, f] = v, j
    return out, arg


def csr(rows, N):
    rows = list(rows) + [[]] * (N - len(rows))
    rowptr = np.zeros(N + 1, np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    colidx = np.array([j for r in rows for j in r], np.int32)
    return rowptr, colidx


@pytest.mark.parametrize("op", ["min", "max"])
@pytest.mark.parametrize("seed", [0, 1])
def test_brute_force_random(op, seed):
    N, F = 60, 12
    rowptr, colidx = synth.ragged_graph(seed, N, max_deg=15, empty_frac=0.1, hubs={5: 59},
                                        self_loops=True, dup_frac=0.2, shuffle=True)
    X = synth.normal(seed, synth.STREAM_Q, (N, F), 1.0, "f32")
    X[X == 0] = 0.5
    out, arg = oracle.segment_reduce(rowptr, colidx, X, op)
    ref_out, ref_arg = brute(rowptr, colidx, X, op)
    assert np.array_equal(bits_of(out), bits_of(ref_out))
    assert np.array_equal(arg, ref_arg)


@pytest.mark.parametrize("op", ["min", "max"])
def test_ties_go_to_smallest_source_bf16(op):
    # small integers, exact in bf16: most rows have several sources at the
    # extreme value, so the tie rule decides the index
    N, F = 80, 16
    rowptr, colidx = synth.ragged_graph(3, N, max_deg=20, empty_frac=0.05, self_loops=True,
                                        dup_frac=0.1, shuffle=True)
    u = synth.uniform01(3, synth.STREAM_Q, N * F).reshape(N, F)
    Xf = (np.floor(u * 5) - 2).astype(np.float32)
    Xf[Xf == 0] = 3.0
    Xb = (Xf.view(np.uint32) >> 16).astype(np.uint16)
    out, arg = oracle.segment_reduce(rowptr, colidx, Xb, op)
    ref_out, ref_arg = brute(rowptr, colidx, Xf, op)
    assert np.array_equal(out, ref_out)
    assert np.array_equal(arg, ref_arg)
    assert (ref_arg >= 0).sum() > 0


def test_selected_value_is_the_source_value():
    N, F = 50, 8
    rowptr, colidx = synth.ragged_graph(4, N, max_deg=12, empty_frac=0.1, dup_frac=0.2)
    X = synth.normal(4, synth.STREAM_K, (N, F), 1.0, "f32")
    for op in ("min", "max"):
        out, arg = oracle.segment_reduce(rowptr, colidx, X, op)
        for i in range(N):
            J = set(colidx[rowptr[i]:rowptr[i + 1]].tolist())
            for f in range(F):
                if not J:
                    assert out[i, f] == 0 and arg[i, f] == -1
                else:
                    assert arg[i, f] in J and out[i, f] == X[arg[i, f], f]


def test_signed_zero_and_infinities():
    # sources: 0:-0.0  1:+0.0  2:-inf  3:+inf  4:1.0
    X = np.array([[-0.0], [0.0], [-np.inf], [np.inf], [1.0]], np.float32)
    rows = [[1, 0], [0, 1], [4, 3, 2], [1, 4], []]
    rowptr, colidx = csr(rows, 5)
    out, arg = oracle.segment_reduce(rowptr, colidx, np.ascontiguousarray(X), "min")
    assert [math.copysign(1, v) for v in out[:2, 0]] == [-1, -1]  # -0 below +0
    assert arg[:2, 0].tolist() == [0, 0]
    assert out[2, 0] == -np.inf and arg[2, 0] == 2
    assert out[3, 0] == 0 and math.copysign(1, out[3, 0]) == 1 and arg[3, 0] == 1
    assert out[4, 0] == 0 and arg[4, 0] == -1
    out, arg = oracle.segment_reduce(rowptr, colidx, np.ascontiguousarray(X), "max")
    assert math.copysign(1, out[0, 0]) == 1 and arg[0, 0] == 1  # +0 above -0
    assert out[2, 0] == np.inf and arg[2, 0] == 3
    assert out[3, 0] == 1.0 and arg[3, 0] == 4


def test_nan_placement_follows_the_key():
    pnan, nnan = f32(0x7FC00000), f32(0xFFC00000)
    X = np.array([[1.0], [pnan], [nnan], [-np.inf], [np.inf]], np.float32)
    rowptr, colidx = csr([[0, 1], [0, 2], [3, 2], [4, 1]], 5)
    out, arg = oracle.segment_reduce(rowptr, colidx, X, "min")
    assert arg[:, 0].tolist() == [0, 2, 2, 4, -1]  # +NaN above +inf; -NaN below -inf
    assert bits_of(out[1, 0]) == 0xFFC00000
    out, arg = oracle.segment_reduce(rowptr, colidx, X, "max")
    assert arg[:, 0].tolist() == [1, 0, 3, 1, -1]
    assert bits_of(out[0, 0]) == 0x7FC00000


def test_subnormals_and_mixed_signs_follow_real_order():
    tiny = [f32(1), f32(2), f32(0x807FFFFF), f32(0x80000001), 1e-38, -1e-38, 3.0, -3.0]
    X = np.array(tiny, np.float32)[:, None].copy()
    n = len(tiny)
    rowptr, colidx = csr([list(range(n))] + [[k] for k in range(1, n)], n)
    for op, fn in (("min", np.argmin), ("max", np.argmax)):
        out, arg = oracle.segment_reduce(rowptr, colidx, X, op)
        assert arg[0, 0] == fn(X[:, 0])
        assert np.array_equal(arg[1:, 0], np.arange(1, n))


def test_rows_subset_matches_all_rows():
    N, F = 70, 6
    rowptr, colidx = synth.ragged_graph(6, N, max_deg=10, empty_frac=0.1, dup_frac=0.1)
    X = synth.normal(6, synth.STREAM_V, (N, F), 1.0, "f32")
    out, arg = oracle.segment_reduce(rowptr, colidx, X, "max")
    rows = np.array([69, 3, 3, 0, 41], np.int64)
    o2, a2 = oracle.segment_reduce(rowptr, colidx, X, "max", rows=rows)
    assert np.array_equal(o2, out[rows]) and np.array_equal(a2, arg[rows])


@pytest.mark.parametrize("case", range(40))
def test_brute_force_on_random_small_graphs(case):
    """Forty seeded random cases (1..40 rows, 1..20 features, empty rows,
    repeats, self-loops, unsorted rows, small-integer values with many ties)
    against the brute force, min and max."""
    rng = np.random.default_rng(9000 + case)
    N, F = int(rng.integers(1, 41)), int(rng.integers(1, 21))
    rowptr, colidx = synth.ragged_graph(9100 + case, N, max_deg=int(rng.integers(0, 12)),
                                        empty_frac=float(rng.choice([0.0, 0.3])), self_loops=bool(case % 3 == 0),
                                        dup_frac=float(rng.choice([0.0, 0.3])), shuffle=bool(case % 4 == 1))
    if case % 2 == 0:
        X = synth.normal(9200 + case, synth.STREAM_Q, (N, F), 1.0, "f32")
        X[X == 0] = 0.5
    else:
        X = (rng.integers(1, 5, size=(N, F)) * rng.choice([-1.0, 1.0], size=(N, F))).astype(np.float32)
    for op in ("min", "max"):
        out, arg = oracle.segment_reduce(rowptr, colidx, X, op)
        ref_out, ref_arg = brute(rowptr, colidx, X, op)
        assert np.array_equal(bits_of(out), bits_of(ref_out))
        assert np.array_equal(arg, ref_arg)
