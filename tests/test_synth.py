"""Generator checks: Philox known answers, determinism, CSR invariants and the
degree statistics each workload recipe is meant to have."""
import numpy as np
import pytest

import synth


def test_philox_known_answers():
    # Known-answer vectors published with Random123 for Philox4x32-10.
    kat = [
        ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
        ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
        ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
         [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
    ]
    for ctr, key, want in kat:
        assert list(synth.philox4x32_10(ctr, key)) == want


def test_normal_moments_and_bf16_rounding():
    x = synth.normal(0, synth.STREAM_Q, (1 << 20,), 0.5, "f32")
    assert abs(x.mean()) < 3e-3 and abs(x.std() - 0.5) < 3e-3
    b = synth.normal(0, synth.STREAM_Q, (1 << 20,), 0.5, "bf16")
    wide = synth.bf16_to_f32(b)
    # round to nearest: |x - bf16(x)| <= half an ulp of bf16 (2^-8 relative)
    assert np.all(np.abs(wide - x) <= np.abs(x) * 2.0 ** -8 + 1e-38)
    # deterministic and independent of how the call is split
    assert np.array_equal(synth.normal(0, synth.STREAM_Q, (1000,), 0.5, "f32"), x[:1000])


def _row_sets(rowptr, colidx):
    return [colidx[rowptr[i]:rowptr[i + 1]] for i in range(rowptr.size - 1)]


def test_er_recipe():
    w = synth.config(0)
    synth.check_csr(w.rowptr, w.colidx, w.N)
    assert w.N == 2000 and w.E == 18000 and w.H == 1 and w.D == 32 and w.dtype == "f32"
    assert np.all(np.diff(w.rowptr) == 9)
    for i, r in enumerate(_row_sets(w.rowptr, w.colidx)):
        assert np.all(np.diff(r) > 0) and i in r  # sorted, distinct, self-loop present
    w2 = synth.config(0)
    assert np.array_equal(w.colidx, w2.colidx) and np.array_equal(w.Q, w2.Q)
    assert w.scale == np.float32(1 / np.sqrt(32))


def test_chung_lu_recipe():
    w = synth.config(1)
    synth.check_csr(w.rowptr, w.colidx, w.N)
    deg = np.diff(w.rowptr) - 1  # in-neighbours besides the self-loop
    assert w.N == 169_343 and 1.0e6 < w.E < 1.5e6
    assert deg.min() >= 1 and 5_000 < deg.max() <= 13_000
    assert 0.4 < np.mean(deg == 1) < 0.6
    i = int(np.argmax(deg))
    r = w.colidx[w.rowptr[i]:w.rowptr[i + 1]]
    assert np.all(np.diff(r) > 0) and i in r


def test_rmat_recipe_small():
    rp, ci = synth.rmat_graph(0, 12, 0.57, 0.19, 0.19, 24)
    N = 1 << 12
    synth.check_csr(rp, ci, N)
    assert ci.size == 24 * N
    rows = np.repeat(np.arange(N), np.diff(rp))
    key = rows.astype(np.int64) * N + ci
    assert np.unique(key).size == key.size  # no repeated pair
    assert np.sum(rows == ci) == N          # exactly one self-loop per node
    deg = np.diff(rp)
    assert deg.max() > 20 * deg.mean()      # heavy skew
    # node ids are permuted: the heaviest rows are not concentrated at low ids
    heavy = np.argsort(deg)[-50:]
    assert heavy.mean() > N / 8


def test_sbm_recipe_small():
    N, bs = 64 * 64, 64
    rp, ci = synth.sbm_graph(0, N, bs, 4)
    synth.check_csr(rp, ci, N)
    rows = np.repeat(np.arange(N), np.diff(rp))
    same = (rows // bs) == (ci // bs)
    inter = np.bincount(rows[~same], minlength=N)
    assert np.all(inter == 4)
    intra = np.bincount(rows[same], minlength=N) - 1  # minus self
    assert abs(intra.mean() - 31.5) < 0.5
    assert np.sum(rows == ci) == N


def test_sbm_partial_block_and_impossible_out_degree():
    # a partial last block still gets its out-of-block sources
    rp, ci = synth.sbm_graph(3, 64 + 10, 64, 4)
    synth.check_csr(rp, ci, 74)
    rows = np.repeat(np.arange(74), np.diff(rp))
    assert np.all(np.bincount(rows[(rows // 64) != (ci // 64)], minlength=74) == 4)
    # fewer ids outside a block than distinct sources asked for is refused
    with pytest.raises(ValueError):
        synth.sbm_graph(3, 65, 64, 4)


def test_lognormal_recipe_small():
    N = 100_000
    rp, ci = synth.lognormal_graph(0, N, total=3_000_000)
    synth.check_csr(rp, ci, N)
    deg = np.diff(rp) - 1
    assert deg.min() >= 1 and abs(deg.sum() / 3e6 - 1) < 0.02
    assert deg.max() > 200 * np.median(deg) / 10


def test_ragged_graph_features():
    rp, ci = synth.ragged_graph(1, 200, 12, empty_frac=0.2, hubs={3: 150}, dup_frac=0.3,
                                shuffle=True)
    synth.check_csr(rp, ci, 200)
    deg = np.diff(rp)
    assert deg[3] == 150 and np.sum(deg == 0) > 20
    rows = _row_sets(rp, ci)
    assert any(np.unique(r).size < r.size for r in rows)        # repeated entries exist
    assert any(np.any(np.diff(r) < 0) for r in rows)             # unsorted rows exist
