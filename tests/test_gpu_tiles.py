"""GPU parity of the dense-tile (MFMA) path for locally dense windows.

Graphs are 64-id block models with irregularities added so that every
fallback runs: a partial last window, rows with a repeated in-window entry
(left to the CSR kernel), a row long enough to be split (front path), empty
rows, rows whose only entries lie outside their window, and windows below the
density threshold."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import TOL_BF16, bf16_bits_to_f32, fwd_gate_error_all_rows, gate_error, run_gpu, workload

pytestmark = pytest.mark.gpu

TILE_SHAPES = [(1, 32), (1, 64), (1, 128), (2, 32), (2, 64), (4, 32)]
CSR_ONLY = {"dense_tiles": -1}


def csr_from_rows(rows):
    rowptr = np.zeros(len(rows) + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    colidx = np.concatenate([np.asarray(r, dtype=np.int32) for r in rows]) if rowptr[-1] else \
        np.zeros(0, dtype=np.int32)
    return rowptr, colidx


def irregular_block_graph(seed, n_windows=12, tail=37):
    N = 64 * n_windows + tail
    rp, ci = synth.sbm_graph(seed, N, 64, 4)
    rows = [list(ci[rp[i]:rp[i + 1]]) for i in range(N)]
    u = synth.uniform01(seed, synth.STREAM_EXTRA + 3, 4 * N)
    rows[3] = rows[3] + [rows[3][0]]                 # repeated in-window entry
    rows[70] = rows[70] + [rows[70][1], rows[70][1]]  # repeated twice
    rows[5] = []                                      # empty row in a dense window
    rows[130] = [int(x) for x in np.floor(u[:300] * N)]  # long row, split into chunks
    rows[200] = [(200 + 64 * 3) % N, (200 + 64 * 5) % N]  # only out-of-window entries
    # window 9 made sparse (below any sensible threshold): keep only self-loops
    for i in range(64 * 9, 64 * 10):
        rows[i] = [i]
    return csr_from_rows(rows)


def check(rowptr, colidx, Q, K, V, scale, tiles, rows=None):
    got = run_gpu(rowptr, colidx, Q, K, V, scale, tuning={"dense_tiles": tiles})
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, rows=rows, want_lse=False)
    if rows is not None:
        got = got[rows]
    assert np.all(np.isfinite(got))
    err = gate_error(got, ref, absagg)
    assert err <= TOL_BF16, "gate error %.3g" % err
    return got


@pytest.mark.parametrize("H,D", TILE_SHAPES)
def test_tiles_irregular(H, D):
    rowptr, colidx = irregular_block_graph(H * 100 + D)
    Q, K, V = synth.features(H * 100 + D, rowptr.size - 1, H, D, "bf16")
    scale = np.float32(1 / math.sqrt(D))
    a = check(rowptr, colidx, Q, K, V, scale, tiles=256)
    check(rowptr, colidx, Q, K, V, scale, tiles=1)
    # the tile path really ran: its products round differently from the CSR
    # step's, which changes some outputs in dense windows, and none in the
    # sparse window 9 (CSR kernel there)
    csr = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=CSR_ONLY)
    assert not np.array_equal(a[:64 * 9], csr[:64 * 9])
    assert np.array_equal(a[64 * 9:64 * 10], csr[64 * 9:64 * 10])


def test_tiles_window_flagged_but_below_threshold():
    """The partition's density estimate samples every 8th light row of a
    window.  Here the sampled rows point only inside their window and the
    others only outside, so the window is flagged (estimate 1280 entries)
    while it holds 160 in-window entries, below the threshold of 256: the
    tile kernel must then stream all of its rows without a tile.  A second
    window has the pattern reversed (estimate 0, 1120 in-window entries): it
    stays on the CSR kernel, untiled."""
    N = 64 * 3
    rows = []
    for i in range(N):
        w = i // 64
        inside = [64 * w + (i + 1 + t) % 64 for t in range(20)]
        outside = [(64 * w + 64 + 3 * t + i) % N for t in range(20)]
        outside = [j if j // 64 != w else (j + 64) % N for j in outside]
        sampled = i % 8 == 0
        if w == 0:
            rows.append(sorted(inside if sampled else outside))
        elif w == 1:
            rows.append(sorted(outside if sampled else inside))
        else:
            rows.append(sorted(set(inside[:10] + outside[:10])))
    rowptr, colidx = csr_from_rows(rows)
    Q, K, V = synth.features(26, N, 2, 64, "bf16")
    got = check(rowptr, colidx, Q, K, V, np.float32(0.125), tiles=256)
    assert np.array_equal(got, run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125)))  # the default


def test_tiles_single_entry_exact():
    N, H, D = 64 * 8 + 5, 2, 64
    rowptr = np.arange(N + 1, dtype=np.int64)
    colidx = np.arange(N, dtype=np.int32)  # self-loop only: one in-window entry per row
    Q, K, V = synth.features(21, N, H, D, "bf16", std=2.0)
    got = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning={"dense_tiles": 1})
    assert np.array_equal(got, bf16_bits_to_f32(V))


def test_tiles_deterministic_and_off_equivalence():
    rowptr, colidx = irregular_block_graph(22)
    Q, K, V = synth.features(22, rowptr.size - 1, 2, 64, "bf16")
    a = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning={"dense_tiles": 256})
    b = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning={"dense_tiles": 256})
    assert np.array_equal(a, b)
    # a threshold no window reaches leaves everything to the CSR kernel
    off = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning=CSR_ONLY)
    none = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning={"dense_tiles": 1 << 20})
    assert np.array_equal(off, none)
    # the default is the tile path at threshold 256
    assert np.array_equal(run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125)), a)


def test_tiles_ignored_for_fp32_and_wide_rows():
    rowptr, colidx = irregular_block_graph(23)
    N = rowptr.size - 1
    Q, K, V = synth.features(23, N, 2, 64, "f32")
    assert np.array_equal(run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125), tuning=CSR_ONLY),
                          run_gpu(rowptr, colidx, Q, K, V, np.float32(0.125),
                                  tuning={"dense_tiles": 256}))
    Qb, Kb, Vb = synth.features(23, N, 8, 64, "bf16")  # H*D = 512: no tile variant
    assert np.array_equal(run_gpu(rowptr, colidx, Qb, Kb, Vb, np.float32(0.125), tuning=CSR_ONLY),
                          run_gpu(rowptr, colidx, Qb, Kb, Vb, np.float32(0.125),
                                  tuning={"dense_tiles": 256}))


@pytest.mark.parametrize("bf16_weights", [0, 1])
@pytest.mark.parametrize("H,D", TILE_SHAPES)
def test_tiles_weight_precision(H, D, bf16_weights):
    """Tiles keep each weight as two bf16 terms (two P*V products) by default:
    only the bf16 output rounding (2^-8) and fp32-level terms are left; with
    bf16_weights the rounded weights add up to 2^-8 of the absolute sum.  lse
    to the fp32 tolerance either way (the normaliser sums the fp32 weights)."""
    import torch
    import paper_2605_31500_amd as gtm
    from tests.helpers import to_device
    rowptr, colidx = irregular_block_graph(H * 100 + D + 1)
    N = rowptr.size - 1
    Q, K, V = synth.features(H * 100 + D + 1, N, H, D, "bf16")
    scale = np.float32(1 / math.sqrt(D))
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dev[2])
    lse = torch.empty((N, H), dtype=torch.float32, device=out.device)
    gtm.gt_attn_fwd_ex(*dev, out, scale, tuning={"dense_tiles": 1, "bf16_weights": bf16_weights}, lse=lse)
    torch.cuda.synchronize()
    got = bf16_bits_to_f32(out.view(torch.int16).cpu().numpy().view(np.uint16))
    ref, absagg, ref_lse = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale)
    assert gate_error(got, ref, absagg) <= 2.0 ** -8 * (1 + bf16_weights) + 1e-4
    l = lse.cpu().numpy()
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isneginf(l), ~fin)
    assert np.all(np.abs(l[fin] - ref_lse[fin]) <= 1e-5 * np.maximum(1.0, np.abs(ref_lse[fin])))


def test_tiles_off_full_sbm_all_rows():
    # the CSR kernel alone on the locally dense workload (tiles are the default there)
    w = workload(3)
    got = run_gpu(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, tuning=CSR_ONLY)
    assert np.all(np.isfinite(got))
    err = fwd_gate_error_all_rows(w, got)
    print("gate error %.3g" % err, flush=True)
    assert err <= TOL_BF16, "gate error %.3g" % err


def test_tiles_rows_at_the_degree_limit():
    # light rows in tile mode hold at most 64 entries: a row of all 64 window
    # ids (full mask), one of 64 out-of-window entries (all streamed), a 32/32
    # mix, 63 entries, and a 65-entry row that belongs to the CSR kernel
    N = 64 * 6 + 11
    rp, ci = synth.sbm_graph(24, N, 64, 4)
    rows = [list(ci[rp[i]:rp[i + 1]]) for i in range(N)]
    outside = [j for j in range(N) if j // 64 != 1]
    rows[10] = list(range(64))
    rows[75] = outside[5:69]
    rows[140] = list(range(128, 160)) + outside[100:132]
    rows[141] = list(range(128, 192)) + [3]
    rows[142] = list(range(128, 191))
    rowptr, colidx = csr_from_rows(rows)
    assert [int(rowptr[i + 1] - rowptr[i]) for i in (10, 75, 140, 141, 142)] == [64, 64, 64, 65, 63]
    Q, K, V = synth.features(24, N, 2, 64, "bf16")
    for tiles in (1, 256):
        check(rowptr, colidx, Q, K, V, np.float32(0.125), tiles=tiles)


@pytest.mark.parametrize("N", [1, 5, 63, 64, 65, 129])
def test_tiles_graphs_smaller_than_or_near_a_window(N):
    # one partial window, exactly one, and one full window plus a few rows
    rp, ci = synth.sbm_graph(25 + N, N, 64, 4 if N >= 68 else 0)
    Q, K, V = synth.features(25 + N, N, 2, 64, "bf16")
    for tiles in (1, 256):
        check(rp, ci, Q, K, V, np.float32(0.125), tiles=tiles)
