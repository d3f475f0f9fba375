"""GPU properties of the HIP path that hold at any size: exact single-entry
rows, closed forms, determinism, split invariance, empty inputs, 64-bit
offsets, the CSR validator and error reporting."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.helpers import (TOL_BF16, TOL_F32, bf16_bits_to_f32, gate_error, run_gpu, sample_rows, workload,
                           score_rounding_bound, to_device, to_host_f32)

pytestmark = pytest.mark.gpu


def gt():
    import paper_2605_31500_amd as m
    return m


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,D", [(1, 32), (4, 32), (2, 64), (8, 64), (8, 128)])
def test_single_entry_rows_exact(H, D, dtype):
    N = 5000
    rowptr, colidx = synth.csr_from_degrees(1, N, np.ones(N, dtype=np.int64), self_loops=False)
    Q, K, V = synth.features(1, N, H, D, dtype, std=2.0)
    got = run_gpu(rowptr, colidx, Q, K, V, np.float32(1 / math.sqrt(D)))
    want = (V if dtype == "f32" else bf16_bits_to_f32(V))[colidx]
    assert np.array_equal(got, want)


def test_zero_query_gives_mean():
    N, H, D = 3000, 4, 32
    rowptr, colidx = synth.ragged_graph(2, N, max_deg=40, empty_frac=0.05, hubs={11: 2999})
    _, K, V = synth.features(2, N, H, D, "f32")
    Q = np.zeros_like(K)
    got = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.3))
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, 0.3)
    assert gate_error(got, ref, absagg) <= TOL_F32


def test_constant_values():
    N, H, D = 4000, 2, 64
    rowptr, colidx = synth.ragged_graph(3, N, max_deg=60, empty_frac=0.0, hubs={5: 3500})
    Q, K, _ = synth.features(3, N, H, D, "f32")
    V = np.full_like(Q, np.float32(0.75))
    got = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2))
    nonempty = np.diff(rowptr) > 0
    np.testing.assert_allclose(got[nonempty], 0.75, rtol=2e-6)
    assert np.all(got[~nonempty] == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_deterministic_and_split_invariant(dtype):
    N, H, D = 20000, 4, 32
    rowptr, colidx = synth.ragged_graph(4, N, max_deg=30, hubs={1: 19999, 2: 5000, 3: 1500})
    Q, K, V = synth.features(4, N, H, D, dtype)
    scale = np.float32(1 / math.sqrt(D))
    settings = [None, {"light_max_deg": 4, "heavy_min_deg": 64, "chunk_edges": 128, "grid_blocks": 0},
                {"light_max_deg": 1, "heavy_min_deg": 2, "chunk_edges": 64, "grid_blocks": 8}]
    outs = []
    for tu in settings:
        a = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tu)
        b = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tu)
        assert np.array_equal(a, b)  # bitwise reproducible for a fixed setting
        outs.append(a)
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale)
    t = TOL_F32 if dtype == "f32" else TOL_BF16
    for o in outs:
        assert gate_error(o, ref, absagg) <= t


def test_no_edges_and_single_node():
    N, H, D = 1000, 2, 32
    rowptr = np.zeros(N + 1, dtype=np.int64)
    colidx = np.zeros(0, dtype=np.int32)
    Q, K, V = synth.features(5, N, H, D, "f32")
    assert np.all(run_gpu(rowptr, colidx, Q, K, V, np.float32(0.1)) == 0)
    rp1 = np.array([0, 1], dtype=np.int64)
    ci1 = np.array([0], dtype=np.int32)
    Q1, K1, V1 = synth.features(6, 1, H, D, "f32")
    assert np.array_equal(run_gpu(rp1, ci1, Q1, K1, V1, np.float32(0.1)), V1)


def test_empty_graph_call_is_a_no_op():
    z = torch.zeros(0, 4, 32, device="cuda")
    gt().gt_attn_fwd(torch.zeros(1, dtype=torch.int64, device="cuda"),
                     torch.zeros(0, dtype=torch.int32, device="cuda"), z, z, z, z.clone(), 0.1)
    torch.cuda.synchronize()


def test_non_default_stream():
    N, H, D = 2000, 4, 32
    rowptr, colidx = synth.ragged_graph(7, N, max_deg=20, hubs={3: 1999})
    Q, K, V = synth.features(7, N, H, D, "f32")
    a = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2))
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2), stream=s)
    assert np.array_equal(a, b)


def test_concurrent_host_threads_and_streams():
    """Four host threads, each with its own stream, issue interleaved calls on
    different graphs and settings (every call has its own workspace); every
    result equals the same call made alone."""
    import threading
    import paper_2605_31500_amd as gtm
    cases = []
    for t in range(4):
        N, H, D = 3000 + 500 * t, 4, 32
        rowptr, colidx = synth.ragged_graph(40 + t, N, max_deg=30, hubs={5: N - 1, 9: 2000})
        Q, K, V = synth.features(40 + t, N, H, D, "f32" if t % 2 == 0 else "bf16")
        tuning = None if t < 2 else {"light_max_deg": 4, "heavy_min_deg": 32, "chunk_edges": 64,
                                    "grid_blocks": 0}
        want = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2), tuning=tuning)
        dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
        cases.append((dev, tuning, want))
    torch.cuda.synchronize()
    results, errors = [None] * 4, []

    def work(t):
        try:
            dev, tuning, _ = cases[t]
            s = torch.cuda.Stream()
            outs = []
            with torch.cuda.stream(s):
                for _ in range(5):
                    out = torch.empty_like(dev[2])
                    gtm.gt_attn_fwd_ex(*dev, out, np.float32(0.2), tuning=tuning, stream=s)
                    outs.append(out)
            s.synchronize()
            results[t] = [to_host_f32(o) for o in outs]
        except Exception as e:  # reported below, in the test's own thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(t,)) for t in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    for t in range(4):
        for got in results[t]:
            assert np.array_equal(got, cases[t][2])


def test_offsets_beyond_4_gib():
    """Feature tensors larger than 2^32 bytes, with every edge touching rows
    whose byte offset is past 4 GiB (64-bit address arithmetic)."""
    H, D = 8, 64                      # 1 KiB per bf16 node row
    N = (1 << 22) + 200_000           # ~4.5 GB per feature tensor
    W = 3000                          # active window at the top of the id range
    lo = N - W
    rp_small, ci_small = synth.ragged_graph(8, W, max_deg=40, hubs={17: 2500}, self_loops=True)
    Qs, Ks, Vs = synth.features(8, W, H, D, "bf16")
    deg_small = np.diff(rp_small)
    rowptr = np.zeros(N + 1, dtype=np.int64)
    rowptr[lo + 1:] = np.cumsum(deg_small)
    colidx = (ci_small.astype(np.int64) + lo).astype(np.int32)
    feats = []
    for small in (Qs, Ks, Vs):
        t = torch.zeros((N, H, D), dtype=torch.bfloat16, device="cuda")
        t[lo:] = to_device(small)
        feats.append(t)
    out = torch.full((N, H, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    scale = np.float32(1 / math.sqrt(D))
    gt().gt_attn_fwd_bf16(to_device(rowptr), to_device(colidx), *feats, out, scale)
    torch.cuda.synchronize()
    got = to_host_f32(out[lo:])
    assert np.all(to_host_f32(out[:1000]) == 0)  # empty rows
    ref, absagg, _ = oracle.gt_attn_fwd(rp_small, ci_small, Qs, Ks, Vs, scale)
    assert gate_error(got, ref, absagg) <= TOL_BF16
    del feats, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["group_per_row", "wave_per_row"])
def test_degree_agnostic_mappings(mode):
    """The degree-agnostic tunings timed by the allocation ablation (every row
    on one lane group, or on one wavefront, with no split) compute the same
    function: parity on the power-law workload, whose hub rows then run whole
    on one group or one wave."""
    import bench
    w = workload(1)
    got = run_gpu(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, tuning=bench.ABLATION_MODES[mode])
    ref, absagg, _ = oracle.gt_attn_fwd(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, want_lse=False)
    assert gate_error(got, ref, absagg) <= TOL_F32


def max_edge_graph():
    """CSR with E = 2^31 - 1 entries, the largest count the boundary accepts.
    Degrees cycle through every row class of the degree partition (empty,
    light, the light/medium and medium/front boundaries, a front row in one
    chunk, rows split into several and into the maximum number of chunks);
    sources are uniform."""
    cyc = np.array([0, 1, 5, 64, 65, 255, 256, 1024, 1025, 65000], dtype=np.int64)
    e_max = (1 << 31) - 1
    reps = e_max // int(cyc.sum())
    deg = np.concatenate([np.tile(cyc, reps), [e_max - reps * int(cyc.sum())]])
    rowptr = np.zeros(deg.size + 1, dtype=np.int64)
    np.cumsum(deg, out=rowptr[1:])
    colidx = np.random.default_rng(31).integers(0, deg.size, size=e_max, dtype=np.int32)
    return rowptr, colidx


def test_max_edge_count():
    rowptr, colidx = max_edge_graph()
    N, E = rowptr.size - 1, int(rowptr[-1])
    assert E == (1 << 31) - 1
    print("max-E graph: N", N, "E", E, flush=True)
    H, D = 1, 32
    Q, K, V = synth.features(31, N, H, D, "f32")
    scale = np.float32(1 / math.sqrt(D))
    got = run_gpu(rowptr, colidx, Q, K, V, scale)
    rows = np.unique(np.concatenate([np.arange(40), np.arange(N - 40, N),
                                     synth_rows(rowptr)]))
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, rows=rows, want_lse=False)
    assert np.all(np.isfinite(got[rows]))
    assert gate_error(got[rows], ref, absagg) <= TOL_F32


def synth_rows(rowptr):
    from tests.helpers import sample_rows
    return sample_rows(rowptr, n_random=300, n_top=16)


def test_csr_validator():
    rowptr, colidx = synth.ragged_graph(9, 500, max_deg=10)
    r, c = to_device(rowptr), to_device(colidx)
    assert gt().gt_csr_validate(r, c)
    bad = colidx.copy()
    bad[len(bad) // 2] = 500
    assert not gt().gt_csr_validate(r, to_device(bad))
    badr = rowptr.copy()
    badr[10], badr[11] = badr[11], badr[10] - 1
    assert not gt().gt_csr_validate(to_device(badr), c)


def test_errors_raise():
    m = gt()
    z = torch.zeros(10, 3, 32, device="cuda")
    rp = torch.zeros(11, dtype=torch.int64, device="cuda")
    ci = torch.zeros(0, dtype=torch.int32, device="cuda")
    with pytest.raises(m.GtError) as e:
        m.gt_attn_fwd(rp, ci, z, z, z, z.clone(), 0.1)  # H = 3 is not compiled
    assert e.value.status == m.GT_ERROR_NOT_SUPPORTED
    z4 = torch.zeros(10, 4, 32, device="cuda")
    with pytest.raises(m.GtError) as e:
        m.gt_attn_fwd(rp, ci, z4, z4, z4, z4, 0.1)  # out aliases Q
    assert e.value.status == m.GT_ERROR_INVALID_VALUE


@pytest.mark.parametrize("tuning", [None, {"light_max_deg": 2, "heavy_min_deg": 6, "chunk_edges": 64}],
                         ids=["default", "forced_split"])
@pytest.mark.parametrize("scale", [2.0, 8.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_peaked_scores(dtype, scale, tuning):
    """Scores spread over hundreds of units (one or two entries carry almost all
    the weight, and most rescale factors of the online softmax and of the chunk
    merge underflow to zero) still match the oracle within the score-rounding
    bound, per row and head."""
    N, H, D = 3000, 4, 32
    rowptr, colidx = synth.ragged_graph(31, N, max_deg=40, hubs={3: 2999, 9: 1800})
    Q, K, V = synth.features(31, N, H, D, dtype)
    got = run_gpu(rowptr, colidx, Q, K, V, np.float32(scale), tuning=tuning)
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
    assert np.all(np.isfinite(got))
    denom = np.maximum(np.maximum(np.abs(ref), absagg), 1e-30)
    err = np.max(np.abs(got - ref) / denom, axis=2)  # [N, H]
    # a weight exp(s_e - m) is off by at most the errors of s_e and of the running max
    bound = (2.0 * score_rounding_bound(rowptr, colidx, Q, K, scale)
             + (TOL_F32 if dtype == "f32" else TOL_BF16))
    assert np.all(err <= bound), "worst ratio %.3g" % np.max(err / bound)
    # the spread is real: on most rows the largest weight is above 0.9
    Qf, Kf = ((bf16_bits_to_f32(x) if dtype == "bf16" else x).astype(np.float64) for x in (Q, K))
    s = np.einsum("ehd,ehd->eh", Qf[np.repeat(np.arange(N), np.diff(rowptr))], Kf[colidx]) * scale
    deg = np.diff(rowptr)
    rows = np.nonzero(deg >= 2)[0]
    top = []
    for i in rows[:300]:
        se = s[rowptr[i]:rowptr[i + 1]]
        w = np.exp(se - se.max(axis=0))
        top.append(np.max(w / w.sum(axis=0), axis=0))
    assert np.median(np.array(top)) > 0.9


def test_binding_rejects_wrong_index_tensors():
    """Index tensors of the wrong dtype or on the host are refused before any
    launch (an int32 rowptr read as int64 would run past its end)."""
    m = gt()
    rp32 = torch.zeros(11, dtype=torch.int32, device="cuda")
    rp = torch.zeros(11, dtype=torch.int64, device="cuda")
    ci = torch.zeros(0, dtype=torch.int32, device="cuda")
    ci64 = torch.zeros(0, dtype=torch.int64, device="cuda")
    X = torch.zeros(10, 32, device="cuda")
    s = torch.zeros(10, device="cuda")
    with pytest.raises(TypeError):
        m.gt_dot_aggr(rp32, ci, X, s)
    with pytest.raises(TypeError):
        m.gt_dot_aggr(rp, ci64, X, s)
    with pytest.raises(TypeError):
        m.gt_csr_validate(rp32, ci)
    with pytest.raises(TypeError):
        m.gt_csr_validate(rp, ci64)
    with pytest.raises(ValueError):
        m.gt_csr_validate(rp.cpu(), ci)
    with pytest.raises(ValueError):
        m.gt_csr_validate(rp[:0], ci)
    z = torch.zeros(10, 4, 32, device="cuda")
    with pytest.raises(TypeError):
        m.gt_attn_fwd(rp32, ci, z, z, z, z.clone(), 0.1)
    with pytest.raises(ValueError):
        m.gt_attn_fwd(rp.cpu(), ci, z, z, z, z.clone(), 0.1)
    assert m.gt_csr_validate(rp, ci)  # N = 10 empty rows is a valid structure
    m.gt_dot_aggr(rp, ci, X, s)
    torch.cuda.synchronize()
    assert torch.count_nonzero(s).item() == 0


def test_profiler_counts_calls():
    m = gt()
    N, H, D = 3000, 4, 32
    rowptr, colidx = synth.ragged_graph(10, N, max_deg=20, hubs={3: 2999})
    Q, K, V = synth.features(10, N, H, D, "f32")
    dt = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dt[2])
    m.gt_profile_enable(True)
    for _ in range(3):
        m.gt_attn_fwd(*dt, out, 0.2)
    ms, calls = m.gt_profile_collect()
    m.gt_profile_enable(False)
    assert calls == 3 and all(x > 0 for x in ms)


def test_workspace_reuse_growth_and_release():
    """Consecutive calls of different sizes reuse pooled workspace memory; the
    counters of every call start at zero and results do not depend on what a
    workspace held before."""
    small = synth.ragged_graph(11, 3000, max_deg=30, hubs={1: 2999, 2: 1500})
    big = synth.ragged_graph(12, 40000, max_deg=50, hubs={5: 39999, 6: 20000, 7: 5000})
    feats = {n: synth.features(13, n, 4, 32, "f32") for n in (3000, 40000)}

    def run(g):
        rp, ci = g
        Q, K, V = feats[rp.size - 1]
        return run_gpu(rp, ci, Q, K, V, np.float32(0.2))

    a1 = run(small)
    b1 = run(big)
    a2 = run(small)
    b2 = run(big)
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2)
    gt().gt_workspace_release()
    assert np.array_equal(run(small), a1)
    rp, ci = big
    Q, K, V = feats[40000]
    ref, absagg, _ = oracle.gt_attn_fwd(rp, ci, Q, K, V, 0.2)
    assert gate_error(b1, ref, absagg) <= TOL_F32


def test_counter_sets_across_mixed_calls():
    """A forward call on a reused workspace block skips the counter clear: it
    uses one of the block's two counter sets, and its partition zeroes the
    other for the block's next call.  Segment reductions in between use the
    block their own way (the next forward clears again).  A sequence of
    forward calls on two graphs, with split rows and with the dense-tile
    path, interleaved with reductions, all on one stream with no
    synchronisation, gives every forward result exactly as a call on its
    own."""
    import paper_2605_31500_amd as gtm
    cases = []
    for seed, n, dtype in ((31, 3000, "f32"), (32, 40_000, "f32"), (33, 4096, "bf16")):
        if dtype == "bf16":  # dense 64-id blocks: the tile path
            rp, ci = synth.sbm_graph(seed, n, 64, 4)
        else:
            rp, ci = synth.ragged_graph(seed, n, max_deg=40, hubs={3: n - 1, 7: n // 2})
        Q, K, V = synth.features(seed, n, 2, 64, dtype)
        want = run_gpu(rp, ci, Q, K, V, np.float32(0.2))
        dev = [to_device(x) for x in (rp, ci, Q, K, V)]
        cases.append((dev, want))
    X = to_device(synth.features(34, 40_000, 1, 32, "f32")[0].reshape(40_000, 32))
    red_out = torch.empty_like(X)
    rp2, ci2 = cases[1][0][0], cases[1][0][1]
    torch.cuda.synchronize()
    gtm.gt_workspace_release()
    order = [0, 1, 0, "r", 2, 1, 1, "r", "r", 0, 2, 2, 1]
    outs = []
    for k in order:
        if k == "r":
            gtm.gt_segment_reduce(rp2, ci2, X, red_out, None, op="min")
            continue
        dev, _ = cases[k]
        o = torch.empty_like(dev[2])
        gtm.gt_attn_fwd_ex(*dev, o, np.float32(0.2))
        outs.append((k, o))
    torch.cuda.synchronize()
    for k, o in outs:
        assert np.array_equal(to_host_f32(o), cases[k][1]), "call on graph %d differs" % k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_regular_entry_point_replays_in_a_hip_graph(dtype):
    """On a stream being captured, a call takes its workspace stream-ordered
    (allocation and free become graph nodes) and clears its counters with the
    fill kernel.  Captured once, the graph is replayed three times, with eager
    work and synchronisations between the replays; every replay equals the
    eager call bit for bit (split rows and, for bf16 2x64, dense tiles)."""
    import paper_2605_31500_amd as gtm
    if dtype == "bf16":
        rowptr, colidx = synth.sbm_graph(72, 8192, 64, 4)
        H, D = 2, 64
    else:
        rowptr, colidx = synth.ragged_graph(71, 20_000, max_deg=60, hubs={2: 19_999, 9: 5000}, self_loops=True)
        H, D = 4, 32
    N = rowptr.size - 1
    Q, K, V = synth.features(71, N, H, D, dtype)
    want = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2))
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dev[2])
    fwd = gtm.gt_attn_fwd if dtype == "f32" else gtm.gt_attn_fwd_bf16
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fwd(*dev, out, np.float32(0.2), stream=s)
    for _ in range(3):
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(to_host_f32(out), want)


def test_calls_return_without_waiting_for_the_device():
    """A call enqueues its work and returns: behind a device-side sleep on its
    stream, five calls take a small fraction of the sleep on the host (freeing
    each call's workspace stream-ordered made every call wait for the previous
    call's kernels), and all five results are right."""
    import time
    import paper_2605_31500_amd as gtm
    N, H, D = 60_000, 4, 32
    rowptr, colidx = synth.chung_lu_graph(21, N)
    Q, K, V = synth.features(21, N, H, D, "f32")
    want = run_gpu(rowptr, colidx, Q, K, V, np.float32(0.2))
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    outs = [torch.empty_like(dev[2]) for _ in range(5)]
    gtm.gt_attn_fwd(*dev, outs[0], np.float32(0.2))  # a free block whose work is done
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    torch.cuda._sleep(int(2e8))  # 2e8 shader clock cycles: about 0.1 s
    t1 = time.perf_counter()
    for o in outs:
        gtm.gt_attn_fwd(*dev, o, np.float32(0.2))
    host = time.perf_counter() - t1
    torch.cuda.current_stream().synchronize()
    total = time.perf_counter() - t0
    print("five calls behind a %.3f s device sleep: %.4f s on the host" % (total, host), flush=True)
    assert total > 0.02
    assert host < 0.25 * total, "calls waited for the device: %.4f of %.4f s" % (host, total)
    for o in outs:
        assert np.array_equal(to_host_f32(o), want)


def test_block_in_use_on_another_stream_is_not_handed_out():
    """A workspace block whose last call is still pending on stream A is not
    given to a call on stream B: B's call gets a block of its own (the pool
    grows), and both results are right."""
    import paper_2605_31500_amd as gtm
    N, H, D = 60_000, 4, 32
    rowptr, colidx = synth.chung_lu_graph(22, N)
    Qa, Ka, Va = synth.features(22, N, H, D, "f32")
    Qb, Kb, Vb = synth.features(23, N, H, D, "f32")
    want_a = run_gpu(rowptr, colidx, Qa, Ka, Va, np.float32(0.2))
    want_b = run_gpu(rowptr, colidx, Qb, Kb, Vb, np.float32(0.2))
    rp, ci = to_device(rowptr), to_device(colidx)
    fa = [to_device(x) for x in (Qa, Ka, Va)]
    fb = [to_device(x) for x in (Qb, Kb, Vb)]
    out_a, out_b = torch.empty_like(fa[0]), torch.empty_like(fb[0])
    torch.cuda.synchronize()
    gtm.gt_workspace_release()
    gtm.gt_attn_fwd(rp, ci, *fa, out_a, np.float32(0.2))  # one block, done after the sync
    torch.cuda.synchronize()
    one_block = gtm.gt_workspace_pool_stats()[0]
    assert one_block > 0
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(sa):
        torch.cuda._sleep(int(2e8))
        gtm.gt_attn_fwd(rp, ci, *fa, out_a, np.float32(0.2), stream=sa)
    with torch.cuda.stream(sb):
        gtm.gt_attn_fwd(rp, ci, *fb, out_b, np.float32(0.2), stream=sb)
    grown = gtm.gt_workspace_pool_stats()[0]
    sa.synchronize()
    sb.synchronize()
    assert grown > one_block, "stream B took the block still pending on stream A"
    assert np.array_equal(to_host_f32(out_a), want_a)
    assert np.array_equal(to_host_f32(out_b), want_b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tuning", [None, "group_per_row", "small_light"])
def test_step_ordered_light_rows(dtype, tuning):
    """Narrow rows (four or more per wave) run their light rows in the
    partition's step order.  With every row light (hubs of a few hundred
    entries cross several index tiles and land in the last step class) and with
    a small light bound, the forward and GATv2 still match the oracle, and the
    order does not change a bit between repeated calls."""
    import bench
    N, H, D = 6000, 1, 32  # 128-byte fp32 rows, 64-byte bf16 rows: 8 and 16 rows per wave
    rowptr, colidx = synth.ragged_graph(50, N, max_deg=40, empty_frac=0.05,
                                        hubs={3: 900, 77: 400, 5000: 200, 5999: 65},
                                        dup_frac=0.05, shuffle=True)
    Q, K, V = synth.features(50, N, H, D, dtype)
    tu = {None: None, "group_per_row": bench.ABLATION_MODES["group_per_row"],
          "small_light": {"light_max_deg": 3, "heavy_min_deg": 300, "chunk_edges": 128,
                          "grid_blocks": 0}}[tuning]
    scale = np.float32(1 / math.sqrt(D))
    t = TOL_F32 if dtype == "f32" else TOL_BF16
    a = run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tu)
    assert np.array_equal(a, run_gpu(rowptr, colidx, Q, K, V, scale, tuning=tu))
    ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
    assert gate_error(a, ref, absagg) <= t
    from tests.test_gpu_gatv2 import attention_vector, run_gpu_gatv2
    att = attention_vector(50, H, D)
    g, _ = run_gpu_gatv2(rowptr, colidx, Q, K, att, 0.2, tuning=tu)
    gref, gabs, _ = oracle.gatv2_fwd(rowptr, colidx, Q, K, att, 0.2, want_lse=False)
    assert gate_error(g, gref, gabs) <= t


@pytest.mark.parametrize("N", [16384, 65536])
@pytest.mark.parametrize("kind", ["gt", "gatv2"])
def test_small_graph_short_chunks(kind, N):
    """Small power-law graphs take short chunks for their hub rows (a few
    hundred entries; on 16K nodes the largest hub is cut into the full 32
    chunks): the hubs and all other rows match the oracle under the
    default partition (every row)."""
    import paper_2605_31500_amd as m
    H, D = 4, 32
    rowptr, colidx = synth.chung_lu_graph(0, N)
    Q, K, V = synth.features(0, N, H, D, "f32")
    rows = np.arange(N, dtype=np.int64)
    assert np.diff(rowptr).max() > 32 * 192  # the largest hub has more entries than 32 short chunks hold
    dt = [to_device(x) for x in (rowptr, colidx, Q, K)]
    out = torch.empty_like(dt[2])
    if kind == "gt":
        m.gt_attn_fwd_ex(*dt, to_device(V), out, 0.25)
        ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, 0.25, rows=rows, want_lse=False)
    else:
        att = synth.normal(N, synth.STREAM_EXTRA + 9, (H, D), 1.0 / math.sqrt(D), "f32")
        m.gt_gatv2_fwd(dt[0], dt[1], dt[2], dt[3], to_device(att), 0.2, out)
        ref, absagg, _ = oracle.gatv2_fwd(rowptr, colidx, Q, K, att, 0.2, rows=rows, want_lse=False)
    torch.cuda.synchronize()
    got = to_host_f32(out)[rows]
    assert gate_error(got, ref, absagg) <= TOL_F32


def test_workspace_memory_comes_back_after_many_streams():
    """Calls on 50 streams created and dropped one after another: workspace
    blocks are not kept per stream (a block whose last use is done serves the
    next call on any stream), so the memory the library holds afterwards is
    bounded by its 256 MiB cache, not 50 workspaces; no block is held once
    the calls are done, and gt_workspace_release() returns all of it to the
    device.  Each call's workspace here is about 40 MB (short chunks give
    many partial states)."""
    import paper_2605_31500_amd as gtm
    N, H, D = 200_000, 4, 32
    rowptr, colidx = synth.chung_lu_graph(3, N)
    Q, K, V = synth.features(3, N, H, D, "f32")
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dev[2])
    tuning = {"light_max_deg": 2, "heavy_min_deg": 3, "chunk_edges": 64, "grid_blocks": 0}
    gtm.gt_attn_fwd_ex(*dev, out, np.float32(0.2), tuning=tuning)
    torch.cuda.synchronize()
    want = to_host_f32(out)
    # streams themselves hold some device memory in the runtime; create and
    # drop 50 first, so that the measurement below sees only the workspace
    for _ in range(50):
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            torch.zeros(1, device="cuda")
        s.synchronize()
        del s
    gtm.gt_workspace_release()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    assert gtm.gt_workspace_pool_stats() == (0, 0)
    for _ in range(50):
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            gtm.gt_attn_fwd_ex(*dev, out, np.float32(0.2), tuning=tuning, stream=s)
        s.synchronize()
        del s
    torch.cuda.synchronize()
    reserved, used = gtm.gt_workspace_pool_stats()
    print("pool after 50 streams: reserved %d MiB, used %d MiB" % (reserved >> 20, used >> 20), flush=True)
    assert used == 0 and 0 < reserved <= (256 << 20) + (64 << 20)
    held = free0 - torch.cuda.mem_get_info()[0]
    assert held <= (256 << 20) + (64 << 20), "held %d MiB after 50 streams" % (held >> 20)
    assert np.array_equal(to_host_f32(out), want)
    gtm.gt_workspace_release()
    torch.cuda.synchronize()
    assert gtm.gt_workspace_pool_stats() == (0, 0)
    back = free0 - torch.cuda.mem_get_info()[0]
    print("device memory not returned: %d MiB" % (back >> 20), flush=True)
    assert back <= (8 << 20), "%d MiB not returned" % (back >> 20)
