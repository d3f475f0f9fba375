"""The allocation-free entry point gt_attn_fwd_noalloc (workspace in the
library's per-device scratch array) against gt_attn_fwd_ex, through the C
ABI: bit-identical outputs on two calls in a row, the second on a smaller
graph, for fp32 and bf16 features with lse; the pool of the allocating entry
points is not touched; a problem whose workspace exceeds the scratch array is
refused before any launch."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.helpers import TOL_BF16, TOL_F32, gate_error, to_device, to_host_f32

pytestmark = pytest.mark.gpu


def run_both(rowptr, colidx, Q, K, V, scale, tuning=None):
    import paper_2605_31500_amd as gt
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    N, H = Q.shape[:2]
    outs = []
    for fn in (gt.gt_attn_fwd_ex, gt.gt_attn_fwd_noalloc):
        out = torch.empty_like(dev[2])
        lse = torch.empty((N, H), dtype=torch.float32, device=dev[2].device)
        fn(*dev, out, scale, tuning=tuning, lse=lse)
        torch.cuda.synchronize()
        outs.append((to_host_f32(out), lse.cpu().numpy()))
    return outs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_generic_entry_two_calls(dtype):
    import paper_2605_31500_amd as gt
    H, D = 4, 32
    scale = np.float32(1 / math.sqrt(D))
    big = synth.ragged_graph(61, 60_000, max_deg=90, empty_frac=0.05,
                             hubs={3: 59_999, 4: 30_000, 9000: 5000}, self_loops=True)
    small = synth.ragged_graph(62, 7_000, max_deg=40, empty_frac=0.1, hubs={1: 6999}, self_loops=True)
    pool_before = gt.gt_workspace_pool_stats()
    for (rowptr, colidx), seed in ((big, 61), (small, 62)):
        N = rowptr.size - 1
        print("graph N", N, "E", colidx.size, dtype, flush=True)
        Q, K, V = synth.features(seed, N, H, D, dtype)
        (ox, lx), (on, ln) = run_both(rowptr, colidx, Q, K, V, scale)
        assert np.array_equal(on, ox) and np.array_equal(ln, lx)
        ref, absagg, _ = oracle.gt_attn_fwd(rowptr, colidx, Q, K, V, scale, want_lse=False)
        assert gate_error(on, ref, absagg) <= (TOL_F32 if dtype == "f32" else TOL_BF16)
    torch.cuda.synchronize()
    # the allocating calls above may have grown the pool; the allocation-free
    # calls leave nothing in use in it
    assert gt.gt_workspace_pool_stats()[1] == 0 and pool_before[1] == 0


def test_noalloc_forced_split_and_tiles():
    # many chunk partials (split rows) and, in bf16, the dense-tile kernel
    H, D = 2, 64
    rowptr, colidx = synth.sbm_graph(63, 64 * 40 + 17, 64, 4)
    N = rowptr.size - 1
    Q, K, V = synth.features(63, N, H, D, "bf16")
    for tuning in ({"light_max_deg": 2, "heavy_min_deg": 6, "chunk_edges": 64, "grid_blocks": 0},
                   {"dense_tiles": 256}):
        (ox, lx), (on, ln) = run_both(rowptr, colidx, Q, K, V, np.float32(0.125), tuning=tuning)
        assert np.array_equal(on, ox) and np.array_equal(ln, lx)


def test_noalloc_refuses_workspace_beyond_scratch():
    import paper_2605_31500_amd as gt
    # 100K rows of 200 entries with 64-entry chunks: about 340 MB of chunk
    # partial states, more than the 256 MiB scratch array
    N, deg = 100_000, 200
    rowptr = np.arange(N + 1, dtype=np.int64) * deg
    colidx = (np.arange(N * deg, dtype=np.int64) % N).astype(np.int32)
    Q = np.zeros((N, 4, 32), dtype=np.float32)
    dev = [to_device(x) for x in (rowptr, colidx, Q, Q, Q)]
    out = torch.empty_like(dev[2])
    with pytest.raises(gt.GtError) as ei:
        gt.gt_attn_fwd_noalloc(*dev, out, 0.1, tuning={"chunk_edges": 64, "heavy_min_deg": 100})
    assert ei.value.status == gt.GT_ERROR_INVALID_VALUE and "scratch" in str(ei.value)
    # the same call through the allocating entry point runs
    gt.gt_attn_fwd_ex(*dev, out, 0.1, tuning={"chunk_edges": 64, "heavy_min_deg": 100})
    torch.cuda.synchronize()
    assert np.all(to_host_f32(out) == 0)


def test_noalloc_calls_leave_device_memory_unchanged():
    import paper_2605_31500_amd as gt
    rowptr, colidx = synth.ragged_graph(64, 20_000, max_deg=60, hubs={2: 19_999}, self_loops=True)
    Q, K, V = synth.features(64, 20_000, 4, 32, "f32")
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out = torch.empty_like(dev[2])
    gt.gt_attn_fwd_noalloc(*dev, out, 0.2)  # the library's code object (and its scratch array) is loaded
    torch.cuda.synchronize()
    free0, pool0 = torch.cuda.mem_get_info()[0], gt.gt_workspace_pool_stats()
    for _ in range(3):
        gt.gt_attn_fwd_noalloc(*dev, out, 0.2)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0 and gt.gt_workspace_pool_stats() == pool0


def test_noalloc_replays_in_a_hip_graph():
    """The allocation-free entry point recorded into a HIP graph (torch's
    graph capture on its capture stream) and replayed three times, with an
    eager call of the same entry point on another graph between the replays
    (it reuses the scratch array): every replay equals the eager result.  The
    call records only kernels, no memset or allocation."""
    import paper_2605_31500_amd as gt
    H, D = 4, 32
    rowptr, colidx = synth.ragged_graph(65, 30_000, max_deg=70, hubs={3: 29_999, 8: 9000}, self_loops=True)
    Q, K, V = synth.features(65, 30_000, H, D, "bf16")
    dev = [to_device(x) for x in (rowptr, colidx, Q, K, V)]
    out_eager = torch.empty_like(dev[2])
    gt.gt_attn_fwd_noalloc(*dev, out_eager, 0.2)
    torch.cuda.synchronize()
    want = to_host_f32(out_eager)
    rp2, ci2 = synth.ragged_graph(66, 5_000, max_deg=40, hubs={1: 4999}, self_loops=True)
    Q2, K2, V2 = synth.features(66, 5_000, H, D, "bf16")
    dev2 = [to_device(x) for x in (rp2, ci2, Q2, K2, V2)]
    out2 = torch.empty_like(dev2[2])
    gt.gt_attn_fwd_noalloc(*dev2, out2, 0.2)
    torch.cuda.synchronize()
    want2 = to_host_f32(out2)

    out = torch.empty_like(dev[2])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on a side stream before capture, as torch asks
        gt.gt_attn_fwd_noalloc(*dev, out, 0.2)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        gt.gt_attn_fwd_noalloc(*dev, out, 0.2)
    for _ in range(3):
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(to_host_f32(out), want)
        out2.zero_()
        gt.gt_attn_fwd_noalloc(*dev2, out2, 0.2)
        torch.cuda.synchronize()
        assert np.array_equal(to_host_f32(out2), want2)
