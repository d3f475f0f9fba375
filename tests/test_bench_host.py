"""Host-side logic of bench.py: the byte models, the counter bookkeeping and
the one-GPU guard (no GPU needed)."""
import json
import os
import subprocess
import sys

import numpy as np

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_model_bytes_match_the_per_edge_formula():
    w = synth.config(0)
    R = w.H * w.D * 4
    want = 8 * (w.N + 1) + 4 * w.E + w.N * R + 2 * w.E * R + w.N * R
    assert bench.model_bytes(w) == want
    # GATv2 gathers one row per entry and reads the [H, D] fp32 attention vector
    assert bench.gatv2_model_bytes(w) == want - w.E * R + 4 * w.H * w.D
    assert bench.compulsory_bytes(w) == 8 * (w.N + 1) + 4 * w.E + 4 * w.N * R


def test_reduce_model_bytes():
    assert bench.reduce_model_bytes(10, 40, 16, 4) == 8 * 11 + 4 * 40 + 40 * 64 + 10 * 64 + 10 * 64


def test_source_hash_covers_every_hip_source(tmp_path, monkeypatch):
    h0 = bench.source_hash()
    assert len(h0) == 16 and h0 == bench.source_hash()
    d = tmp_path / "csrc"
    d.mkdir()
    (d / "a.hip").write_text("x")
    (d / "b.hpp").write_text("y")
    monkeypatch.setattr(bench, "KERNEL_SRC_DIR", str(d))
    h1 = bench.source_hash()
    (d / "b.hpp").write_text("z")  # a change in an included header changes the hash
    assert bench.source_hash() != h1
    (d / "notes.txt").write_text("ignored")
    h2 = bench.source_hash()
    (d / "notes.txt").write_text("still ignored")
    assert bench.source_hash() == h2


def test_stored_traffic_only_for_the_current_sources(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({"w": {"kernel_source_sha256_16": bench.source_hash(),
                                   "hbm_bytes_per_launch": 123},
                             "old": {"kernel_source_sha256_16": "0" * 16,
                                     "hbm_bytes_per_launch": 456}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.stored_traffic("w") == 123
    assert bench.stored_traffic("old") is None
    assert bench.stored_traffic("missing") is None


def test_committed_traffic_entries_are_well_formed():
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, e in rec.items():
        # each figure is a scaled counter truncated to whole bytes
        assert abs(e["hbm_bytes_per_launch"] - e["fetch_bytes_per_launch"] - e["write_bytes_per_launch"]) <= 1
        assert os.path.exists(os.path.join(ROOT, "profiles", e["summary"])), key


def test_ablation_modes_keep_heavy_above_light():
    for mode, tu in bench.ABLATION_MODES.items():
        assert tu["dense_tiles"] < 0, mode  # the partition alone is compared
        if "light_max_deg" in tu:
            assert tu["heavy_min_deg"] > tu["light_max_deg"] > 0, mode
            assert max(tu.values()) < 2 ** 31


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_paper_context_is_labelled():
    # the paper's ratios are quoted with their hardware and quantity, never as a target
    for key, ctx in bench.PAPER_CONTEXT.items():
        assert "A100" in ctx["hardware"] and "t_DGL / t" in ctx["quantity"], key


def test_cpu_baseline_parity_and_single_thread():
    """The CPU-baseline leg: its first oracle pass over all rows gives the gate
    error of a GPU output; here the output is the oracle's own, rounded to
    fp32, so the error is the fp32 rounding (<= 2^-24) and a planted error in
    one element is found."""
    import oracle
    w = synth.config(0)
    ref, _, _ = oracle.gt_attn_fwd(w.rowptr, w.colidx, w.Q, w.K, w.V, w.scale, want_absagg=False,
                                   want_lse=False)
    got = ref.astype(np.float32)
    res = bench.cpu_baseline(w, 0.05, got=got, single_thread_configs=(0,))
    assert 0 <= res["gate_error"] <= 2.0 ** -24
    cb = res["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1
    assert cb["single_thread"]["er-2k-h1d32-f32"]["seconds"] > 0
    assert oracle.threads() == cb["cores"]  # restored after the single-thread run
    got[123, 0, 7] += 1.0
    assert bench.cpu_baseline(w, 0.0, got=got)["gate_error"] > 0.1
