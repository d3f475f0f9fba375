"""The bench line's contract, end to end on the GPU: one JSON line with the
metric, whole-call throughput, the roofline object of the attention kernel and
the oracle timed on the host (a short run of the default workload)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_default_bench_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1",
                        "--cpu-seconds", "0.5"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["metric"] == "fused graph-attention fwd GEdges/s at 1 MI355X; achieved HBM GB/s vs peak"
    assert line["unit"] == "GEdges/s" and line["value"] > 0 and line["n_gpus"] == 1
    assert line["steps"] == 3 and line["warmup"] == 1 and line["higher_is_better"] is True
    assert line["config"]["workload"] == "rmat-s21-h4d32-f32" and line["dtype"] == "f32"
    assert line["config"]["N"] == 2097152 and line["config"]["E"] == 50331648
    rf = line["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert 0 < rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-3)
    assert rf["traffic"] is None or rf["traffic"] > 0
    cb = line["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "GEdges/s" and cb["value"] > 0 and cb["cores"] >= 1
    assert "rows" in cb["sample"]
    st = cb["single_thread"]
    assert set(st) == {"er-2k-h1d32-f32", "chunglu-arxiv-169k-h4d32-f32"}
    assert all(v["seconds"] > 0 and v["GEdges_per_s"] > 0 for v in st.values())
    # the timed output, every row, against the oracle
    assert line["parity"]["rows"] == "all" and line["parity"]["tolerance"] == 1e-5
    assert 0 <= line["parity"]["gate_error"] <= 1e-5
    assert 0 < rf["whole_call_frac"] <= rf["frac"]
