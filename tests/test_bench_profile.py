"""The rocprofv3 summary arithmetic of bench_profile.py on a synthetic capture
(CPU only): copy calibration, per-call byte counts, L2 hit rate, the traffic
entry bench.py reads, and the commands recorded in the summary."""
import csv
import json
import os

import pytest

import bench
import bench_profile as bp


def write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def counter_rows(kernel, values, dispatches=2):
    return [[kernel, c, v] for _ in range(dispatches) for c, v in values.items()]


@pytest.fixture
def capture(tmp_path, monkeypatch):
    out = tmp_path / "out"
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bp, "PROFILES", str(prof))
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    copy = "__amd_rocclr_copyBuffer"
    # the copy moves 1 GiB each way; its counters read half of that for fetch
    write_csv(str(out / "copycal/pmc_FETCH_SIZE/x_counter_collection.csv"), hdr,
              counter_rows(copy, {"FETCH_SIZE": 524288.0}))
    write_csv(str(out / "copycal/pmc_WRITE_SIZE/x_counter_collection.csv"), hdr,
              counter_rows(copy, {"WRITE_SIZE": 1048576.0}))
    k = "void (anonymous namespace)::gt_attn_kernel<float, 4, 32, 0>((anonymous namespace)::AttnParams)"
    other = "void (anonymous namespace)::gt_partition_kernel<4>((anonymous namespace)::PartParams)"
    d = out / "gt"
    write_csv(str(d / "trace/bench_kernel_stats.csv"),
              ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"],
              [[k, 10, 2000000, 200000, 90, 195000, 210000, 1], [other, 10, 100000, 10000, 10, 9000, 11000, 1]])
    groups = {"FETCH_SIZE": {"FETCH_SIZE": 1000.0}, "WRITE_SIZE": {"WRITE_SIZE": 100.0},
              "TCC_HIT_sum_TCC_MISS_sum": {"TCC_HIT_sum": 25.0, "TCC_MISS_sum": 75.0},
              "_".join(bp.SQ_GROUP): {"SQ_LDS_BANK_CONFLICT": 0.0, "SQ_LDS_IDX_ACTIVE": 10.0, "SQ_INSTS_LDS": 1.0,
                                      "SQ_INSTS_VALU": 256.0 * 100, "SQ_INSTS_VMEM_RD": 5.0, "SQ_WAVES": 64.0,
                                      "GRBM_GUI_ACTIVE": 8 * 200.0},
              "_".join(bp.TA_GROUP): {"TA_TA_BUSY_sum": 256.0 * 150, "TA_ADDR_STALLED_BY_TC_CYCLES_sum": 100.0,
                                      "GRBM_GUI_ACTIVE": 8 * 200.0},
              # per CU: 100 of 200 cycles stalled; 0.5 requests per CU-cycle at 300 cycles each
              "_".join(bp.TCP_GROUP): {"TCP_PENDING_STALL_CYCLES_sum": 256.0 * 100,
                                       "TCP_TCC_READ_REQ_sum": 256.0 * 100, "TCP_TCC_READ_REQ_LATENCY_sum": 256.0 * 100 * 300,
                                       "GRBM_GUI_ACTIVE": 8 * 200.0}}
    for g, vals in groups.items():
        write_csv(str(d / ("pmc_" + g) / "x_counter_collection.csv"), hdr,
                  counter_rows(k, vals) + counter_rows(other, {c: 1e9 for c in vals}))
    live = {"config": {"workload": "wl-test"},
            "roofline": {"algorithmic_bytes_per_launch": 2_000_000, "kernel_ms": 0.2, "kernel": "gt_attn_kernel"}}
    (d / "live.json").write_text("noise\n" + json.dumps(live) + "\n")
    return out, prof


def test_summary_arithmetic(capture):
    out, prof = capture
    name, entry = bp.summarize(str(out), "gt", "abcd")
    assert name == "gt_attn_kernel_wl-test"
    # fetch scale 2, write scale 1; only the named kernel's counters count
    assert entry["fetch_bytes_per_launch"] == 1000 * 1024 * 2
    assert entry["write_bytes_per_launch"] == 100 * 1024
    assert entry["hbm_bytes_per_launch"] == 1000 * 1024 * 2 + 100 * 1024
    assert entry["l2_hit_rate"] == 0.25 and entry["kernel_source_sha256_16"] == "abcd"
    tj = json.loads((prof / "traffic.json").read_text())
    assert tj["wl-test"] == entry
    text = (prof / (name + ".md")).read_text()
    assert "| `gt_attn_kernel<float, 4, 32, 0>` | 10 | 200.00 |" in text
    assert "VALU issue share" in text and "| 50.0 % |" in text  # 25600 / (256 x 1600/8)
    assert "texture-address unit busy" in text and "| 75.0 % |" in text  # 38400 / (256 x 200)
    assert "vector L1 stalled on data pending from L2" in text and "| 50.0 % |" in text
    assert "| 300 cycles |" in text           # latency sum / requests
    assert "| L1 misses in flight per CU (requests per CU-cycle × latency) | | 150 |" in text  # 0.5 x 300
    assert "-- python3 %s --steps 50" % bp.BENCH in text     # the program follows `--` directly
    assert "rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum" in text


def test_bench_reads_the_entry_only_for_matching_sources(capture, monkeypatch):
    out, prof = capture
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(prof / "traffic.json"))
    bp.summarize(str(out), "gt", "0000000000000000")  # taken on other sources
    assert bench.stored_traffic("wl-test") is None
    bp.summarize(str(out), "gt", bench.source_hash())
    assert bench.stored_traffic("wl-test") == 1000 * 1024 * 2 + 100 * 1024


def test_unknown_mode_is_refused():
    with pytest.raises(SystemExit):
        bp.main(["summarize", "nope"])
