"""rocprofv3 capture and summaries for the bench modes.

    python bench_profile.py capture copycal gt gatv2 ...   # on a GPU machine
    python bench_profile.py summarize gt gatv2 ...         # anywhere, from the captures
    python bench_profile.py list

capture runs, for each named mode, bench.py once without the profiler (the
live line), once under `rocprofv3 --kernel-trace --stats`, and once under
`rocprofv3 --pmc` per counter group (the profiler collects one group per
pass).  `copycal` profiles a plain 1 GiB device copy with the two HBM byte
counters; its readings calibrate FETCH_SIZE and WRITE_SIZE.  Raw output goes
to OUT/<mode>/ (default captures/, kept out of version control).  Every GPU
run is a child process with its own time limit; this script never touches
the GPU, and it stops at the first run that fails.

summarize turns OUT/<mode>/ into profiles/<summary>.md (the commands, the
kernel table, the calibrated HBM bytes, the L2 hit rate, LDS bank conflicts
and the VALU issue share) and updates the mode's entry in
profiles/traffic.json, which bench.py reads as `roofline.traffic` while the
library sources still hash to the value recorded there.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import signal
import subprocess
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
PROFILES = os.path.join(ROOT, "profiles")

GT_MODEL = "per-edge model: rowptr + colidx + Q + K,V per CSR entry + out"
CAPTURES = {
    "gt": dict(args=[], kernels=["gt_attn_kernel"], key="{w}",
               title="Graph-transformer attention forward", model=GT_MODEL,
               summary="gt_attn_kernel_{w}"),
    "c1": dict(args=["--config", "1"], kernels=["gt_attn_kernel"], key="{w}",
               title="Graph-transformer attention forward", model=GT_MODEL, summary="gt_attn_kernel_{w}"),
    "gatv2": dict(args=["--gatv2", "--config", "1"], kernels=["gt_attn_kernel"], key="{w}:gatv2",
                  title="GATv2 attention forward",
                  model="per-edge model: rowptr + colidx + L + R per CSR entry + out + attention vector",
                  summary="gt_attn_kernel_gatv2_{w}"),
    # bf16 rows with H*D <= 128 run the dense-tile kernel (it finds no dense
    # window on R-MAT) before the CSR kernel: both are the attention phase
    "c2": dict(args=["--config", "2"], kernels=["gt_tile_kernel", "gt_attn_kernel"], key="{w}",
               title="Graph-transformer attention forward", model=GT_MODEL, summary="gt_attn_kernel_{w}"),
    "c3": dict(args=["--config", "3"], kernels=["gt_tile_kernel", "gt_attn_kernel"], key="{w}",
               title="Graph-transformer attention forward, dense tiles (default)", model=GT_MODEL,
               summary="gt_tile_kernel_{w}"),
    "c3csr": dict(args=["--config", "3", "--dense-tiles", "-1"], kernels=["gt_attn_kernel"], key="{w}:csr",
                  title="Graph-transformer attention forward, CSR kernel only (dense tiles off)", model=GT_MODEL,
                  summary="gt_attn_kernel_{w}-csr"),
    "c4": dict(args=["--config", "4"], kernels=["gt_attn_kernel"], key="{w}",
               title="Graph-transformer attention forward", model=GT_MODEL, summary="gt_attn_kernel_{w}"),
    "bwd": dict(args=["--backward", "--config", "1"], kernels=["gt_bwd_kernel"], key="{w}:backward",
                title="Graph-transformer attention backward (both passes)", model="backward per-edge model",
                summary="gt_bwd_kernel_{w}"),
    "reduce": dict(args=["--reduce", "min", "--config", "1"], kernels=["gt_reduce_kernel"], key="{g}:reduce-min-f512",
                   title="Segment min aggregation",
                   model="rowptr + colidx + one gathered row per entry + out + int32 sources",
                   summary="gt_reduce_kernel_{w}"),
}
SQ_GROUP = ["SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_INSTS_LDS", "SQ_INSTS_VALU", "SQ_INSTS_VMEM_RD",
            "SQ_WAVES", "GRBM_GUI_ACTIVE"]
TA_GROUP = ["TA_TA_BUSY_sum", "TA_ADDR_STALLED_BY_TC_CYCLES_sum", "GRBM_GUI_ACTIVE"]
# vector L1: cycles stalled on data pending from L2, its requests to L2 and their summed latency
# (cycles), for the misses it holds in flight (Little's law)
TCP_GROUP = ["TCP_PENDING_STALL_CYCLES_sum", "TCP_TCC_READ_REQ_sum", "TCP_TCC_READ_REQ_LATENCY_sum",
             "GRBM_GUI_ACTIVE"]
COUNTER_GROUPS = [["FETCH_SIZE"], ["WRITE_SIZE"], ["TCC_HIT_sum", "TCC_MISS_sum"], SQ_GROUP, TA_GROUP, TCP_GROUP]
COPY_MIB = 1024
N_XCD, N_CU = 8, 256

BENCH = os.path.join(ROOT, "bench.py")
LIVE_TAIL = ["--steps", "50", "--warmup", "10", "--no-cpu-baseline"]
PMC_TAIL = ["--steps", "5", "--warmup", "1", "--no-cpu-baseline"]


def group_dir(group):
    return "pmc_" + "_".join(group)


def trace_cmd(out, mode):
    return (["rocprofv3", "--kernel-trace", "--stats", "--output-format", "csv", "-d",
             os.path.join(out, mode, "trace"), "-o", "bench", "--", "python3", BENCH]
            + CAPTURES[mode]["args"] + LIVE_TAIL)


def pmc_cmd(out, mode, group):
    return (["rocprofv3", "--pmc"] + group + ["--output-format", "csv", "-d",
                                              os.path.join(out, mode, group_dir(group)), "-o", "bench", "--",
                                              "python3", BENCH] + CAPTURES[mode]["args"] + PMC_TAIL)


def copy_cmd(out, counter):
    return ["rocprofv3", "--pmc", counter, "--output-format", "csv", "-d",
            os.path.join(out, "copycal", "pmc_" + counter), "-o", "copy", "--", "python3", BENCH,
            "--copy-calibration", str(COPY_MIB), "--steps", "5"]


def shown(cmd, limit):
    # the form recorded in the summaries: profiler runs from /tmp with TMPDIR
    # there, each under its own time limit
    return "cd /tmp && export TMPDIR=/tmp && timeout -s KILL %d %s" % (limit, " ".join(cmd))


def run(cmd, limit, out_path, cwd=None, env=None, stderr_to_out=True):
    """Runs cmd in a session of its own; past the time limit the whole process
    group (the profiler and the program under it) is killed."""
    print("step: " + " ".join(cmd), flush=True)
    with open(out_path, "w") as f:
        p = subprocess.Popen(cmd, stdout=f, stderr=subprocess.STDOUT if stderr_to_out else subprocess.DEVNULL,
                             cwd=cwd, env=env, start_new_session=True)
        try:
            rc = p.wait(timeout=limit)
        except subprocess.TimeoutExpired:
            os.killpg(p.pid, signal.SIGKILL)
            p.wait()
            raise SystemExit("time limit (%d s) reached: %s" % (limit, out_path))
    if rc != 0:
        raise SystemExit("exit status %d: %s" % (rc, out_path))


def capture(out, modes):
    env = dict(os.environ, TMPDIR="/tmp")
    for mode in modes:
        if mode == "copycal":
            os.makedirs(os.path.join(out, "copycal"), exist_ok=True)
            for c in ("FETCH_SIZE", "WRITE_SIZE"):
                run(copy_cmd(out, c), 120, os.path.join(out, "copycal", "pmc_%s.out" % c), "/tmp", env)
            continue
        d = os.path.join(out, mode)
        os.makedirs(d, exist_ok=True)
        run(["python3", BENCH] + CAPTURES[mode]["args"] + LIVE_TAIL, 240, os.path.join(d, "live.json"),
            stderr_to_out=False)
        run(trace_cmd(out, mode), 300, os.path.join(d, "trace.out"), "/tmp", env)
        for g in COUNTER_GROUPS:
            run(pmc_cmd(out, mode, g), 120, os.path.join(d, group_dir(g) + ".out"), "/tmp", env)
        print("done: " + mode, flush=True)


# ------------------------------------------------------------------ summaries

def rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def one(pattern):
    found = sorted(glob.glob(pattern))
    if not found:
        raise SystemExit("missing capture output: " + pattern)
    return found[0]


def short(name):
    n = name.replace("(anonymous namespace)::", "")
    if n.startswith("void "):
        n = n[5:]
    return n.split("(")[0] if "(" in n else n


def copy_scales(out):
    """FETCH_SIZE and WRITE_SIZE (KiB) of the plain copy, and the factors that
    turn each into bytes moved."""
    vals = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        f = one(os.path.join(out, "copycal", "pmc_" + c, "*_counter_collection.csv"))
        v = [float(r["Counter_Value"]) for r in rows(f) if r["Counter_Name"] == c and "copyBuffer" in r["Kernel_Name"]]
        if not v:
            raise SystemExit("no copy dispatch in " + f)
        vals[c] = sum(v) / len(v)
    kib = COPY_MIB * 1024
    return vals["FETCH_SIZE"], vals["WRITE_SIZE"], kib / vals["FETCH_SIZE"], kib / vals["WRITE_SIZE"]


def kernel_table(trace_dir, kernels):
    stats = rows(one(os.path.join(trace_dir, "*_kernel_stats.csv")))
    total = sum(float(r["TotalDurationNs"]) for r in stats)
    table = [(short(r["Name"]), int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
              float(r["MaxNs"]) / 1e3, 100 * float(r["TotalDurationNs"]) / total,
              any(short(r["Name"]).startswith(k) for k in kernels)) for r in stats]
    return table


def counters(d, group, kernels):
    """Per call: each counter summed over the named kernels (each kernel's
    dispatches averaged); also the dispatch count averaged."""
    per = {}
    for r in rows(one(os.path.join(d, group_dir(group), "*_counter_collection.csv"))):
        if not any(short(r["Kernel_Name"]).startswith(k) for k in kernels):
            continue
        per.setdefault((short(r["Kernel_Name"]), r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    out, n = {}, 0
    for (_, c), v in per.items():
        out[c] = out.get(c, 0.0) + sum(v) / len(v)
        n = max(n, len(v))
    missing = [c for c in group if c not in out]
    if missing:
        raise SystemExit("counters %s missing in %s" % (missing, d))
    return out, n


def summarize(out, mode, source_hash):
    spec = CAPTURES[mode]
    d = os.path.join(out, mode)
    with open(os.path.join(d, "live.json")) as f:
        live = json.loads(f.read().strip().splitlines()[-1])
    w = live["config"]["workload"]
    g = live["config"].get("graph", w)
    name = spec["summary"].format(w=w)
    kernels = spec["kernels"]
    table = kernel_table(os.path.join(d, "trace"), kernels)
    main = [k for k in table if k[6]]
    if not main:
        raise SystemExit("no %s dispatch in the trace of %s" % (kernels, mode))
    kavg = sum(k[2] for k in main)  # per call: the named kernels' average durations, summed
    cf, cw, fscale, wscale = copy_scales(out)
    fetch, nd = counters(d, ["FETCH_SIZE"], kernels)
    write, _ = counters(d, ["WRITE_SIZE"], kernels)
    l2, _ = counters(d, ["TCC_HIT_sum", "TCC_MISS_sum"], kernels)
    sq, _ = counters(d, SQ_GROUP, kernels)
    ta, _ = counters(d, TA_GROUP, kernels)
    tcp, _ = counters(d, TCP_GROUP, kernels)
    fb = fetch["FETCH_SIZE"] * 1024 * fscale
    wb = write["WRITE_SIZE"] * 1024 * wscale
    alg = live["roofline"]["algorithmic_bytes_per_launch"]
    hit = l2["TCC_HIT_sum"] / max(l2["TCC_HIT_sum"] + l2["TCC_MISS_sum"], 1.0)
    cycles = sq["GRBM_GUI_ACTIVE"] / N_XCD
    valu = sq["SQ_INSTS_VALU"] / (N_CU * cycles)
    conf = sq["SQ_LDS_BANK_CONFLICT"] / max(sq["SQ_LDS_IDX_ACTIVE"] - sq["SQ_LDS_BANK_CONFLICT"], 1.0)
    ta_cycles = ta["GRBM_GUI_ACTIVE"] / N_XCD
    ta_busy = ta["TA_TA_BUSY_sum"] / (N_CU * ta_cycles)  # one texture-address unit per CU
    tcp_cycles = tcp["GRBM_GUI_ACTIVE"] / N_XCD
    pending = tcp["TCP_PENDING_STALL_CYCLES_sum"] / (N_CU * tcp_cycles)  # one vector L1 per CU
    l1_lat = tcp["TCP_TCC_READ_REQ_LATENCY_sum"] / max(tcp["TCP_TCC_READ_REQ_sum"], 1.0)
    in_flight = tcp["TCP_TCC_READ_REQ_sum"] / (N_CU * tcp_cycles) * l1_lat
    kl = " + ".join("`%s`" % k[0] for k in main)
    L = ["# %s on %s" % (spec["title"], w), "",
         "Library sources (`paper_2605_31500_amd/csrc/*.hip`, `*.hpp`), sha256[:16] as computed by "
         "`bench.source_hash()` = `%s`. Written by `bench_profile.py summarize %s` from the output of "
         "`bench_profile.py capture %s`." % (source_hash, mode, mode), "",
         "## Kernel trace (`rocprofv3 --kernel-trace --stats`)", "", "```", shown(trace_cmd(out, mode), 300), "```",
         "", "| kernel | calls | average µs | min µs | max µs | share |", "|---|---|---|---|---|---|"]
    L += ["| `%s` | %d | %.2f | %.2f | %.2f | %.1f %% |" % k[:6] for k in table]
    L += ["", "Live measurement by `bench.py` with the same arguments, run without the profiler on the same box "
              "just before: %.2f µs per call for %s (HIP events on the launch stream); rocprofv3 average: %.2f µs."
          % (live["roofline"]["kernel_ms"] * 1e3, live["roofline"]["kernel"], kavg), "",
          "## Counters (`rocprofv3 --pmc`, one pass per group)", "", "```"]
    L += [shown(pmc_cmd(out, mode, grp), 120) for grp in COUNTER_GROUPS]
    L += [shown(copy_cmd(out, c), 120) for c in ("FETCH_SIZE", "WRITE_SIZE")]
    L += ["```", "",
          "Calibration: a plain %d MiB device copy (`__amd_rocclr_copyBuffer`) reads FETCH_SIZE = %.0f KiB and "
          "WRITE_SIZE = %.0f KiB per dispatch for %d KiB moved each way, so the scale factors are %.4f (fetch) "
          "and %.4f (write)." % (COPY_MIB, cf, cw, COPY_MIB * 1024, fscale, wscale), "",
          "| per call of %s (%d dispatches averaged per kernel) | counter | value |" % (kl, nd), "|---|---|---|",
          "| HBM fetch | FETCH_SIZE %.0f KiB × %.4f | %.4f GB |" % (fetch["FETCH_SIZE"], fscale, fb / 1e9),
          "| HBM write | WRITE_SIZE %.0f KiB × %.4f | %.4f GB |" % (write["WRITE_SIZE"], wscale, wb / 1e9),
          "| HBM total | | %.4f GB |" % ((fb + wb) / 1e9),
          "| L2 hit rate | TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum) = %.0f / %.0f | %.1f %% |"
          % (l2["TCC_HIT_sum"], l2["TCC_HIT_sum"] + l2["TCC_MISS_sum"], 100 * hit),
          "| LDS bank conflicts | SQ_LDS_BANK_CONFLICT %.0f / (SQ_LDS_IDX_ACTIVE %.0f − conflicts) | %.3f |"
          % (sq["SQ_LDS_BANK_CONFLICT"], sq["SQ_LDS_IDX_ACTIVE"], conf),
          "| VALU issue share | SQ_INSTS_VALU %.3g / (%d CUs × GRBM_GUI_ACTIVE %.3g / %d XCDs) | %.1f %% |"
          % (sq["SQ_INSTS_VALU"], N_CU, sq["GRBM_GUI_ACTIVE"], N_XCD, 100 * valu),
          "| LDS instructions, vector-memory reads, waves | SQ_INSTS_LDS, SQ_INSTS_VMEM_RD, SQ_WAVES | "
          "%.3g, %.3g, %.0f |" % (sq["SQ_INSTS_LDS"], sq["SQ_INSTS_VMEM_RD"], sq["SQ_WAVES"]),
          "| texture-address unit busy | TA_TA_BUSY_sum %.3g / (%d CUs × GRBM_GUI_ACTIVE %.3g / %d XCDs) | %.1f %% |"
          % (ta["TA_TA_BUSY_sum"], N_CU, ta["GRBM_GUI_ACTIVE"], N_XCD, 100 * ta_busy),
          "| texture-address stalls on the cache | TA_ADDR_STALLED_BY_TC_CYCLES_sum / TA_TA_BUSY_sum | %.3f |"
          % (ta["TA_ADDR_STALLED_BY_TC_CYCLES_sum"] / max(ta["TA_TA_BUSY_sum"], 1.0)),
          "| vector L1 stalled on data pending from L2 | TCP_PENDING_STALL_CYCLES_sum %.3g / (%d CUs × cycles) | "
          "%.1f %% |" % (tcp["TCP_PENDING_STALL_CYCLES_sum"], N_CU, 100 * pending),
          "| L1 → L2 read latency | TCP_TCC_READ_REQ_LATENCY_sum / TCP_TCC_READ_REQ_sum (%.3g requests) | "
          "%.0f cycles |" % (tcp["TCP_TCC_READ_REQ_sum"], l1_lat),
          "| L1 misses in flight per CU (requests per CU-cycle × latency) | | %.0f |" % in_flight, "",
          "Algorithmic bytes per call (%s): %.4f GB; measured HBM / algorithmic = %.3f. FETCH_SIZE counts L2 "
          "misses sent to the fabric, which the 256 MB Infinity Cache may serve, so it bounds DRAM reads from "
          "above. The VALU share counts one wave-level VALU instruction per CU per cycle as the issue limit "
          "(fp32 FMA without packed math)." % (spec["model"], alg / 1e9, (fb + wb) / alg), "",
          "At the rocprofv3 average: the counted bytes move at %.0f GB/s (%.1f %% of 8 TB/s); the "
          "algorithmic bytes correspond to %.0f GB/s." % ((fb + wb) / (kavg * 1e-6) / 1e9,
                                                         100 * (fb + wb) / (kavg * 1e-6) / 8e12,
                                                         alg / (kavg * 1e-6) / 1e9)]
    if alg / (kavg * 1e-6) > 8e12:
        L += ["", "The algorithmic rate is above the 8 TB/s HBM peak: the per-edge model charges every gathered "
                  "row to HBM, while L2 and the Infinity Cache serve the repeated ones. It counts cache-served "
                  "bytes and is not a fraction of HBM bandwidth; the counted bytes are the one to compare with "
                  "the peak."]
    with open(os.path.join(PROFILES, name + ".md"), "w") as f:
        f.write("\n".join(L) + "\n")
    entry = None
    if spec["key"]:
        entry = {"kernel": ",".join(kernels), "kernel_source_sha256_16": source_hash,
                 "fetch_bytes_per_launch": int(fb), "write_bytes_per_launch": int(wb),
                 "hbm_bytes_per_launch": int(fb) + int(wb), "fetch_scale": round(fscale, 4),
                 "write_scale": round(wscale, 4), "l2_hit_rate": round(hit, 4), "summary": name + ".md"}
        tf = os.path.join(PROFILES, "traffic.json")
        try:
            with open(tf) as f:
                tj = json.load(f)
        except (OSError, ValueError):
            tj = {}
        tj[spec["key"].format(w=w, g=g)] = entry
        with open(tf, "w") as f:
            json.dump(tj, f, indent=1, sort_keys=True)
    print("%-55s kernel %9.2f us  HBM %.3f GB  HBM/model %.3f  L2 hit %.3f  VALU %.2f  TA %.2f  LDS conflicts %.3f"
          "  L1 pending %.2f  in flight %.0f  latency %.0f"
          % (name, kavg, (fb + wb) / 1e9, (fb + wb) / alg, hit, valu, ta_busy, conf, pending, in_flight, l1_lat),
          flush=True)
    return name, entry


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("action", choices=["capture", "summarize", "list"])
    ap.add_argument("modes", nargs="*", help="capture modes (or 'all'); capture also takes 'copycal'")
    ap.add_argument("--out", default=os.path.join(ROOT, "captures"), help="raw capture directory")
    a = ap.parse_args(argv)
    if a.action == "list":
        for m, s in CAPTURES.items():
            print("%-8s bench.py %s" % (m, " ".join(s["args"])))
        return 0
    modes = list(CAPTURES) if a.modes in ([], ["all"]) else a.modes
    for m in modes:
        if m not in CAPTURES and not (a.action == "capture" and m == "copycal"):
            raise SystemExit("unknown mode %r (see: bench_profile.py list)" % m)
    if a.action == "capture":
        capture(os.path.abspath(a.out), modes)
    else:
        sys.path.insert(0, ROOT)
        import bench
        h = bench.source_hash()
        for m in modes:
            summarize(os.path.abspath(a.out), m, h)
    return 0


if __name__ == "__main__":
    sys.exit(main())
