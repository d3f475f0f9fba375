"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two drivers, each built here with the sanitizers and -fno-sanitize-recover
and run in a child process:
  * tests/sanitize/oracle_driver.c with oracle/gt_oracle.c and synth/synth.c
    (gcc, no OpenMP): every generator and every oracle function on small
    graphs with empty rows, repeated entries, a single row and row subsets;
  * tests/sanitize/abi_driver.cpp with the library source (hipcc, sanitizers
    on the host compilation only): every entry point's host validation,
    status strings, per-thread error messages, and the pool and profiler
    calls that need no device.
Builds are kept under _build/sanitize/, keyed by a hash of their sources."""
import hashlib
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "_build", "sanitize")
SAN = os.path.join(ROOT, "tests", "sanitize")


def cached_build(name, sources, cmd_of):
    h = hashlib.sha256()
    for src in sources:
        h.update(open(src, "rb").read())
    h.update(" ".join(cmd_of("X")).encode())
    exe = os.path.join(BUILD, "%s-%s" % (name, h.hexdigest()[:12]))
    if not os.path.exists(exe):
        os.makedirs(BUILD, exist_ok=True)
        tmp = exe + ".tmp%d" % os.getpid()
        r = subprocess.run(cmd_of(tmp), capture_output=True, text=True, timeout=900)
        if r.returncode != 0:
            raise AssertionError("build failed:\n" + (r.stdout + r.stderr)[-4000:])
        os.replace(tmp, exe)
    return exe


def run_clean(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert "0 failure(s)" in out


def test_oracle_and_generator_under_asan_ubsan():
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    srcs = [os.path.join(SAN, "oracle_driver.c"), os.path.join(ROOT, "oracle", "gt_oracle.c"),
            os.path.join(ROOT, "synth", "synth.c")]
    exe = cached_build("oracle_driver", srcs, lambda out: [
        "gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
        "-fno-sanitize-recover=all"] + srcs + ["-lm", "-o", out])
    run_clean(exe)


def test_library_host_code_under_asan_ubsan():
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    csrc = os.path.join(ROOT, "paper_2605_31500_amd", "csrc")
    srcs = [os.path.join(csrc, n) for n in sorted(os.listdir(csrc)) if n.endswith((".hip", ".hpp"))]
    srcs += [os.path.join(ROOT, "include", "gt_attn.h"), os.path.join(SAN, "abi_driver.cpp")]
    exe = cached_build("abi_driver", srcs, lambda out: [
        hipcc, "--offload-arch=gfx950", "-O0", "-std=c++17",
        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
        "-Xarch_host", "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
        os.path.join(csrc, "gt_attn.hip"), os.path.join(SAN, "abi_driver.cpp"), "-o", out])
    run_clean(exe)
