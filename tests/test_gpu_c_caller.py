"""The library from a standalone C program on the GPU (tests/c_caller_gpu.c):
no Python or torch in the process, device memory from the HIP runtime, the
contract entry points on the null stream, every output element against the
float64 oracle.  The program is compiled with gcc (host code only) before it
runs."""
import os
import shutil
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_caller_gpu.c")
PKG = os.path.join(ROOT, "paper_2605_31500_amd")
ORACLE = os.path.join(ROOT, "oracle")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_standalone_c_program_matches_the_oracle(tmp_path):
    import oracle
    import paper_2605_31500_amd as gt
    gt.load_library()
    oracle.threads()  # the oracle library is built
    exe = str(tmp_path / "c_caller_gpu")
    lib = os.path.join(ROCM, "lib")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-isystem", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), SRC, "-o", exe,
           "-L", PKG, "-lgtattn", "-L", ORACLE, "-lgt_oracle", "-L", lib, "-lamdhip64", "-lm",
           "-Wl,-rpath," + ":".join([PKG, ORACLE, lib])]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    print("c_caller_gpu built; running", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_caller_gpu ok" in r.stdout
