"""The C ABI from plain C: tests/c_caller.c includes include/gt_attn.h as
C11, takes the address of every entry point the header declares (so each one
must resolve at link time against libgtattn.so) and makes calls that fail
host-side validation, so it runs without a GPU."""
import os
import re
import shutil
import subprocess

import pytest

from tests.test_abi import declared_functions

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_caller.c")
PKG = os.path.join(ROOT, "paper_2605_31500_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_c_caller_lists_every_declared_function():
    listed = set(re.findall(r"\(any_fn\)(gt_[a-z0-9_]+)", open(SRC).read()))
    assert listed == set(declared_functions())


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_header_compiles_as_c_and_links(tmp_path):
    import paper_2605_31500_amd as gt
    gt.load_library()  # the in-tree library exists
    exe = str(tmp_path / "c_caller")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-isystem", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), SRC, "-o", exe,
           "-L", PKG, "-lgtattn", "-Wl,-rpath," + PKG, "-Wl,-rpath-link," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_caller ok" in r.stdout
