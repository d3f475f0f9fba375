"""C-ABI library checks that need no GPU: the library loads, exports every
function include/gt_attn.h declares, and rejects bad arguments on the host
before any device work (every call here fails validation, so no pointer is
ever dereferenced and no kernel is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gt_attn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gt_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2605_31500_amd as gt
    return gt.load_library()


def test_exports_every_declared_symbol(lib):
    import paper_2605_31500_amd as gt
    names = declared_functions()
    assert set(names) == set(gt.EXPORTED_SYMBOLS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code in range(5):
        assert lib.gt_status_string(code)
    assert lib.gt_status_string(99) == b"unknown status"


FAKE = 0x10000  # never dereferenced: each call below fails validation first


def call(lib, dtype=0, rowptr=FAKE, colidx=FAKE, Q=FAKE, K=FAKE + 0x100000, V=FAKE + 0x200000,
         out=FAKE + 0x300000, lse=None, N=10, E=20, H=4, D=32, scale=0.1):
    P = ctypes.c_void_p
    return lib.gt_attn_fwd_ex(dtype, P(rowptr), P(colidx), P(Q), P(K), P(V), P(out), P(lse), N, E,
                              H, D, ctypes.c_float(scale), None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=3), 2), (dict(D=48), 2), (dict(D=512), 2), (dict(D=1024, dtype=1), 2),
    (dict(H=8, D=512, dtype=1), 2), (dict(dtype=7), 2),
    (dict(N=-1), 1), (dict(E=-5), 1), (dict(E=1 << 31), 1), (dict(N=1 << 31), 1),
    (dict(H=0), 1), (dict(scale=float("inf")), 1), (dict(scale=float("nan")), 1),
    (dict(rowptr=0), 1), (dict(colidx=0), 1), (dict(Q=0), 1), (dict(out=0), 1),
    (dict(K=FAKE + 8), 1),                      # misaligned
    (dict(out=FAKE + 0x200000 + 1024), 1),      # out overlaps V
    (dict(out=FAKE), 1),                        # out aliases Q
    (dict(lse=FAKE + 0x300000 + 4), 1),         # lse overlaps out
    (dict(lse=FAKE + 0x400002), 1),             # lse misaligned
])
def test_host_validation(lib, kw, status):
    assert call(lib, **kw) == status
    assert lib.gt_last_error_message()


@pytest.mark.parametrize("field", ["light_max_deg", "heavy_min_deg", "chunk_edges", "grid_blocks",
                                   "dense_tiles"])
def test_oversized_tuning_field_is_refused(lib, field):
    # a count near INT32_MAX would overflow the partition's rounding: refused
    # on the host, before any device work (the pointers are never touched)
    import paper_2605_31500_amd as gt
    P = ctypes.c_void_p
    for value, status in (((1 << 31) - 1, 1), ((1 << 31) - (1 << 16) + 1, 1)):
        tu = gt.GtTuning(**{field: value})
        assert lib.gt_attn_fwd_ex(0, P(FAKE), P(FAKE), P(FAKE), P(FAKE + 0x100000), P(FAKE + 0x200000),
                                  P(FAKE + 0x300000), None, 10, 20, 4, 32, ctypes.c_float(0.1),
                                  ctypes.byref(tu), None) == status
        assert b"tuning" in lib.gt_last_error_message()
        assert lib.gt_segment_reduce(0, 0, P(FAKE), P(FAKE), P(FAKE), P(FAKE + 0x100000),
                                     P(FAKE + 0x200000), 10, 20, 64, ctypes.byref(tu), None) == status


@pytest.mark.parametrize("kw,status", [(dict(H=3), 2), (dict(N=-1), 1), (dict(out=FAKE), 1),
                                       (dict(scale=float("nan")), 1)])
def test_noalloc_entry_host_validation(lib, kw, status):
    # the allocation-free entry point validates like gt_attn_fwd_ex
    a = dict(dtype=0, rowptr=FAKE, colidx=FAKE, Q=FAKE, K=FAKE + 0x100000, V=FAKE + 0x200000,
             out=FAKE + 0x300000, N=10, E=20, H=4, D=32, scale=0.1)
    a.update(kw)
    P = ctypes.c_void_p
    assert lib.gt_attn_fwd_noalloc(a["dtype"], P(a["rowptr"]), P(a["colidx"]), P(a["Q"]), P(a["K"]), P(a["V"]),
                                   P(a["out"]), None, a["N"], a["E"], a["H"], a["D"], ctypes.c_float(a["scale"]),
                                   None, None) == status
    assert lib.gt_last_error_message()


def test_empty_graph_is_a_no_op(lib):
    # N == 0 enqueues nothing and touches no pointer
    assert call(lib, N=0, E=0, rowptr=FAKE) == 0
    assert lib.gt_last_error_message() == b""


def test_profile_without_calls(lib):
    assert lib.gt_profile_enable(1) == 0
    ms = (ctypes.c_double * 3)()
    calls = ctypes.c_int64(-1)
    assert lib.gt_profile_collect(ms, ctypes.byref(calls)) == 0
    assert calls.value == 0 and list(ms) == [0.0, 0.0, 0.0]
    assert lib.gt_profile_enable(0) == 0


def test_binding_refuses_host_tensors():
    import torch
    import paper_2605_31500_amd as gt
    z = torch.zeros(3, 1, 32)
    with pytest.raises(ValueError):
        gt.gt_attn_fwd(torch.zeros(4, dtype=torch.int64), torch.zeros(0, dtype=torch.int32), z, z,
                       z, z, 0.1)


def call_gatv2(lib, dtype=0, rowptr=FAKE, colidx=FAKE, L=FAKE, R=FAKE + 0x100000,
               att=FAKE + 0x500000, slope=0.2, out=FAKE + 0x300000, lse=None, N=10, E=20, H=4,
               D=32):
    P = ctypes.c_void_p
    return lib.gt_gatv2_fwd(dtype, P(rowptr), P(colidx), P(L), P(R), P(att),
                            ctypes.c_float(slope), P(out), P(lse), N, E, H, D, None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=3), 2), (dict(D=16), 2), (dict(dtype=5), 2), (dict(N=-2), 1),
    (dict(att=0), 1),                           # null attention vector
    (dict(att=FAKE + 0x500004), 1),             # att misaligned
    (dict(slope=float("inf")), 1), (dict(slope=float("nan")), 1),
    (dict(att=FAKE + 0x300000 + 512), 1),       # att overlaps out
    (dict(L=0), 1), (dict(R=FAKE + 4), 1),
    (dict(out=FAKE + 0x100000), 1),             # out aliases R
])
def test_gatv2_host_validation(lib, kw, status):
    assert call_gatv2(lib, **kw) == status
    assert lib.gt_last_error_message()


def test_gatv2_empty_graph_is_a_no_op(lib):
    assert call_gatv2(lib, N=0, E=0) == 0


def call_reduce(lib, dtype=0, op=0, rowptr=FAKE, colidx=FAKE, X=FAKE, out=FAKE + 0x100000,
                arg=FAKE + 0x200000, N=10, E=20, F=64):
    P = ctypes.c_void_p
    return lib.gt_segment_reduce(dtype, op, P(rowptr), P(colidx), P(X), P(out), P(arg), N, E, F,
                                 None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(F=48), 2), (dict(F=8), 2), (dict(F=2048), 2), (dict(dtype=1, F=16), 2),
    (dict(dtype=1, F=4096), 2), (dict(op=2), 2), (dict(dtype=3), 2),
    (dict(N=-1), 1), (dict(E=-1), 1), (dict(F=0), 1),
    (dict(X=0), 1), (dict(out=0), 1), (dict(rowptr=0), 1), (dict(colidx=0), 1),
    (dict(X=FAKE + 4), 1),                      # misaligned
    (dict(arg=FAKE + 0x200008), 1),             # arg misaligned
    (dict(out=FAKE + 1024), 1),                 # out overlaps X
    (dict(arg=FAKE + 0x100000 + 256), 1),       # arg overlaps out
])
def test_reduce_host_validation(lib, kw, status):
    assert call_reduce(lib, **kw) == status
    assert lib.gt_last_error_message()


def test_reduce_empty_graph_is_a_no_op(lib):
    assert call_reduce(lib, N=0, E=0) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(F=48), 2), (dict(F=1024), 2), (dict(mapping=2), 2), (dict(load_bytes=8), 2),
    (dict(N=-1), 1), (dict(X=0), 1), (dict(out=0), 1), (dict(X=FAKE + 4), 1),
    (dict(out=FAKE + 2), 1), (dict(out=FAKE + 64), 1),   # misaligned out; out overlaps X
])
def test_dot_aggr_host_validation(lib, kw, status):
    a = dict(rowptr=FAKE, colidx=FAKE, X=FAKE, out=FAKE + 0x200000, N=10, E=20, F=64, mapping=0,
             load_bytes=16)
    a.update(kw)
    P = ctypes.c_void_p
    assert lib.gt_dot_aggr(P(a["rowptr"]), P(a["colidx"]), P(a["X"]), P(a["out"]), a["N"], a["E"],
                           a["F"], a["mapping"], a["load_bytes"], None) == status
    assert lib.gt_last_error_message()


def call_bwd(lib, dtype=0, rowptr=FAKE, colidx=FAKE, rowptr_t=FAKE, colidx_t=FAKE, Q=FAKE,
             K=FAKE + 0x100000, V=FAKE + 0x200000, out=FAKE + 0x300000, dout=FAKE + 0x400000,
             lse=FAKE + 0x500000, dQ=FAKE + 0x600000, dK=FAKE + 0x700000, dV=FAKE + 0x800000,
             N=10, E=20, H=4, D=32, scale=0.1):
    P = ctypes.c_void_p
    return lib.gt_attn_bwd(dtype, P(rowptr), P(colidx), P(rowptr_t), P(colidx_t), P(Q), P(K), P(V),
                           P(out), P(dout), P(lse), P(dQ), P(dK), P(dV), N, E, H, D,
                           ctypes.c_float(scale), None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2), (dict(H=3), 2), (dict(D=48), 2), (dict(dtype=1, H=8, D=512), 2),
    (dict(N=-1), 1), (dict(E=-1), 1), (dict(H=0), 1), (dict(scale=float("inf")), 1),
    (dict(rowptr_t=0), 1), (dict(colidx_t=0), 1), (dict(dout=0), 1),
    (dict(lse=0), 1), (dict(lse=FAKE + 0x500002), 1),          # lse null / misaligned
    (dict(dQ=0), 1), (dict(dK=FAKE + 0x700004), 1),            # gradient null / misaligned
    (dict(dQ=FAKE), 1),                                        # dQ aliases Q
    (dict(dV=FAKE + 0x700000 + 1024), 1),                      # dV overlaps dK
    (dict(dK=FAKE + 0x600000), 1),                             # dK is dQ (same pointer)
    (dict(dV=FAKE + 0x600000), 1),                             # dV is dQ
    (dict(dK=FAKE + 0x500000), 1),                             # dK overlaps lse
])
def test_bwd_host_validation(lib, kw, status):
    assert call_bwd(lib, **kw) == status
    assert lib.gt_last_error_message()


def test_bwd_empty_graph_is_a_no_op(lib):
    assert call_bwd(lib, N=0, E=0) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without the built library the binding raises; it has no other path."""
    import paper_2605_31500_amd as gt
    monkeypatch.setattr(gt, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        gt.load_library(str(tmp_path / "libgtattn.so"))


def test_product_sources_do_not_reach_the_oracle():
    """The package (binding and HIP sources) neither imports nor names the
    test oracle, so no product call can be served by it."""
    pkg = os.path.join(ROOT, "paper_2605_31500_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\boracle\b", text), os.path.join(dirpath, f)
    assert not re.search(r"\boracle\b", open(HEADER).read())
