"""libtri.so loads and exports every entry point include/tri.h declares (CPU;
no compute call is made)."""
import ctypes as C
import os
import re

import pytest

from tests.native_libs import ROOT, ensure_libtri

HEADER = os.path.join(ROOT, "include", "tri.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tri_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("tri_spec_cache_create", "tri_rmsnorm", "tri_rope_qk", "tri_swiglu",
                 "tri_residual_rmsnorm", "tri_decode_chain"):
        assert must in names


def test_every_declared_symbol_is_exported():
    lib = C.CDLL(ensure_libtri())
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_declares_every_symbol():
    ensure_libtri()
    from paper_2609_37241_amd import _lib as L
    assert set(L.SIGNATURES) == set(declared_functions())


def test_binding_fails_loudly_without_the_library(tmp_path):
    ensure_libtri()
    from paper_2609_37241_amd import _lib as L
    with pytest.raises(ImportError):
        L.load(str(tmp_path / "libtri.so"))


def test_struct_layouts_match_the_header(tmp_path):
    from paper_2609_37241_amd import _lib as L
    src = tmp_path / "sz.c"
    src.write_text('#include "tri.h"\n#include <stdio.h>\n#include <stddef.h>\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu %zu %zu %d %d %d\\n",'
                   ' sizeof(tri_selection), sizeof(tri_chain_args), sizeof(tri_stats),'
                   ' sizeof(tri_version_info), offsetof(tri_chain_args, pos),'
                   ' offsetof(tri_selection, key), sizeof(tri_resident_info),'
                   ' offsetof(tri_resident_info, launches), TRI_RESIDENT_SLOTS,'
                   ' TRI_RESIDENT_MAX_GRID, TRI_RESIDENT_ANY_GRID_SLOTS);return 0;}\n')
    exe = tmp_path / "sz"
    import subprocess
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [C.sizeof(L.Selection), C.sizeof(L.ChainArgs), C.sizeof(L.Stats),
            C.sizeof(L.VersionInfo), L.ChainArgs.pos.offset, L.Selection.key.offset,
            C.sizeof(L.ResidentInfo), L.ResidentInfo.launches.offset, L.RESIDENT_SLOTS,
            L.RESIDENT_MAX_GRID, L.RESIDENT_ANY_GRID_SLOTS]
    assert got == want


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; --gpus N > 1 exits with status 2 and says
    so, before touching torch or a device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_host_cost_microbenchmark_runs():
    """The host-cost microbenchmark (library over a launch that does nothing)
    returns positive figures, and Algorithm 1's scan to the last of 4096
    versions costs clearly more than a scan of one version and than a
    lookup through the key memo."""
    import ctypes as C
    path = os.path.join(ROOT, "paper_2609_37241_amd", "libtri_hostcost.so")
    if not os.path.exists(path):
        import __graft_entry__
        __graft_entry__.build()
    lib = C.CDLL(path)
    ns = (C.c_int32 * 2)(1, 4096)
    out = (C.c_double * 8)()
    assert lib.trib_hostcost(ns, 2, out) == 0
    assert all(out[i] > 0 for i in (1, 2, 3, 4, 5, 6, 7))     # out[0] is a difference
    assert out[7] > 10 * out[6] and out[7] > 10 * out[3]
