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
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(tri_selection),'
                   ' sizeof(tri_chain_args), sizeof(tri_stats), sizeof(tri_version_info),'
                   ' offsetof(tri_chain_args, pos), offsetof(tri_selection, key));return 0;}\n')
    exe = tmp_path / "sz"
    import subprocess
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [C.sizeof(L.Selection), C.sizeof(L.ChainArgs), C.sizeof(L.Stats),
            C.sizeof(L.VersionInfo), L.ChainArgs.pos.offset, L.Selection.key.offset]
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
