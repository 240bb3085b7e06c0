"""Several processes compile and tune into one code directory at once (CPU,
recording backend).

Six processes each make a cache with auto-install, compiled specializations
and install-time tuning on one shared code directory, meet at a barrier and
make the same calls. Afterwards the directory must hold exactly the files a
single process writes, each whole and with the same content, and no
temporary file; a fresh cache then loads every object and every stored
choice without compiling or timing.
"""
import ctypes as C
import multiprocessing as mp
import os

from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import chain_call, elem_offset, rn_call, sw_call
from tests.test_host_cache import c_call

BF, F = S.DT_BF16, S.DT_F32
FLAGS = S.FLAG_AUTO_INSTALL | S.FLAG_JIT | S.FLAG_AUTOTUNE
N_PROC = 6


def calls():
    return [chain_call(BF, 1, 4096, 11008, 32, 32, 128),
            chain_call(BF, 2, 4096, 14336, 32, 8, 128, rope_off=elem_offset(BF)),  # 3 launches
            rn_call(F, 3, 4096), sw_call(BF, 100, 11008)]


def _run(lib, code_dir):
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), 0, FLAGS) == 0
    try:
        assert lib.tri_spec_set_code_dir(h, str(code_dir).encode()) == 0
        for c in calls():
            assert c_call(lib, h, c) == 0
        from paper_2609_37241_amd._lib import VersionInfo
        infos = []
        for i in range(len(calls())):
            v = VersionInfo()
            assert lib.tri_spec_version_info(h, i, C.byref(v)) == 0
            infos.append((v.jit, v.tuned, v.candidate))
        return infos
    finally:
        lib.tri_spec_cache_destroy(h)


def _worker(code_dir, barrier, results):
    try:
        lib = load_fake()
        lib.trifake_reset()
        barrier.wait(timeout=120)
        _run(lib, code_dir)
        results.put(("ok", os.getpid()))
    except BaseException as e:  # noqa: BLE001 - reported to the parent
        results.put(("error", repr(e)))


def _files(d):
    return {p: open(os.path.join(d, p), "rb").read() for p in sorted(os.listdir(d))}


def test_processes_share_one_code_directory(tmp_path):
    lib = load_fake()                         # built before any child loads it
    ref, shared = tmp_path / "single", tmp_path / "shared"
    ref.mkdir()
    shared.mkdir()
    lib.trifake_reset()
    _run(lib, ref)
    want = _files(ref)
    assert any(n.endswith(".co") for n in want) and any(n.startswith("tri-tune-") for n in want)

    ctx = mp.get_context("spawn")
    barrier, results = ctx.Barrier(N_PROC), ctx.Queue()
    procs = [ctx.Process(target=_worker, args=(str(shared), barrier, results))
             for _ in range(N_PROC)]
    for p in procs:
        p.start()
    got = [results.get(timeout=300) for _ in procs]
    for p in procs:
        p.join(timeout=60)
    assert all(r[0] == "ok" for r in got), got
    assert all(p.exitcode == 0 for p in procs)
    assert _files(shared) == want             # same names, whole files, nothing temporary

    lib.trifake_reset()
    infos = _run(lib, shared)
    assert lib.trifake_compile_count() == 0
    assert all(jit == 2 for jit, _, _ in infos)                      # every object loaded
    assert all(tuned in (S.TUNE_NONE, S.TUNE_STORED) for _, tuned, _ in infos)
    assert any(tuned == S.TUNE_STORED for _, tuned, _ in infos)
