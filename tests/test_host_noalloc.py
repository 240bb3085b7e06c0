"""CPU tests of the allocation-free entry point (tri_residual_rmsnorm_noalloc)
against the recording backend: it never installs, a split version takes the
GPU's fixed scratch instead of its own, calls beyond that scratch are
refused before anything is launched, and every other version launches
exactly as tri_residual_rmsnorm does. Expected selections come from the
oracle's selection model."""
import ctypes as C

import pytest

from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import res_call
from tests.test_host_cache import c_call, c_record, c_stats

BF, F = S.DT_BF16, S.DT_F32


@pytest.fixture(scope="module")
def lib():
    lib = load_fake()
    lib.trifake_noalloc_scratch.restype = C.c_void_p
    lib.trifake_noalloc_scratch.argtypes = [C.POINTER(C.c_int64)]
    return lib


@pytest.fixture
def fresh(lib):
    caches = []

    def make(flags=0):
        lib.trifake_reset()
        h = C.c_void_p()
        assert lib.tri_spec_cache_create(C.byref(h), 0, flags) == 0
        caches.append(h)
        return h
    yield make
    for h in caches:
        lib.tri_spec_cache_destroy(h)


def noalloc(lib, cache, c: S.Call, stream=None):
    p, s = c.ptr, c.stride
    return lib.tri_residual_rmsnorm_noalloc(cache, c.dtype, p.get("x"), s["x"], p.get("res"),
                                            s["res"], p.get("w"), p.get("y"), s["y"],
                                            p.get("res_out"), s["res_out"], c.T, c.H, c.eps,
                                            stream)


def last_launch(lib):
    kv, dt, sub = C.c_int32(), C.c_int32(), C.c_int32()
    grid, block, stream = C.c_uint32(), C.c_uint32(), C.c_void_p()
    buf = C.create_string_buffer(512)
    n = lib.trifake_get(lib.trifake_launch_count() - 1, C.byref(kv), C.byref(dt), C.byref(sub),
                        C.byref(grid), C.byref(block), C.byref(stream), buf, 512)
    return (kv.value, dt.value, sub.value, grid.value, block.value), buf.raw[:n]


def test_a_miss_installs_nothing_even_under_auto_install(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    c = res_call(BF, 5, 4096)
    assert noalloc(lib, cache, c) == S.MISS
    assert lib.trifake_launch_count() == 0
    assert c_stats(lib, cache) == (1, 0, 1, 0, 0, 0, 0)    # calls, hits, misses, ..., versions
    rec = c_record(lib, cache)
    assert rec[1] == S.MISS and rec[2] == -1 and rec[7] == S.make_key(c)
    # the recorded key installs like any other miss; then the call hits
    assert lib.tri_spec_install_last_miss(cache, None) == 0
    assert noalloc(lib, cache, c) == S.OK
    assert c_stats(lib, cache) == (2, 1, 1, 0, 0, 1, 1)


def test_a_version_without_split_launches_like_the_ordinary_entry(lib, fresh):
    cache = fresh()
    c = res_call(BF, 5, 4096, pad=64)
    assert c_call(lib, cache, c) == S.MISS and lib.tri_spec_install_last_miss(cache, None) == 0
    assert c_call(lib, cache, c, stream=0xAB0) == 0
    want, want_args = last_launch(lib)
    want_rec = c_record(lib, cache)
    assert noalloc(lib, cache, c, stream=0xAB0) == 0
    got, got_args = last_launch(lib)
    assert (got, got_args) == (want, want_args) and got[0] == S.RN_BLOCK[2]
    assert c_record(lib, cache) == want_rec


@pytest.mark.parametrize("dtype,H,T", [(BF, 65536, 3), (F, 20480, 7), (BF, 1048576, 2)])
def test_a_split_version_takes_the_fixed_scratch(lib, fresh, dtype, H, T):
    """Same kernel, grid, record and row arguments as the ordinary entry;
    only the scratch address differs: the fixed array instead of the
    version's own."""
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    c = res_call(dtype, T, H)
    assert c_call(lib, cache, c) == 0
    want, want_args = last_launch(lib)
    want_rec = c_record(lib, cache)
    assert want[0] == S.RN_SPLIT and len(want_args) == 96
    lookups = C.c_int64()
    fixed = lib.trifake_noalloc_scratch(C.byref(lookups))
    assert lookups.value == 1                  # looked up once, at cache creation
    assert noalloc(lib, cache, c) == 0
    got, got_args = last_launch(lib)
    assert got == want and got_args[:88] == want_args[:88]
    assert int.from_bytes(got_args[88:96], "little") == fixed
    assert int.from_bytes(want_args[88:96], "little") not in (0, fixed)
    assert c_record(lib, cache) == want_rec
    assert c_stats(lib, cache)[:4] == (2, 1, 1, 0)


def test_calls_beyond_the_fixed_scratch_are_refused(lib, fresh):
    """bf16 rows of 65536 split 4 ways: a call of T rows needs 8 + 5 T words
    of the 2^17-word array, so 26212 rows fit (131068 words) and 26213 do
    not (131073): UNSUPPORTED, nothing launched, counted as an error."""
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    words = S.NOALLOC_SCRATCH_BYTES // 8
    assert S.split_words(26212, 4) <= words < S.split_words(26213, 4)
    for T, want in ((26212, S.OK), (26213, S.E_UNSUPPORTED)):
        c = res_call(BF, T, 65536)
        assert c_call(lib, cache, c) == 0           # the ordinary entry (own scratch) installs
        n = lib.trifake_launch_count()
        before = c_stats(lib, cache)
        assert noalloc(lib, cache, c) == want
        assert lib.trifake_launch_count() == n + (want == S.OK)
        after = c_stats(lib, cache)
        assert after[3] - before[3] == (want != S.OK)


def test_errors_match_the_ordinary_entry(lib, fresh):
    cache = fresh()
    for c in (res_call(BF, 3, 4096, null=("res",)), res_call(BF, -1, 4096),
              res_call(BF, 3, 4096, eps=-1.0), res_call(F, 3, 1 << 24)):
        assert noalloc(lib, cache, c) == c_call(lib, cache, c) < 0
    assert noalloc(lib, cache, res_call(BF, 0, 4096)) == S.OK     # T = 0: no-op
    assert lib.tri_residual_rmsnorm_noalloc(None, BF, None, 0, None, 0, None, None, 0, None, 0,
                                            1, 8, 1e-6, None) == S.E_INVALID
    assert lib.trifake_launch_count() == 0
