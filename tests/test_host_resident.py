"""Resident argument blocks (TRI_CACHE_RESIDENT_ARGS) on the CPU, against the
recording backend: which launches take a held block, what block the kernel
finds in its slot, the slot pools shared by caches (one per kernel family
and dtype), and the cases that must launch with kernel arguments instead
(full table or pool, a captured stream, a failed device check or copy,
large grids, compiled specializations, the allocation-free entry point).
Selection records and statistics stay those of the oracle's selection model.
"""
import ctypes as C

import pytest

from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import (add_call, chain_call, elem_offset, emb_call, mf_call,
                                   qkn_call, res_call, rn_call, rope_call, silu_call, sw_call)
from tests.test_host_cache import _chain_struct, c_call, c_layers, call_zoo, run_both
import workloads as wl

BF, F = S.DT_BF16, S.DT_F32
AUTO, JIT, RES = 1, 2, 16
SLOTS, MAX_GRID, ANY_GRID_SLOTS = 40, 512, 10
TAG = 0x52455300
CHAIN_BYTES = 288
INV_FREQ = slice(112, 120)   # RopeArgs.inv_freq inside the chain block: per-version constants
FAM_CHAIN, FAM_NORM, FAM_ROPE, FAM_SW, FAM_ELT, FAM_EMB = range(6)


def family(kv, sub=1):
    """The resident table family of a kernel variant (None: no table; `sub`
    0 with a norm variant: the plain form, whose wide-row kernel has no
    argument-free twin)."""
    if kv == S.RN_WIDE and sub == 0:
        return None
    if kv == S.CH_FUSED:
        return FAM_CHAIN
    if kv in S.NORM_VARIANTS:
        return FAM_NORM
    if S.ROPE_SCALAR <= kv <= S.ROPE_QKN_VEC_I:
        return FAM_ROPE
    if S.SW_SCALAR <= kv <= S.SW_ROWS:
        return FAM_SW
    if S.ELT_SCALAR <= kv <= S.ELT_ROWS:
        return FAM_ELT
    if kv in (S.EMB_SCALAR, S.EMB_VEC):
        return FAM_EMB
    return None


class PoolModel:
    """The slot each launch of one resident cache takes: a held block keeps
    its slot; a new block takes the lowest free slot of its family and dtype
    (below ANY_GRID_SLOTS for launches beyond MAX_GRID workgroups), or none
    (-1: kernel arguments)."""

    def __init__(self):
        self.used, self.held = {}, {}

    def expect(self, kv, dt, grid, raw, sub=1):
        fam = family(kv, sub)
        if fam is None:
            return -1
        key = (fam, dt, raw, grid)
        if key not in self.held:
            used = self.used.setdefault((fam, dt), set())
            limit = SLOTS if grid <= MAX_GRID else ANY_GRID_SLOTS
            free = [k for k in range(limit) if k not in used]
            if not free:
                return -1
            used.add(free[0])
            self.held[key] = free[0]
        return self.held[key]


@pytest.fixture(scope="module")
def lib():
    return load_fake()


@pytest.fixture
def fresh(lib):
    caches = []

    def make(capacity=0, flags=0):
        lib.trifake_reset()
        h = C.c_void_p()
        assert lib.tri_spec_cache_create(C.byref(h), capacity, flags) == 0
        caches.append(h)
        return h
    yield make
    for h in caches:
        lib.tri_spec_cache_destroy(h)


def info(lib, cache):
    from paper_2609_37241_amd._lib import ResidentInfo
    r = ResidentInfo()
    assert lib.tri_spec_resident_info(cache, C.byref(r)) == 0
    return r.enabled, r.held, r.launches


def counts(lib):
    out = (C.c_int64 * 2)()
    lib.trifake_resident_counts(out)
    return out[0], out[1]


def launches(lib, start=0):
    """(slot, kernel variant, dtype, sub, grid, block, argument block) of every
    launch from `start` on (a resident launch's block is the one its slot holds)."""
    out = []
    for i in range(start, lib.trifake_launch_count()):
        kv, dt, sub = C.c_int32(), C.c_int32(), C.c_int32()
        grid, block = C.c_uint32(), C.c_uint32()
        stream = C.c_void_p()
        buf = C.create_string_buffer(CHAIN_BYTES)
        assert lib.trifake_get(i, C.byref(kv), C.byref(dt), C.byref(sub), C.byref(grid),
                               C.byref(block), C.byref(stream), buf, CHAIN_BYTES) >= 0
        out.append((lib.trifake_slot(i), kv.value, dt.value, sub.value, grid.value,
                    block.value, buf.raw))
    return out


def masked(raw):
    return raw[:INV_FREQ.start] + raw[INV_FREQ.stop:]


def llama(i=0, T=1, dtype=BF):
    """The 1-token Llama-7B chain; layer i's activations sit i MiB further on."""
    return chain_call(dtype, T, 4096, 11008, 32, 32, 128, res_off=i << 20, rope_off=i << 20,
                      sw_off=i << 20)


def test_resident_launch_finds_the_ordinary_block(lib, fresh):
    c = llama()
    plain = fresh(flags=AUTO)
    assert c_call(lib, plain, c) == 0
    (slot0, *ordinary, raw0), = launches(lib)
    assert slot0 == -1
    assert info(lib, plain) == (0, 0, 0)
    cache = fresh(flags=AUTO | RES)
    for _ in range(5):
        assert c_call(lib, cache, c) == 0
    got = launches(lib)
    assert len(got) == 5
    slot = got[0][0]
    assert 0 <= slot < SLOTS
    for s, *geom, raw in got:
        # the same kernel variant, geometry and block, from the same slot
        assert s == slot and geom == ordinary
        assert masked(raw) == masked(raw0)
    grid, size = C.c_uint32(), C.c_uint32()
    assert lib.trifake_resident_tag(FAM_CHAIN, BF, slot, C.byref(grid), C.byref(size)) == \
        TAG + slot
    assert (grid.value, size.value) == (ordinary[3], CHAIN_BYTES)
    assert counts(lib)[0] == 1                  # one copy, on the first call
    assert info(lib, cache) == (1, 1, 5)


def test_selection_parity_over_call_zoo_with_resident_blocks(lib, fresh):
    """Records and statistics are the model's; a launch of at most 512
    workgroups takes a held block while its family's table for the dtype has
    room; blocks are held in first-seen order and repeats find their slot
    again."""
    cache = fresh(capacity=4096, flags=RES)
    m = S.SpecCacheModel(capacity=4096)
    for _ in range(2):
        for c in call_zoo():
            run_both(lib, cache, m, c)
    pm = PoolModel()
    got = launches(lib)
    for slot, kv, dt, sub, grid, block, raw in got:
        assert slot == pm.expect(kv, dt, grid, raw, sub), (kv, dt, grid)
    assert {f for f, _ in pm.used} == {FAM_CHAIN, FAM_NORM, FAM_ROPE, FAM_SW, FAM_ELT, FAM_EMB}
    enabled, n_held, _ = info(lib, cache)
    assert (enabled, n_held) == (1, len(pm.held))
    assert counts(lib)[0] == n_held


def test_mixed_stream_with_resident_blocks(lib, fresh):
    cache = fresh(flags=RES)
    m = S.SpecCacheModel()
    for T, dt, layout in wl.mixed_stream()[:3000]:
        d = BF if dt == wl.BF16 else F
        off = elem_offset(d) if layout == wl.LAYOUT_UNALIGNED else 0
        pad = wl.MIXED_PAD if layout == wl.LAYOUT_STRIDED else 0
        c = chain_call(d, T, wl.MIXED_H, wl.MIXED_I, wl.MIXED_NQ, wl.MIXED_NK, wl.MIXED_HD,
                       res_off=off, rope_off=off, sw_off=off, res_pad=pad, rope_pad=pad,
                       sw_pad=pad)
        run_both(lib, cache, m, c)
    got = launches(lib)
    pm = PoolModel()
    for slot, kv, dt, sub, grid, block, raw in got:
        assert slot == pm.expect(kv, dt, grid, raw, sub), (kv, dt, grid)
    res = [g for g in got if g[0] >= 0]
    # few distinct blocks: nearly every launch is resident, three-launch
    # chains and 512-token calls included
    assert len(res) > 0.99 * len(got)
    assert any(g[1] != S.CH_FUSED for g in res) and any(g[4] > MAX_GRID for g in res)
    assert counts(lib)[0] == info(lib, cache)[1]


def test_layers_hold_one_block_per_layer(lib, fresh):
    cache = fresh(flags=AUTO | RES)
    calls = [llama(i) for i in range(32)]
    for step in range(3):
        n0 = lib.trifake_launch_count()
        assert c_layers(lib, cache, calls) == 0
        got = launches(lib, n0)
        assert [g[0] for g in got] == list(range(32))   # layer i holds slot i
    assert counts(lib)[0] == 32
    assert info(lib, cache) == (1, 32, 96)
    # the single entry point finds the same slots, in any order
    for i in (7, 3, 31, 0):
        n0 = lib.trifake_launch_count()
        assert c_call(lib, cache, calls[i]) == 0
        assert launches(lib, n0)[0][0] == i
    assert counts(lib)[0] == 32


def test_blocks_beyond_the_table_launch_with_arguments(lib, fresh):
    cache = fresh(flags=AUTO | RES)
    calls = [llama(i) for i in range(SLOTS + 5)]
    assert c_layers(lib, cache, calls) == 0
    got = launches(lib)
    assert [g[0] for g in got] == list(range(SLOTS)) + [-1] * 5
    plain = {masked(g[-1]) for g in got[SLOTS:]}
    assert len(plain) == 5                                # their own argument blocks
    assert info(lib, cache)[:2] == (1, SLOTS)
    # the dtypes have tables of their own
    n0 = lib.trifake_launch_count()
    assert c_call(lib, cache, llama(0, dtype=F)) == 0
    assert launches(lib, n0)[0][0] == 0
    assert info(lib, cache)[:2] == (1, SLOTS + 1)


def test_slots_return_to_the_pool_when_the_cache_is_destroyed(lib):
    lib.trifake_reset()
    a, b = C.c_void_p(), C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(a), 0, AUTO | RES) == 0
    assert lib.tri_spec_cache_create(C.byref(b), 0, AUTO | RES) == 0
    try:
        assert c_layers(lib, a, [llama(i) for i in range(SLOTS)]) == 0
        n0 = lib.trifake_launch_count()
        assert c_call(lib, b, llama(100)) == 0            # the pool is empty
        assert launches(lib, n0)[0][0] == -1
        assert info(lib, b)[:2] == (1, 0)
        syncs = counts(lib)[1]
        lib.tri_spec_cache_destroy(a)
        a = None
        assert counts(lib)[1] == syncs + 1                # the device went idle first
        n0 = lib.trifake_launch_count()
        assert c_call(lib, b, llama(100)) == 0
        assert launches(lib, n0)[0][0] == 0               # a freed slot, rewritten
        assert lib.trifake_resident_tag(FAM_CHAIN, BF, 0, None, None) == TAG
    finally:
        if a:
            lib.tri_spec_cache_destroy(a)
        lib.tri_spec_cache_destroy(b)
    # a cache that held nothing does not wait for the device
    lib.trifake_reset()
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), 0, RES) == 0
    lib.tri_spec_cache_destroy(h)
    assert counts(lib) == (0, 0)


def test_new_blocks_are_not_written_while_the_stream_is_captured(lib, fresh):
    cache = fresh(flags=AUTO | RES)
    c1, c2, c3 = llama(0), llama(1), llama(2)
    assert c_call(lib, cache, c1) == 0
    lib.trifake_force_capturing(1)
    assert c_call(lib, cache, c2) == 0                  # new: kernel arguments
    assert c_call(lib, cache, c1) == 0                  # held: still resident
    lib.trifake_force_capturing(0)
    assert c_call(lib, cache, c2) == 0
    assert [g[0] for g in launches(lib)] == [0, -1, 0, 1]
    assert counts(lib)[0] == 2
    # a graph build captures on its own stream: held layers resident, new ones not
    from paper_2609_37241_amd._lib import ChainArgs
    keep = []
    arr = (ChainArgs * 3)(*[_chain_struct(c, keep) for c in (c1, c3, c2)])
    g = C.c_void_p()
    n0 = lib.trifake_launch_count()
    assert lib.tri_graph_build_layers(cache, arr, 3, C.byref(g)) == 0
    assert [x[0] for x in launches(lib, n0)] == [0, -1, 1]
    assert counts(lib)[0] == 2
    lib.tri_graph_destroy(g)


def test_failed_check_or_copy_launches_with_arguments(lib, fresh):
    lib.trifake_reset()
    lib.trifake_resident_check_fail(1)
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), 0, AUTO | RES) == 0
    try:
        assert c_call(lib, h, llama()) == 0
        assert c_call(lib, h, llama()) == 0
        assert [g[0] for g in launches(lib)] == [-1, -1]
        assert info(lib, h) == (0, 0, 0)
    finally:
        lib.tri_spec_cache_destroy(h)
        lib.trifake_resident_check_fail(0)
    cache = fresh(flags=AUTO | RES)
    lib.trifake_resident_write_fail(1)
    assert c_call(lib, cache, llama()) == 0
    lib.trifake_resident_write_fail(0)
    assert c_call(lib, cache, llama()) == 0
    # the slot of the failed copy went back to the pool and is taken again
    assert [g[0] for g in launches(lib)] == [-1, 0]
    assert info(lib, cache) == (1, 1, 1)


def test_large_launches_take_only_the_first_slots(lib, fresh):
    cache = fresh(flags=AUTO | RES)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    for T in (1, 8, 64, 512, 4096):
        run_both(lib, cache, m, llama(T=T), install=False)
    # a chain whose norm rows are split runs three launches, each resident
    run_both(lib, cache, m, chain_call(BF, 2, 65536, 11008, 32, 32, 128), install=False)
    got = launches(lib)
    assert sum(g[4] > MAX_GRID for g in got) >= 2
    assert [g[0] for g in got[:5]] == [0, 1, 2, 3, 4]    # every size, slots in order
    assert [family(g[1]) for g in got[-3:]] == [FAM_NORM, FAM_ROPE, FAM_SW]
    assert all(g[0] >= 0 for g in got[-3:])
    assert got[-3][1] == S.RN_SPLIT and len(got[-3][-1]) == CHAIN_BYTES


def test_large_launch_without_a_first_slot_carries_its_arguments(lib, fresh):
    """Slots 0-9 taken by small launches: a large launch carries its
    arguments, a small one still takes slot 10 and on."""
    big = fresh(flags=AUTO | RES)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    for i in range(ANY_GRID_SLOTS):
        run_both(lib, big, m, llama(i), install=False)
    run_both(lib, big, m, llama(0, T=512), install=False)
    run_both(lib, big, m, llama(ANY_GRID_SLOTS), install=False)
    got = launches(lib)
    assert got[-2][4] > MAX_GRID
    assert [g[0] for g in got] == list(range(ANY_GRID_SLOTS)) + [-1, ANY_GRID_SLOTS]


def test_compiled_specializations_carry_their_arguments(lib, fresh):
    jc = fresh(flags=AUTO | RES | JIT)
    assert c_call(lib, jc, llama()) == 0
    assert c_call(lib, jc, llama()) == 0
    assert [g[0] for g in launches(lib)] == [-1, -1]
    assert info(lib, jc) == (1, 0, 0)


def test_resident_info_arguments(lib, fresh):
    from paper_2609_37241_amd._lib import ResidentInfo
    r = ResidentInfo()
    assert lib.tri_spec_resident_info(None, C.byref(r)) == S.E_INVALID
    cache = fresh()
    assert lib.tri_spec_resident_info(cache, None) == S.E_INVALID
    assert info(lib, cache) == (0, 0, 0)


STANDALONE = [
    (FAM_NORM, lambda o: rn_call(BF, 1, 4096, off=o)),
    (FAM_NORM, lambda o: res_call(F, 4, 4096, off=o)),
    (FAM_NORM, lambda o: rn_call(F, 1024, 128, off=o)),        # the paper's rms_norm case
    (FAM_ROPE, lambda o: rope_call(BF, 1, 32, 8, 128, off=o)),
    (FAM_ROPE, lambda o: qkn_call(BF, 1, 32, 8, 128, off=o)),
    (FAM_SW, lambda o: sw_call(BF, 1, 11008, off=o)),
    (FAM_ELT, lambda o: silu_call(BF, 1, 4096, off=o)),
    (FAM_ELT, lambda o: add_call(F, 2, 4096, off=o)),
    (FAM_ELT, lambda o: mf_call(BF, 2, 4096, off=o)),
    (FAM_EMB, lambda o: emb_call(BF, 8, 4096, 32000, off=o)),
]


@pytest.mark.parametrize("fam,make", STANDALONE)
def test_standalone_ops_take_held_blocks_of_their_family(lib, fresh, fam, make):
    """Each op's launch finds its own argument block in its family's table:
    the same kernel variant, geometry and bytes as an ordinary cache's
    launch; a second block of the same op takes the next slot."""
    plain = fresh(flags=AUTO)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    run_both(lib, plain, m, make(0), install=False)
    (slot0, *ordinary, raw0), = launches(lib)
    assert slot0 == -1
    cache = fresh(flags=AUTO | RES)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    for c in (make(0), make(0), make(1 << 20), make(0)):
        run_both(lib, cache, m, c, install=False)
    got = launches(lib)
    assert [g[0] for g in got] == [0, 0, 1, 0]
    for slot, *geom, raw in (got[0], got[1], got[3]):
        assert geom == ordinary
        n = lib.trifake_resident_tag(fam, geom[1], slot, None, None)
        assert n == TAG + slot
        if fam == FAM_ROPE:                   # but the version's own frequency table
            assert raw[:24] + raw[32:] == raw0[:24] + raw0[32:]
        else:
            assert raw == raw0
    assert family(got[0][1]) == fam
    assert info(lib, cache) == (1, 2, 4)


def test_noalloc_entry_always_carries_its_arguments(lib, fresh):
    cache = fresh(flags=AUTO | RES)
    c = res_call(BF, 1, 4096)
    assert c_call(lib, cache, c) == 0                   # installs; resident
    from tests.test_host_noalloc import noalloc
    assert noalloc(lib, cache, c) == 0
    assert [g[0] for g in launches(lib)] == [0, -1]
    assert counts(lib)[0] == 1


# ---- random calls: a resident cache launches exactly what an ordinary one does -------------
from hypothesis import given, strategies as st  # noqa: E402

from tests.test_host_fuzz import (SETTINGS, chain_calls, norm_calls, rope_calls,  # noqa: E402
                                  short_calls)


def _version_fields(kv):
    """Byte ranges of a launch's block that hold the version's own device
    memory (RoPE frequency table, split-row scratch): equal within a cache,
    different between two caches."""
    if kv == S.CH_FUSED:
        return [INV_FREQ]
    if S.ROPE_SCALAR <= kv <= S.ROPE_QKN_VEC_I:
        return [slice(24, 32)]
    if kv == S.RN_SPLIT:
        return [slice(88, 96)]
    return []


def _masked_block(kv, raw):
    b = bytearray(raw)
    for sl in _version_fields(kv):
        b[sl] = bytes(sl.stop - sl.start)
    return bytes(b)


def _run_log(lib, calls, flags):
    lib.trifake_reset()
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), S.MAX_CAPACITY, flags) == 0
    try:
        sts = [c_call(lib, h, c) for c in calls]
        return sts, launches(lib), info(lib, h)
    finally:
        lib.tri_spec_cache_destroy(h)


@SETTINGS
@given(st.lists(st.one_of(norm_calls(), rope_calls(), short_calls(), chain_calls()),
                min_size=1, max_size=8))
def test_random_calls_launch_the_same_from_resident_blocks(lib, calls):
    calls = calls + calls                       # every block seen twice
    st_a, log_a, _ = _run_log(lib, calls, AUTO)
    st_b, log_b, (enabled, n_held, n_res) = _run_log(lib, calls, AUTO | RES)
    assert st_a == st_b
    assert len(log_a) == len(log_b)
    pm = PoolModel()
    for (sa, *ga, ra), (sb, *gb, rb) in zip(log_a, log_b):
        assert sa == -1 and ga == gb
        kv, dt, sub, grid = gb[0], gb[1], gb[2], gb[3]
        assert _masked_block(kv, rb) == _masked_block(kv, ra)
        assert sb == pm.expect(kv, dt, grid, rb, sub)
    assert (enabled, n_held) == (1, len(pm.held))
    assert n_res == sum(1 for g in log_b if g[0] >= 0)
