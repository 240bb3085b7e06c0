"""CPU tests of generic (range-guarded) versions in the library against the
oracle's selection model (recording backend): selection records, statistics
and launches call by call, and the guard of every version, over the call
zoo and over the whole mixed-shape stream with exact versions installed
before and during it, so that overlapping versions make Algorithm 1's
first match in creation order decide."""
import ctypes as C

import pytest

from oracle import selection as S
from tests.selection_calls import chain_call, elem_offset, res_call, rn_call
from tests.test_host_cache import (c_call, c_install, c_record, c_stats, call_zoo, lib,  # noqa
                                   m_stats, run_both)
import workloads as wl

BF, F = S.DT_BF16, S.DT_F32
G = S.FLAG_GENERIC


@pytest.fixture
def fresh(lib):   # noqa: F811
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


def c_guards(lib, cache):
    """(b_lo, b_hi, h_lo, h_hi, h_mod) of every version, creation order."""
    from paper_2609_37241_amd._lib import Stats, VersionInfo
    st = Stats()
    lib.tri_spec_stats(cache, C.byref(st))
    out = []
    for i in range(st.n_versions):
        v = VersionInfo()
        assert lib.tri_spec_version_info(cache, i, C.byref(v)) == 0
        out.append((v.b_lo, v.b_hi, v.h_lo, v.h_hi, v.h_mod))
    return out


def m_guards(m):
    return [(g.b_lo, g.b_hi, g.h_lo, g.h_hi, g.h_mod) for g in m.guards]


def c_install_key(lib, cache, key, candidate=-1):
    buf = (C.c_uint64 * 6)(*key)
    return lib.tri_spec_install_key(cache, buf, candidate)


def mixed_call(T, dt, layout):
    d = BF if dt == wl.BF16 else F
    off = elem_offset(d) if layout == wl.LAYOUT_UNALIGNED else 0
    pad = wl.MIXED_PAD if layout == wl.LAYOUT_STRIDED else 0
    return chain_call(d, T, wl.MIXED_H, wl.MIXED_I, wl.MIXED_NQ, wl.MIXED_NK, wl.MIXED_HD,
                      res_off=off, rope_off=off, sw_off=off, res_pad=pad, rope_pad=pad,
                      sw_pad=pad)


@pytest.mark.parametrize("auto", [False, True], ids=["miss-install", "auto-install"])
def test_generic_parity_over_call_zoo(lib, fresh, auto):
    flags = G | (S.FLAG_AUTO_INSTALL if auto else 0)
    cache = fresh(capacity=4096, flags=flags)
    m = S.SpecCacheModel(capacity=4096, flags=flags)
    for c in call_zoo():
        run_both(lib, cache, m, c, install=not auto)
    assert c_guards(lib, cache) == m_guards(m)
    assert any(g[0] >= 0 for g in m_guards(m)) and any(g[2] for g in m_guards(m))
    for c in call_zoo():
        assert run_both(lib, cache, m, c, install=not auto) != S.MISS


def test_mixed_stream_with_overlapping_versions(lib, fresh):
    """All 10,000 calls of the mixed stream on a generic auto-installing
    cache. Before the stream, exact keys for every third distinct key of the
    stream's first 200 calls are installed; after 5,000 calls, every other
    distinct key of the stream is installed exactly (most are already
    matched by a generic version and add nothing). Records, statistics and
    launches agree with the model on every call; some calls hit exact
    versions that a later generic version overlaps."""
    flags = G | S.FLAG_AUTO_INSTALL
    cache = fresh(flags=flags)
    m = S.SpecCacheModel(flags=flags)
    stream = wl.mixed_stream()
    keys = []
    for T, dt, layout in stream[:200]:
        k = S.make_key(mixed_call(T, dt, layout))
        if k not in keys:
            keys.append(k)
    for k in keys[::3]:
        assert c_install_key(lib, cache, k) == m.install_key(k) == S.OK
    n_pre = len(m.versions)
    hit_exact_overlapped = 0
    for n, (T, dt, layout) in enumerate(stream):
        if n == 5000:
            later = []
            for T2, dt2, l2 in stream:
                k = S.make_key(mixed_call(T2, dt2, l2))
                if k not in later:
                    later.append(k)
            for k in later[::2]:
                assert c_install_key(lib, cache, k) == m.install_key(k) == S.OK
        c = mixed_call(T, dt, layout)
        run_both(lib, cache, m, c, install=False)
        v = m.last.version
        if v < n_pre and any(m.guards[j].holds(S.make_key(c))
                             for j in range(v + 1, len(m.guards))):
            hit_exact_overlapped += 1
    assert c_guards(lib, cache) == m_guards(m)
    assert c_stats(lib, cache) == m_stats(m)
    assert m.stats.hits + m.stats.misses == wl.MIXED_CALLS
    assert hit_exact_overlapped > 0                      # overlap actually decided calls
    assert sum(g.b_lo >= 0 for g in m.guards) >= 2       # generic versions were made
    # far fewer versions than one per key: 9 token buckets x 2 dtypes x 3 layouts
    assert len(m.versions) < 54


def test_overlap_order_through_the_library(lib, fresh):
    """The hand-worked overlap cases: an exact version created first wins for
    its key; an exact key behind a generic version installs nothing; a
    generic norm version serves every row length of its range."""
    cache = fresh(flags=G | S.FLAG_AUTO_INSTALL)
    c8 = chain_call(BF, 8, 4096, 11008, 32, 32, 128)
    assert c_install_key(lib, cache, S.make_key(c8)) == S.OK
    assert c_call(lib, cache, chain_call(BF, 4, 4096, 11008, 32, 32, 128)) == S.OK
    assert c_guards(lib, cache) == [(-1, -1, 0, 0, 0), (0, 6, 0, 0, 0)]
    for T, want in ((8, 0), (5, 0), (7, 0), (1, 1), (2, 1), (9, 1), (64, 1)):
        assert c_call(lib, cache, chain_call(BF, T, 4096, 11008, 32, 32, 128)) == S.OK
        assert c_record(lib, cache)[2] == want, T
    # behind the generic version: nothing is added
    k16 = S.make_key(chain_call(BF, 16, 4096, 11008, 32, 32, 128))
    assert c_install_key(lib, cache, k16) == S.OK and len(c_guards(lib, cache)) == 2
    # norm rows
    assert c_call(lib, cache, rn_call(BF, 4, 4000)) == S.OK
    assert c_guards(lib, cache)[2] == (0, 22, 2056, 4096, S.H_MULTIPLE)
    for H, T in ((2056, 1), (3000, 9), (4096, 1000)):
        assert c_call(lib, cache, rn_call(BF, T, H)) == S.OK
        rec = c_record(lib, cache)
        assert rec[2] == 2 and rec[6][0] == (S.RN_BLOCK[2], T, 256)
    assert c_stats(lib, cache)[2] == 2                   # misses: the chain and the norm


def test_memo_returns_the_first_match_after_later_installs(lib, fresh):
    """A key's first match is remembered; a later install never changes it
    (versions are only appended), and a key never seen is scanned."""
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    calls = [rn_call(BF, T, H) for H in (4096, 8192, 1024) for T in (1, 3, 9, 100)]
    for _ in range(3):
        for c in calls + calls[::-1]:
            run_both(lib, cache, m, c, install=False)


def _zero_allocs(lib):
    lib.trifake_zero_allocs.argtypes = [C.POINTER(C.c_int64)]
    counts = (C.c_int64 * 2)()
    lib.trifake_zero_allocs(counts)
    return counts[0], counts[1]


def test_generic_split_version_serves_its_run_with_a_scratch_for_the_top(lib, fresh):
    """Residual bf16 rows of 65536 (S = 4): one generic version serves
    buckets 0..19, with a zeroed scratch of 8 + 5 * 2^19 words allocated at
    install; a call in bucket 20 is a miss on both sides (the policy then
    takes the 1024-lane workgroup, whose version needs no scratch)."""
    flags = G | S.FLAG_AUTO_INSTALL
    cache = fresh(flags=flags)
    m = S.SpecCacheModel(flags=flags)
    n0, b0 = _zero_allocs(lib)
    for T in (3, 1, 64, 5000):
        run_both(lib, cache, m, res_call(BF, T, 65536), install=False)
    assert c_guards(lib, cache) == m_guards(m) == [(0, 19, 0, 0, 0)]
    n1, b1 = _zero_allocs(lib)
    assert (n1 - n0, b1 - b0) == (1, 8 * (8 + 5 * (1 << 19)))
    assert c_stats(lib, cache) == m_stats(m) and m.stats.misses == 1
    # a bucket-20 key: a miss that installs the next version
    key20 = S._with_bucket(S.make_key(res_call(BF, 3, 65536)), 20)
    assert c_install_key(lib, cache, key20) == m.install_key(key20) == S.OK
    assert len(c_guards(lib, cache)) == len(m.versions) == 2
    assert _zero_allocs(lib)[0] == n1                        # RN_WIDE: no scratch


def test_tuned_split_choice_is_clamped_to_the_buckets_its_scratch_holds(lib, fresh):
    """bf16 rows of 32768: the policy's 256-lane workgroup holds at every
    bucket, but a tuned split (S = 2) only where 8 + 3 * 2^b words fit, so
    the generic version's run is 0..20 (scratch sized for 2^20 rows), not
    0..22, and only its own row length; the same guard comes out of the
    model. A bucket-21 miss then makes a version of the policy's plan over
    every bucket and the row class, where another length lands."""
    from tests.test_host_tuning import scripted_timer, set_costs
    costs = [(S.RN_SPLIT, -1, 0, 0.5)]
    flags = G | S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE
    cache = fresh(flags=flags)
    set_costs(lib, costs)
    m = S.SpecCacheModel(flags=flags, timer=scripted_timer(costs))
    n0, b0 = _zero_allocs(lib)
    c = rn_call(BF, 3, 32768)
    assert c_call(lib, cache, c) == m.call(c) == S.OK
    assert m.choice == [2] and c_record(lib, cache) == m.last.as_tuple()
    assert c_guards(lib, cache) == m_guards(m) == [(0, 20, 0, 0, 0)]
    n1, b1 = _zero_allocs(lib)
    assert (n1 - n0, b1 - b0) == (1, 8 * (8 + 3 * (1 << 20)))
    for T in (1, 700, 1 << 20):
        cc = rn_call(BF, T, 32768)
        assert c_call(lib, cache, cc) == m.call(cc) == S.OK
        assert c_record(lib, cache) == m.last.as_tuple() and m.last.version == 0
    for T, H, v in (((1 << 20) + 1, 32768, 1), (700, 24576, 1)):
        cc = rn_call(BF, T, H)
        assert c_call(lib, cache, cc) == m.call(cc) == S.OK
        assert c_record(lib, cache) == m.last.as_tuple() and m.last.version == v
    assert c_guards(lib, cache) == m_guards(m)
    assert c_stats(lib, cache) == m_stats(m) and m.stats.misses == 2
