"""Install-time tuning of the native cache on the CPU, against the recording
backend (whose timer charges scripted costs per launch).

Checks that the library's candidate plans are the oracle's, that a pinned
candidate makes the selections the model makes, that a tuning cache times
every candidate on a call of the key's own shapes, keeps what the choice rule
keeps and stores it in the code directory (the Triton autotuner scheme the
paper describes in Sec. 2).
"""
import ctypes as C

import pytest

from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import (add_call, chain_call, elem_offset, emb_call, mf_call,
                                   qkn_call, res_call, rn_call, rope_call, silu_call, sw_call)
from tests.test_host_cache import (LLAMA3, ROPE_EXTS, _launch_at, c_call, c_record, c_stats,
                                   jit_sources, m_stats)

BF, F = S.DT_BF16, S.DT_F32
TUNE_STREAM = 0x72000000
SCRATCH = 0x5C0000000000


@pytest.fixture(scope="module")
def lib():
    return load_fake()


@pytest.fixture
def fresh(lib):
    caches = []

    def make(capacity=0, flags=0, code_dir=None):
        lib.trifake_reset()
        h = C.c_void_p()
        assert lib.tri_spec_cache_create(C.byref(h), capacity, flags) == 0
        if code_dir is not None:
            assert lib.tri_spec_set_code_dir(h, str(code_dir).encode()) == 0
        caches.append(h)
        return h
    yield make
    for h in caches:
        lib.tri_spec_cache_destroy(h)


def info(lib, cache, i=0):
    from paper_2609_37241_amd._lib import VersionInfo
    v = VersionInfo()
    assert lib.tri_spec_version_info(cache, i, C.byref(v)) == 0
    return v


def install(lib, cache, key, cand=-1):
    return lib.tri_spec_install_key(cache, (C.c_uint64 * 6)(*key), cand)


def counts(lib):
    out = (C.c_int64 * 5)()
    lib.trifake_tune_counts(out)
    return dict(zip(("timers", "destroyed", "allocs", "frees", "bytes"), out))


def tuning_zoo():
    """Valid calls over every op, dtype, layout class and RoPE variant."""
    calls = []
    for d in (F, BF):
        off = elem_offset(d)
        for T in (1, 3, 8, 64, 512, 8192, 8193):
            calls += [rn_call(d, T, 512), rn_call(d, T, 4096), res_call(d, T, 1024),
                      res_call(d, T, 40000), rn_call(d, T, 4096, off=off),
                      res_call(d, T, 4096, pad=64), rn_call(d, T, 100),
                      rope_call(d, T, 32, 8, 128), rope_call(d, T, 4, 0, 64),
                      rope_call(d, T, 64, 64, 128), rope_call(d, T, 2, 2, 96),
                      rope_call(d, T, 32, 8, 128, off=off), rope_call(d, T, 32, 8, 128, pad=64),
                      qkn_call(d, T, 32, 8, 128), qkn_call(d, T, 4, 0, 64),
                      qkn_call(d, T, 32, 8, 128, w_off=off),
                      sw_call(d, T, 11008), sw_call(d, T, 688), sw_call(d, T, 11003),
                      sw_call(d, T, 11008, pad=64), sw_call(d, T, 11008, off=off),
                      silu_call(d, T, 4096), add_call(d, T, 1001), mf_call(d, T, 4096),
                      add_call(d, T, 4096, pad=64), mf_call(d, T, 4096, m_off=4),
                      emb_call(d, T, 4096, 100),
                      chain_call(d, T, 4096, 11008, 32, 32, 128),
                      chain_call(d, T, 256, 688, 4, 4, 64),
                      chain_call(d, T, 8192, 28672, 64, 8, 128, base=5e5),
                      chain_call(d, T, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True),
                      chain_call(d, T, 4096, 14336, 32, 8, 128, sw_pad=64),
                      chain_call(d, T, 4096, 14336, 32, 8, 128, rope_off=off)]
            for ext in ROPE_EXTS:
                calls.append(rope_call(d, T, 32, 8, 128, base=5e5, ext=ext))
                calls.append(qkn_call(d, T, 8, 2, 128, base=5e5, ext=ext))
                calls.append(chain_call(d, T, 4096, 14336, 32, 8, 128, base=5e5, ext=ext))
    return calls


def distinct_keys(calls):
    seen, out = set(), []
    for c in calls:
        assert S.validate(c) is None, c
        k = S.make_key(c)
        if k not in seen:
            seen.add(k)
            out.append((k, c))
    return out


# ---- candidate lists and pinned candidates ------------------------------------------------
def test_candidates_and_pinned_selections_match_the_model(lib, fresh):
    """Every candidate of every key, pinned with tri_spec_install_key: the
    version's plan and the call's selection record are the model's."""
    keys = distinct_keys(tuning_zoo())
    n_max = max(len(S.candidates(k)) for k, _ in keys)
    assert n_max >= 13
    checked = 0
    for i in range(n_max):
        cache = fresh(capacity=S.MAX_CAPACITY)
        m = S.SpecCacheModel(capacity=S.MAX_CAPACITY)
        for k, c in keys:
            cands = S.candidates(k)
            if i >= len(cands):
                assert install(lib, cache, k, i) == S.E_INVALID
                continue
            assert install(lib, cache, k, i) == S.OK and m.install_key(k, i) == S.OK
            v = info(lib, cache, len(m.versions) - 1)
            want = cands[i]
            assert (v.variant, tuple(v.roles), v.n_launches) == \
                (want.variant, want.roles, len(want.kernels)), (k, i)
            assert tuple(v.kernels)[:v.n_launches] == want.kernels
            assert (v.rope_slices, v.rope_tokens) == (want.slices, want.tokens)
            assert (v.candidate, v.n_candidates, v.tuned) == (i, len(cands), S.TUNE_NONE)
            assert c_call(lib, cache, c) == S.OK and m.call(c) == S.OK
            assert c_record(lib, cache) == m.last.as_tuple(), (k, i)
            checked += 1
        assert c_stats(lib, cache) == m_stats(m)
    assert checked > 1000


def test_install_key_errors_and_idempotence(lib, fresh):
    cache = fresh()
    k = S.make_key(rope_call(BF, 8, 32, 8, 128, base=5e5))
    assert install(lib, cache, k, 4) == S.E_INVALID          # four candidates
    assert install(lib, cache, k, -2) == S.E_INVALID
    assert lib.tri_spec_install_key(cache, None, 0) == S.E_INVALID
    assert lib.tri_spec_install_key(None, (C.c_uint64 * 6)(*k), 0) == S.E_INVALID
    bad = list(k)
    bad[0] = (bad[0] & ~0xFF) | 0x3F
    assert install(lib, cache, bad, 0) == S.E_INVALID
    assert c_stats(lib, cache)[5:] == (0, 0)
    assert install(lib, cache, k, 3) == S.OK
    assert install(lib, cache, k, 1) == S.OK                 # already there: kept
    v = info(lib, cache)
    assert (v.variant, v.candidate, v.n_candidates) == (S.ROPE_SCALAR, 3, 4)
    full = fresh(capacity=1)
    assert install(lib, full, k, 0) == S.OK
    assert install(lib, full, S.make_key(rn_call(BF, 1, 4096)), 0) == S.E_FULL


# ---- tuning against scripted costs ---------------------------------------------------------
def ksub_of(key, cand, i):
    """The kernel sub-selector of launch i of a candidate: the residual flag
    of norm kernels, the op of element-wise kernels, the id width of the
    embedding kernel, and for the fused chain (norm role - 11) * 8 + GPT-J
    pairs * 4 + QK norm * 2 + nontemporal SwiGLU."""
    f = S.unpack_key(key)
    kv = cand.kernels[i]
    if kv == S.CH_FUSED:
        rn, ro, sw = cand.roles
        return ((rn - 11) * 8 + 4 * (ro in (S.ROPE_VEC_I, S.ROPE_QKN_VEC_I))
                + 2 * (ro in (S.ROPE_QKN_VEC, S.ROPE_QKN_VEC_I)) + (sw == S.SW_FLAT_NT))
    if 10 <= kv <= 18:
        return int(f["op"] in (S.OP_RES_RMSNORM, S.OP_CHAIN))
    if 60 <= kv <= 63:
        return f["op"]
    if kv in (S.EMB_SCALAR, S.EMB_VEC):
        return f["rope_bits"] & 1
    return 0


def launch_cost(costs, kv, sub, grid):
    c = 1.0
    for (k, s, g, ms) in costs:
        if k == kv and (s < 0 or s == sub) and (g == 0 or g == grid):
            c = ms
    return c


def scripted_timer(costs):
    """The model's timer for the recording backend's scripted costs."""
    def timer(key, i, cand):
        _, _, launches = S.cand_plan(key, cand, S.tune_tokens(key))
        return sum(launch_cost(costs, kv, ksub_of(key, cand, j), g)
                   for j, (kv, g, _) in enumerate(launches))
    return timer


def set_costs(lib, costs):
    for (k, s, g, ms) in costs:
        lib.trifake_set_cost(k, s, g, ms)


LLAMA_CHAIN = chain_call(BF, 1, 4096, 11008, 32, 32, 128)
# fused Llama-7B decode chain: ksub 3 * 8 + 1 = 25 is the nontemporal form;
# grid 1 + 1 + 6 = 8 is one slice: candidate 3 (one slice, nontemporal)
FAST3 = [(S.CH_FUSED, 25, 8, 0.5)]


def test_tuning_keeps_the_scripted_fastest(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE)
    set_costs(lib, FAST3)
    assert c_call(lib, cache, LLAMA_CHAIN) == S.OK
    v = info(lib, cache)
    assert (v.candidate, v.n_candidates, v.tuned) == (3, 7, S.TUNE_MEASURED)
    assert (tuple(v.roles), v.rope_slices) == ((14, 31, 42), 1)
    assert v.tune_ms >= 0.0
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE,
                         timer=scripted_timer(FAST3))
    assert m.call(LLAMA_CHAIN) == S.OK
    assert m.choice == [3] and c_record(lib, cache) == m.last.as_tuple()
    cnt = counts(lib)
    assert (cnt["timers"], cnt["destroyed"], cnt["allocs"], cnt["frees"]) == (1, 1, 1, 1)
    assert cnt["bytes"] >= S.tune_operand_bytes(S.make_key(LLAMA_CHAIN))


def test_tuning_launch_sequence(lib, fresh):
    """Two warm-up and five timed rounds over the candidates in order, each
    call the candidate's launches for the top of the bucket, on the tuning
    stream, with argument blocks in the tuning memory."""
    c = chain_call(BF, 3, 4096, 11008, 32, 32, 128)     # bucket 2: 4 tokens
    key = S.make_key(c)
    cands = S.candidates(key)
    cache = fresh(flags=S.FLAG_AUTOTUNE)
    assert install(lib, cache, key) == S.OK
    want = []
    for _ in range(2 + 5):
        for cand in cands:
            for j, (kv, g, b) in enumerate(S.cand_plan(key, cand, 4)[2]):
                want.append((kv, ksub_of(key, cand, j), g, b))
    assert lib.trifake_launch_count() == len(want)
    got = []
    for i in range(len(want)):
        kv, dt, sub, grid, block, stream = _launch_at(lib, i)
        assert dt == BF and stream == TUNE_STREAM + 1
        got.append((kv, sub, grid, block))
    assert got == want
    # the fused launch's argument block: x pointer in the tuning memory, T = 4
    import struct
    raw = C.create_string_buffer(288)
    kv, dt, sub, grid, block, stream = C.c_int32(), C.c_int32(), C.c_int32(), C.c_uint32(), \
        C.c_uint32(), C.c_void_p()
    lib.trifake_get(0, C.byref(kv), C.byref(dt), C.byref(sub), C.byref(grid), C.byref(block),
                    C.byref(stream), raw, 288)
    x, res = struct.unpack_from("<2Q", raw.raw, 0)
    T = struct.unpack_from("<q", raw.raw, 72)[0]
    assert SCRATCH <= x < SCRATCH + counts(lib)["bytes"] and x % 256 == 0
    assert T == 4


@pytest.mark.parametrize("scale,want", [(0.98, 0), (0.96, 3), (1.0, 0)])
def test_tuning_margin(lib, fresh, scale, want):
    costs = [(S.CH_FUSED, 25, 8, scale)]
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE)
    set_costs(lib, costs)
    assert c_call(lib, cache, LLAMA_CHAIN) == S.OK
    assert info(lib, cache).candidate == want
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE, timer=scripted_timer(costs))
    m.call(LLAMA_CHAIN)
    assert m.choice == [want]


def test_every_zoo_key_is_tuned_on_a_call_of_its_own_shape(lib, fresh):
    """The tuning call rebuilt from each key hits that key (else tuning is
    skipped): every key with several candidates is measured."""
    cache = fresh(capacity=S.MAX_CAPACITY, flags=S.FLAG_AUTOTUNE)
    n_tuned = 0
    for i, (k, c) in enumerate(distinct_keys(tuning_zoo())):
        lib.trifake_reset()
        assert install(lib, cache, k) == S.OK
        v = info(lib, cache, i)
        n = len(S.candidates(k))
        assert v.n_candidates == n
        if n == 1:
            assert v.tuned == S.TUNE_NONE and counts(lib)["timers"] == 0
            continue
        if S.tune_operand_bytes(k) > S.TUNE_SCRATCH_MAX:
            assert v.tuned == S.TUNE_SKIPPED and counts(lib)["allocs"] == 0
            continue
        assert v.tuned == S.TUNE_MEASURED, (hex(k[0]), c.op, c.T)
        assert v.candidate == 0                  # equal default costs: the policy's plan
        assert counts(lib)["bytes"] >= S.tune_operand_bytes(k)
        n_tuned += 1
    assert n_tuned > 300


def test_tuning_model_parity_over_calls(lib, fresh):
    """Auto-install with tuning against the model over a call stream, with
    costs that favour non-default plans of several kernel families."""
    costs = [(S.SW_FLAT_NT, -1, 0, 0.5), (S.ELT_ROWS, -1, 0, 0.25), (S.RN_LOOP, -1, 0, 0.7),
             (S.ROPE_SCALAR, -1, 0, 0.9), (S.CH_FUSED, 25, 0, 0.8), (S.CH_FUSED, 24, 10, 0.6)]
    cache = fresh(capacity=S.MAX_CAPACITY, flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE)
    set_costs(lib, costs)
    m = S.SpecCacheModel(capacity=S.MAX_CAPACITY, flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE,
                         timer=scripted_timer(costs))
    for c in tuning_zoo():
        assert c_call(lib, cache, c) == m.call(c) == S.OK
        assert c_record(lib, cache) == m.last.as_tuple(), c
    assert c_stats(lib, cache) == m_stats(m)
    for i in range(len(m.versions)):
        v = info(lib, cache, i)
        assert (v.candidate, v.tuned) == (m.choice[i], m.tuned[i])
    assert sum(ch != 0 for ch in m.choice) > 50


def test_tuning_skips_oversized_and_failed_workloads(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTOTUNE)
    big = S.make_key(sw_call(BF, 1 << 22, 4096))
    assert S.tune_operand_bytes(big) > S.TUNE_SCRATCH_MAX
    assert install(lib, cache, big) == S.OK
    v = info(lib, cache)
    assert (v.candidate, v.tuned) == (0, S.TUNE_SKIPPED)
    assert counts(lib)["timers"] == 0 and counts(lib)["allocs"] == 0
    lib.trifake_scratch_fail(1)
    k = S.make_key(sw_call(BF, 4, 4096))
    assert install(lib, cache, k) == S.OK
    v = info(lib, cache, 1)
    assert (v.candidate, v.tuned) == (0, S.TUNE_SKIPPED)
    cnt = counts(lib)
    assert cnt["timers"] == cnt["destroyed"] == 1 and cnt["frees"] == 0
    # one candidate: nothing timed
    e = S.make_key(emb_call(BF, 4, 4096, 100))
    assert install(lib, cache, e) == S.OK and info(lib, cache, 2).tuned == S.TUNE_NONE


def test_pinned_candidate_is_not_tuned(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTOTUNE)
    set_costs(lib, FAST3)
    assert install(lib, cache, S.make_key(LLAMA_CHAIN), 5) == S.OK
    v = info(lib, cache)
    assert (v.candidate, v.tuned) == (5, S.TUNE_NONE) and counts(lib)["timers"] == 0


def test_import_with_tuning_tunes_each_key(lib, fresh):
    keys = [S.make_key(c) for c in (LLAMA_CHAIN, sw_call(BF, 64, 11008), rn_call(BF, 1, 512),
                                    emb_call(BF, 1, 64, 10))]
    cache = fresh(flags=S.FLAG_AUTOTUNE)
    set_costs(lib, FAST3 + [(S.SW_ROWS, -1, 0, 0.1)])
    buf = (C.c_uint64 * 24)(*[w for k in keys for w in k])
    done = C.c_uint32()
    assert lib.tri_spec_import_keys(cache, buf, 4, C.byref(done)) == 0 and done.value == 4
    got = [(info(lib, cache, i).candidate, info(lib, cache, i).tuned) for i in range(4)]
    assert got == [(3, S.TUNE_MEASURED), (2, S.TUNE_MEASURED), (0, S.TUNE_MEASURED),
                   (0, S.TUNE_NONE)]


# ---- stored choices ---------------------------------------------------------------------------
def test_code_directory_stores_tuning_results(lib, fresh, tmp_path):
    key = S.make_key(LLAMA_CHAIN)
    a = fresh(flags=S.FLAG_AUTOTUNE, code_dir=tmp_path)
    set_costs(lib, FAST3)
    assert install(lib, a, key) == S.OK and info(lib, a).tuned == S.TUNE_MEASURED
    (f,) = [p for p in tmp_path.iterdir()]
    assert f.name.startswith("tri-tune-") and f.name.endswith(".txt")
    assert f.read_text() == "3\n"
    # another cache (other costs) reads the stored choice and times nothing
    b = fresh(flags=S.FLAG_AUTOTUNE, code_dir=tmp_path)
    lib.trifake_set_cost(S.CH_FUSED, -1, 0, 0.1)
    assert install(lib, b, key) == S.OK
    v = info(lib, b)
    assert (v.candidate, v.tuned) == (3, S.TUNE_STORED) and counts(lib)["timers"] == 0
    # unusable contents are timed again and replaced
    for junk in ("99\n", "-1\n", "x\n", "", "3x\n"):
        f.write_text(junk)
        c = fresh(flags=S.FLAG_AUTOTUNE, code_dir=tmp_path)
        set_costs(lib, FAST3)
        assert install(lib, c, key) == S.OK
        assert (info(lib, c).candidate, info(lib, c).tuned) == (3, S.TUNE_MEASURED), junk
        assert f.read_text() == "3\n"
    # another architecture names another file
    d = fresh(flags=S.FLAG_AUTOTUNE, code_dir=tmp_path)
    lib.trifake_set_arch(b"gfx942")
    assert install(lib, d, key) == S.OK and info(lib, d).tuned == S.TUNE_MEASURED
    assert len(list(tmp_path.iterdir())) == 2
    # skipped tunings store nothing
    e = fresh(flags=S.FLAG_AUTOTUNE, code_dir=tmp_path)
    assert install(lib, e, S.make_key(sw_call(BF, 1 << 22, 4096))) == S.OK
    assert len(list(tmp_path.iterdir())) == 2


def test_jit_compiles_only_the_kept_plan(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE | S.FLAG_JIT)
    set_costs(lib, FAST3)
    assert c_call(lib, cache, LLAMA_CHAIN) == S.OK
    (src,) = jit_sources(lib)
    # fused template: RN_BLOCK_2 norm, plain RoPE, nontemporal SwiGLU; one slice
    assert "body_chain<1, false, 2, true, false, false>(a, gridDim.x)" in src
    assert "a.rope.mode = 0u;" in src
    v = info(lib, cache)
    assert (v.candidate, v.tuned, v.jit) == (3, S.TUNE_MEASURED, 1)


def test_create_accepts_the_tuning_flag(lib):
    # 8 is the generic-version flag, 16 resident argument blocks; 32 and above
    # are not flags
    for flags, ok in ((4, True), (7, True), (15, True), (16, True), (31, True), (32, False),
                      (36, False)):
        h = C.c_void_p()
        st = lib.tri_spec_cache_create(C.byref(h), 0, flags)
        assert (st == 0) == ok, flags
        if st == 0:
            lib.tri_spec_cache_destroy(h)
