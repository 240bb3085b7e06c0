"""Pins of the oracle's generic (range-guarded) versions and of Algorithm 1's
ordering once versions overlap (Sec. 3.2: the first version whose guards
hold runs; Fig. 4's guards are a rank check and a shape bound, which hold
across many concrete inputs).

The ranges below are worked out by hand from the install-policy table, not
by calling the code under test with other arguments: which token buckets
keep one plan (decode-sized buckets 0-6 split a token's heads over
workgroups, larger ones do not; SwiGLU and the chain stream nontemporally
once a call at the top of the bucket moves more than 320 MiB) and which
hidden sizes one norm kernel serves (vectors per row 1-64, 65-128, 129-256,
257-512, 513-1024, 1025-2048, 2049-4096).
"""
import pytest

from oracle import selection as S
from tests.selection_calls import chain_call, rn_call, res_call, sw_call

BF, F = S.DT_BF16, S.DT_F32
G = S.FLAG_GENERIC | S.FLAG_AUTO_INSTALL


@pytest.mark.parametrize("call,b_lo,b_hi,h", [
    # bf16 4096 = 512 vectors: the two-vectors-per-work-item workgroup, rows
    # of 257..512 vectors = 2056..4096 elements, any bucket
    (rn_call(BF, 5, 4096), 0, 22, (2056, 4096, S.H_MULTIPLE)),
    # bf16 512 = 64 vectors: one wavefront, rows of 1..64 vectors = 8..512
    (res_call(BF, 1, 512), 0, 22, (8, 512, S.H_MULTIPLE)),
    # f32 20000 = 5000 vectors is past 4096: a split row, exact version
    # (tested below); f32 16384 = 4096 vectors: 16 per work-item, 2049..4096
    (rn_call(F, 3, 16384), 0, 22, (8196, 16384, S.H_MULTIPLE)),
    # unaligned rows take the scalar kernel at every length (bf16 rows of 100
    # elements: a 200-byte stride is not 16-byte aligned; an odd pointer);
    # aligned ragged rows (100 elements padded to a 208-byte stride, 100 % 8
    # != 0) take it at every length that is not a whole number of vectors
    (rn_call(BF, 2, 100), 0, 22, (1, (1 << 24) - 1, S.H_ANY)),
    (rn_call(BF, 2, 4096, off=2), 0, 22, (1, (1 << 24) - 1, S.H_ANY)),
    (rn_call(BF, 2, 100, pad=4), 0, 22, (1, (1 << 24) - 1, S.H_RAGGED)),
    # SwiGLU bf16 I = 11008: 3 * 2^b * 11008 * 2 bytes exceeds 320 MiB from
    # b = 13 (2^13 = 8192 > 5081.8) on
    (sw_call(BF, 8, 11008), 0, 12, None),
    (sw_call(BF, 8192, 11008), 13, 22, None),
    # the Llama-7B chain: one token moves 2 * (4*4096 + 2*64*128 + 3*11008)
    # = 131584 bytes; decode buckets 0..6 share the head-slice geometry,
    # 7..11 one token per RoPE workgroup with cached SwiGLU, and from 12 on
    # (4096 tokens: 539 MB > 335.5 MB) the SwiGLU role streams
    (chain_call(BF, 1, 4096, 11008, 32, 32, 128), 0, 6, None),
    (chain_call(BF, 64, 4096, 11008, 32, 32, 128), 0, 6, None),
    (chain_call(BF, 65, 4096, 11008, 32, 32, 128), 7, 11, None),
    (chain_call(BF, 2048, 4096, 11008, 32, 32, 128), 7, 11, None),
    (chain_call(BF, 2049, 4096, 11008, 32, 32, 128), 12, 22, None),
])
def test_generic_ranges_by_hand(call, b_lo, b_hi, h):
    g = S.generic_guard(S.make_key(call))
    assert (g.b_lo, g.b_hi) == (b_lo, b_hi)
    assert (g.h_lo, g.h_hi, g.h_mod) == (h if h else (0, 0, S.H_ANY))


@pytest.mark.parametrize("call,b_hi", [
    # residual f32 rows of 20000 = 5000 vectors: S = ceil(5000 / 2048) = 3
    # workgroups per row; a call of 2^b rows needs 8 + 2^b * (3 + 1) scratch
    # words, at most 2^22 = 4,194,304: 2^19 -> 2,097,160 fits, 2^20 ->
    # 4,194,312 does not, and from bucket 20 on the row goes to the
    # 1024-lane workgroup (5000 <= 8192 vectors)
    (res_call(F, 3, 20000), 19),
    # bf16 rows of 65536 = 8192 vectors, S = 4: 8 + 5 * 2^19 = 2,621,448
    # fits, 8 + 5 * 2^20 = 5,242,888 does not
    (res_call(BF, 3, 65536), 19),
    # plain bf16 rows of 2^20 = 131072 vectors (beyond the 1024-lane
    # workgroup), S = 64: 8 + 65 * 2^15 = 2,129,928 fits, 8 + 65 * 2^16 =
    # 4,259,848 does not; beyond, the two-pass loop
    (rn_call(BF, 2, 1 << 20), 15),
])
def test_split_rows_get_the_buckets_their_scratch_holds(call, b_hi):
    """A split version covers the run of buckets over which the policy keeps
    the split, which ends where the scratch for the top of the bucket no
    longer fits; the row length stays exact (S depends on it)."""
    key = S.make_key(call)
    g = S.generic_guard(key)
    assert (g.b_lo, g.b_hi, g.h_lo) == (0, b_hi, 0)
    f = S.unpack_key(key)
    assert S.split_fits(f["dtype"], f["H"], b_hi) and not S.split_fits(f["dtype"], f["H"], b_hi + 1)
    assert g.holds(S.make_key(call)) and g.holds(S._with_bucket(key, 0))
    assert not g.holds(S._with_bucket(key, b_hi + 1))
    other = dict(F=res_call(F, 3, 20008), BF=res_call(BF, 3, 65544))
    assert not g.holds(S.make_key(other["F" if call.dtype == F else "BF"]))


@pytest.mark.parametrize("call,h", [
    # plain rows of 4097..7168 vectors take the 1024-lane workgroup at every
    # bucket: f32 4097 * 4 = 16388 .. 7168 * 4 = 28672, bf16 32776 .. 57344
    (rn_call(F, 3, 20000), (16388, 28672)),
    (rn_call(BF, 7, 57344), (32776, 57344)),
    (rn_call(BF, 1, 32776), (32776, 57344)),
])
def test_plain_wide_rows_get_every_bucket_and_their_class(call, h):
    g = S.generic_guard(S.make_key(call))
    assert (g.b_lo, g.b_hi, g.h_lo, g.h_hi, g.h_mod) == (0, 22) + h + (S.H_MULTIPLE,)
    assert S.candidates(S.make_key(call))[0].kernels == (S.RN_WIDE,)


def test_plain_rows_of_7169_to_8192_vectors_split_up_to_256_rows():
    # bf16 65536 = 8192 vectors: split (S = 4) up to bucket 8, where the
    # run ends; from bucket 9 the 1024-lane form to the last bucket; the
    # row length is exact either way
    g = S.generic_guard(S.make_key(rn_call(BF, 3, 65536)))
    assert (g.b_lo, g.b_hi, g.h_lo) == (0, 8, 0)
    assert S.candidates(S.make_key(rn_call(BF, 3, 65536)))[0].kernels == (S.RN_SPLIT,)
    g = S.generic_guard(S.make_key(rn_call(BF, 700, 65536)))
    assert (g.b_lo, g.b_hi, g.h_lo) == (9, 22, 0)
    assert S.candidates(S.make_key(rn_call(BF, 700, 65536)))[0].kernels == (S.RN_WIDE,)


def test_a_tuned_split_choice_clamps_the_run():
    """bf16 rows of 32768 = 4096 vectors: the policy's plan is the 256-lane
    workgroup with 16 vectors per lane at every bucket (0..22, rows of
    2049..4096 vectors); the tuning candidates are [that, the 1024-lane
    workgroup, the split over S = 2, the two-pass loop]. A version running
    the split keeps buckets whose scratch 8 + 3 * 2^b words fits: b <= 20
    (3,145,736), not 21 (6,291,464), and only its own row length."""
    key = S.make_key(rn_call(BF, 3, 32768))
    cands = S.candidates(key)
    assert [c.kernels[0] for c in cands] == [S.RN_BLOCK[16], S.RN_WIDE, S.RN_SPLIT, S.RN_LOOP]
    g = S.generic_guard(key, cands[2])
    assert (g.b_lo, g.b_hi, g.h_lo) == (0, 20, 0)
    for c in (cands[0], cands[1], cands[3]):
        gc = S.generic_guard(key, c)
        assert (gc.b_lo, gc.b_hi, gc.h_lo, gc.h_hi) == (0, 22, 16392, 32768)
    # through the model: a timer that favours the split
    m = S.SpecCacheModel(flags=G | S.FLAG_AUTOTUNE,
                         timer=lambda k, i, c: 0.5 if S.RN_SPLIT in c.kernels else 1.0)
    assert m.call(rn_call(BF, 3, 32768)) == S.OK and m.choice == [2]
    assert (m.guards[0].b_lo, m.guards[0].b_hi) == (0, 20)
    assert m.call(rn_call(BF, 1 << 20, 32768)) == S.OK and m.last.version == 0   # bucket 20
    assert m.call(rn_call(BF, (1 << 20) + 1, 32768)) == S.OK                    # bucket 21
    # the bucket-21 miss made a version of the policy's plan over every bucket
    # and the whole row class: another row length of the class lands there
    assert m.call(rn_call(BF, 3, 16392)) == S.OK and m.last.version == 1
    assert m.stats.misses == 2 and len(m.versions) == 2


def test_generic_guard_holds_exactly_on_its_class():
    g = S.generic_guard(S.make_key(rn_call(BF, 5, 4096)))
    assert g.holds(S.make_key(rn_call(BF, 1, 2056)))          # 257 vectors, bucket 0
    assert g.holds(S.make_key(rn_call(BF, 1 << 22, 4096)))    # bucket 22
    assert not g.holds(S.make_key(rn_call(BF, 5, 2048)))      # 256 vectors: another kernel
    assert not g.holds(S.make_key(rn_call(BF, 5, 4104)))      # 513 vectors
    assert not g.holds(S.make_key(rn_call(BF, 5, 4095)))      # ragged: the scalar kernel
    assert not g.holds(S.make_key(rn_call(F, 5, 4096)))       # another dtype
    assert not g.holds(S.make_key(res_call(BF, 5, 4096)))     # another op
    assert not g.holds(S.make_key(rn_call(BF, 5, 4096, pad=64)))   # other layout flags


def test_exact_version_first_wins_over_a_later_generic_one():
    """Algorithm 1: an exact version created first is selected for its key
    although the generic version created later also matches it."""
    m = S.SpecCacheModel(flags=G)
    c8 = chain_call(BF, 8, 4096, 11008, 32, 32, 128)        # bucket 3
    assert m.install_key(S.make_key(c8)) == S.OK             # exact, version 0
    c4 = chain_call(BF, 4, 4096, 11008, 32, 32, 128)        # bucket 2: a miss
    assert m.call(c4) == S.OK and m.stats.misses == 1 and len(m.versions) == 2
    assert (m.guards[1].b_lo, m.guards[1].b_hi) == (0, 6)
    assert m.guards[1].holds(S.make_key(c8))                 # the two overlap
    assert m.call(c8) == S.OK and m.last.version == 0        # first match: exact
    # T = 5..8 is bucket 3, the exact key; the rest of buckets 0..6 the generic one
    for T, want in ((1, 1), (2, 1), (5, 0), (7, 0), (9, 1), (33, 1), (64, 1)):
        assert m.call(chain_call(BF, T, 4096, 11008, 32, 32, 128)) == S.OK
        assert m.last.version == want, T
    assert m.stats.misses == 1


def test_exact_key_behind_a_generic_version_adds_nothing():
    """Installed after a generic version that matches it, an exact version
    could never be selected: the install adds nothing."""
    m = S.SpecCacheModel(flags=G)
    assert m.call(chain_call(BF, 4, 4096, 11008, 32, 32, 128)) == S.OK
    k8 = S.make_key(chain_call(BF, 8, 4096, 11008, 32, 32, 128))
    assert m.install_key(k8) == S.OK and len(m.versions) == 1
    assert m.call(chain_call(BF, 8, 4096, 11008, 32, 32, 128)) == S.OK
    assert m.last.version == 0 and m.stats.misses == 1


def test_generic_norm_versions_serve_row_lengths_in_their_range():
    m = S.SpecCacheModel(flags=G)
    assert m.install_key(S.make_key(rn_call(BF, 4, 3000))) == S.OK     # 375 vectors: exact
    assert m.call(rn_call(BF, 4, 4000)) == S.OK                        # miss -> generic
    assert len(m.versions) == 2 and m.guards[1].h_lo == 2056
    # the exact key is (3000, bucket 2: T = 3..4); every other bucket and
    # length of 257..512 vectors takes the generic version
    for H, T, want in ((3000, 4, 0), (3000, 3, 0), (3000, 2, 1), (3000, 5, 1), (2056, 1, 1),
                       (4096, 100, 1), (4000, 4, 1)):
        assert m.call(rn_call(BF, T, H)) == S.OK
        assert m.last.version == want, (H, T)
        # the launch: 256 work-items, one workgroup per row, at every length
        assert m.last.launch[0] == (S.RN_BLOCK[2], T, 256)
    assert m.call(rn_call(BF, 4, 2048)) == S.OK and len(m.versions) == 3   # 256 vectors: a miss


def test_generic_records_carry_the_call_key_and_its_tokens():
    m = S.SpecCacheModel(flags=G)
    assert m.call(chain_call(BF, 100, 4096, 11008, 32, 32, 128)) == S.OK
    c = chain_call(BF, 1000, 4096, 11008, 32, 32, 128)
    assert m.call(c) == S.OK and m.last.version == 0 and m.stats.misses == 1
    assert m.last.key == S.make_key(c)
    # fused: 1000 norm rows + 1000 RoPE tokens + ceil(1000 * 11008 / 8 / 256) SwiGLU
    assert m.last.launch[0] == (S.CH_FUSED, 1000 + 1000 + 5375, 256)


def test_plain_cache_keeps_exact_versions():
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    for T in (1, 2, 4, 8):
        assert m.call(chain_call(BF, T, 4096, 11008, 32, 32, 128)) == S.OK
    assert len(m.versions) == 4 and all(g.b_lo < 0 for g in m.guards)


@pytest.mark.parametrize("call", [
    chain_call(BF, 8, 4096, 11008, 32, 8, 128), chain_call(F, 300, 4096, 14336, 32, 8, 128),
    sw_call(F, 77, 28672), rn_call(BF, 9, 1024), res_call(F, 3, 8000)])
def test_generic_ranges_keep_one_plan_and_are_maximal(call):
    """Invariant: every bucket of the range gives the key's plan; the buckets
    just outside do not (or are out of [0, 22])."""
    key = S.make_key(call)
    g = S.generic_guard(key)
    P = S.candidates(key)[0]
    for b in range(g.b_lo, g.b_hi + 1):
        assert S.candidates(S._with_bucket(key, b))[0] == P
    for b in (g.b_lo - 1, g.b_hi + 1):
        if 0 <= b <= 22:
            assert S.candidates(S._with_bucket(key, b))[0] != P
