"""Pins for the selection model: ordered dispatch (Algorithm 1, Sec. 3.2),
the miss / install / error paths (Sec. 3.5) and the install policy table,
worked by hand for the decode shapes (CPU only)."""
import pytest

from oracle import selection as S
from tests.selection_calls import (chain_call, elem_offset, qkn_call, res_call, rn_call,
                                   rope_call, sw_call)

BF, F = S.DT_BF16, S.DT_F32


def test_bucket_closed_form():
    # ceil(log2 T) for T >= 1, via the bit length of T - 1.
    for T in range(1, 1 << 16):
        assert S.bucket(T) == (T - 1).bit_length()
    for T in (1 << 20, (1 << 20) + 1, S.T_MAX):
        assert S.bucket(T) == (T - 1).bit_length()


def test_key_round_trip():
    c = chain_call(BF, 8, 4096, 14336, 32, 8, 128, base=500000.0)
    f = S.unpack_key(S.make_key(c))
    assert (f["op"], f["dtype"], f["bucket"], f["flags"]) == (S.OP_CHAIN, BF, 3, 0x3F)
    assert (f["H"], f["I"], f["hd"], f["nq"], f["nk"]) == (4096, 14336, 128, 32, 8)
    assert f["base_bits"] == 0x48F42400          # 500000.0f


def test_unused_key_fields_are_zero():
    f = S.unpack_key(S.make_key(rn_call(F, 3, 256)))
    assert (f["I"], f["hd"], f["nq"], f["nk"], f["base_bits"]) == (0, 0, 0, 0, 0)
    f = S.unpack_key(S.make_key(sw_call(F, 3, 688)))
    assert (f["H"], f["hd"], f["base_bits"]) == (0, 0, 0)


# ---- policy worked by hand --------------------------------------------------------
def test_policy_llama7b_decode_chain():
    # bf16: 8 elements per 16 B. H = 4096 -> 512 vectors -> 2 per work-item ->
    # RN_BLOCK_2, one workgroup per row. RoPE: 64 heads x (64 / 8 = 8 lanes) =
    # 512 lanes -> two workgroups per token at decode sizes. T = 1 -> bucket 0
    # -> SwiGLU one vector per thread: 11008 / 8 = 1376 vectors -> 6 blocks.
    v, roles, launches = S.plan(S.make_key(chain_call(BF, 1, 4096, 11008, 32, 32, 128)), 1)
    assert v == S.CH_FUSED
    assert roles == (14, 31, 41)
    assert launches == [(50, 1 + 2 + 6, 256)]


def test_policy_gqa_decode_chain():
    # T = 8 -> bucket 3: norm one block per row (8); RoPE 40 heads x 8 lanes
    # = 320 -> two blocks per token (16); SwiGLU 8 * 14336 / 8 = 14336 vectors
    # -> 56 blocks.
    v, roles, launches = S.plan(S.make_key(chain_call(BF, 8, 4096, 14336, 32, 8, 128,
                                                      base=500000.0)), 8)
    assert (v, roles, launches) == (S.CH_FUSED, (14, 31, 41), [(50, 8 + 16 + 56, 256)])


def test_policy_prefill_chain():
    # T = 8192 -> bucket 13, beyond decode sizes: H = 8192 bf16 -> 1024 vectors
    # -> 4 per work-item -> RN_BLOCK_4, one block per row (8192); RoPE one token
    # per block (8192 blocks, no head slices beyond decode sizes); SwiGLU role
    # 8192 * 28672 / 8 = 29360128 vectors, one per work-item, streaming ->
    # 114688 blocks.
    v, roles, launches = S.plan(S.make_key(chain_call(BF, 8192, 8192, 28672, 64, 8, 128,
                                                      base=500000.0)), 8192)
    assert (v, roles) == (S.CH_FUSED, (15, 31, 42))
    assert launches == [(50, 8192 + 8192 + 114688, 256)]


def test_policy_qwen3_decode_chain_with_qk_norm():
    # As the Llama-7B decode, but the RoPE role is the QK-norm vector role (34)
    # and the key carries flag 0x40; SwiGLU 12288 / 8 = 1536 vectors -> 6 blocks.
    c = chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True)
    assert S.unpack_key(S.make_key(c))["flags"] == 0x7F
    v, roles, launches = S.plan(S.make_key(c), 1)
    assert (v, roles, launches) == (S.CH_FUSED, (14, 34, 41), [(50, 1 + 2 + 6, 256)])


def test_qk_norm_is_a_guard():
    # Same shapes with and without the head norm are different versions.
    plain = chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6)
    qkn = chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True)
    assert S.make_key(plain) != S.make_key(qkn)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    assert m.call(plain) == S.OK and m.call(qkn) == S.OK
    assert len(m.versions) == 2 and m.last.roles[1] == S.ROPE_QKN_VEC


def test_qk_norm_weight_alignment_selects_scalar_role():
    # A head-norm weight one element off 16 B drops the vector path; the
    # chain then runs as three launches with the scalar QK-norm role.
    c = qkn_call(BF, 4, 32, 8, 128, w_off=elem_offset(BF))
    assert S.plan(S.make_key(c), 4)[2] == [(S.ROPE_QKN_SCALAR, 4, 256)]
    c = qkn_call(BF, 4, 32, 8, 128)          # 40 heads x 8 lanes: two blocks per token
    assert S.plan(S.make_key(c), 4)[2] == [(S.ROPE_QKN_VEC, 8, 256)]
    ch = chain_call(BF, 4, 4096, 12288, 32, 8, 128, qk_norm=True, w_off=elem_offset(BF))
    v, roles, launches = S.plan(S.make_key(ch), 4)
    assert v == S.CH_SEQ and roles[1] == S.ROPE_QKN_SCALAR and len(launches) == 3


def test_qk_norm_without_k_heads_needs_no_k_weight():
    c = qkn_call(F, 2, 4, 0, 64, null=("k", "k_w"))
    assert S.validate(c) is None
    c = qkn_call(F, 2, 4, 4, 64, null=("k_w",))
    assert S.validate(c) == S.E_INVALID


def test_qk_eps_is_checked_only_with_the_head_norm():
    bad = float("nan")
    assert S.validate(chain_call(BF, 1, 256, 688, 4, 4, 64, qk_eps=bad)) is None
    assert S.validate(chain_call(BF, 1, 256, 688, 4, 4, 64, qk_norm=True,
                                 qk_eps=bad)) == S.E_INVALID


def test_policy_tiny_f32_chain():
    # f32: 4 per 16 B. H = 256 -> 64 vectors -> 1 per lane -> RN_WAVE_1.
    # hd 64 -> 32 pairs -> 8 vectors per half (power of two) -> ROPE_VEC.
    # SwiGLU 4 * 688 / 4 = 688 vectors -> 3 blocks.
    v, roles, launches = S.plan(S.make_key(chain_call(F, 4, 256, 688, 4, 4, 64)), 4)
    assert (v, roles, launches) == (S.CH_FUSED, (11, 31, 41), [(50, 1 + 4 + 3, 256)])


@pytest.mark.parametrize("H,dtype,want", [
    (64, F, (11, 2)), (256, BF, (11, 2)), (520, BF, (12, 2)), (1024, BF, (12, 2)),
    (1032, BF, (13, 5)), (4096, F, (15, 5)), (8192, F, (16, 5)), (16384, F, (17, 5)),
    (32768, BF, (17, 5)), (100, BF, (10, 5)), (4097, F, (10, 5)),
    # beyond 16 vectors per work-item (4096 vectors): split over
    # S = ceil(vectors / 2048) workgroups, T * S of them, up to S = 64
    (32776, BF, (20, 15)), (65536, BF, (20, 20)), (65544, BF, (20, 25)),
    (16388, F, (20, 15)), (32768, F, (20, 20)), (32772, F, (20, 25)),
    (1048576, BF, (20, 320)), (524288, F, (20, 320)),
    # S = 65: beyond the split and beyond 8192 vectors -> two passes
    (1048584, BF, (18, 5)), (524292, F, (18, 5))])
def test_rmsnorm_policy_by_row_size(H, dtype, want):
    # 5 rows (bucket 3): rows of <= 128 vectors take a wavefront each, 4 per
    # block (2 blocks); longer rows one block per row (5 blocks). bf16 32776
    # = f32 16388 = 4097 vectors -> 3 split workgroups per row; bf16 65536 =
    # f32 32768 = 8192 vectors -> 4; 8193 vectors -> 5; bf16 2^20 = f32 2^19
    # = 131072 vectors -> 64 (the most); one more vector -> 65: two passes.
    v, g = S.rn_role(dtype, H, S.ALIGN | S.CONTIG, 5, 3)
    assert (v, g) == want


@pytest.mark.parametrize("dtype,H,b,want", [
    # S = 64: scratch words 8 + 2^b * 65 <= 2^22 holds up to b = 15
    (BF, 1048576, 15, S.RN_SPLIT), (BF, 1048576, 16, S.RN_LOOP),
    # S = 3 (4097 vectors): 8 + 2^b * 4 <= 2^22 up to b = 19; beyond, the
    # row still fits a 1024-lane workgroup
    (BF, 32776, 19, S.RN_SPLIT), (BF, 32776, 20, S.RN_WIDE), (F, 16388, 22, S.RN_WIDE),
    # S = 4 (8192 vectors): 8 + 2^b * 5 <= 2^22 up to b = 19
    (F, 32768, 19, S.RN_SPLIT), (F, 32768, 20, S.RN_WIDE)])
def test_split_rows_need_their_scratch_to_fit(dtype, H, b, want):
    assert S.rn_role(dtype, H, S.ALIGN | S.CONTIG, 1, b)[0] == want


@pytest.mark.parametrize("dtype,H,b,want", [
    # plain rows of 4097..7168 vectors: the 1024-lane workgroup at any bucket
    (BF, 32776, 0, S.RN_WIDE), (BF, 57344, 3, S.RN_WIDE), (F, 28672, 22, S.RN_WIDE),
    (F, 16388, 19, S.RN_WIDE),
    # 7169..8192 vectors: split like residual rows (S = 4) up to bucket 8
    # (256 rows), the 1024-lane workgroups from bucket 9 on
    (BF, 57352, 3, S.RN_SPLIT), (BF, 65536, 8, S.RN_SPLIT), (BF, 65536, 9, S.RN_WIDE),
    (BF, 65536, 19, S.RN_WIDE), (BF, 65536, 20, S.RN_WIDE),
    (F, 32768, 3, S.RN_SPLIT), (F, 32768, 8, S.RN_SPLIT), (F, 32768, 9, S.RN_WIDE),
    (BF, 57352, 9, S.RN_WIDE),
    # 8193 vectors and more: split while the scratch fits (S = 5: 8 + 6 * 2^b
    # <= 2^22 up to b = 19), then two passes
    (BF, 65544, 19, S.RN_SPLIT), (BF, 65544, 20, S.RN_LOOP),
    # up to 4096 vectors the same as the residual rows
    (BF, 32768, 3, S.RN_BLOCK[16]), (F, 256, 3, S.RN_WAVE[1])])
def test_plain_rows_policy(dtype, H, b, want):
    assert S.rn_role(dtype, H, S.ALIGN | S.CONTIG, 1, b, res=False)[0] == want
    cands = [c.kernels[0] for c in S.candidates(S.make_key(rn_call(dtype, 1 << b, H)))]
    assert cands[0] == want
    if want == S.RN_WIDE:                       # tuning may still split, or loop
        assert cands[1:] == ([S.RN_SPLIT] if S.split_fits(dtype, H, b) else []) + [S.RN_LOOP]


@pytest.mark.parametrize("dtype, H, T, want", [
    # plain rows of 5120 and 7168 vectors: a workgroup per row up to 256
    # rows, then 256 workgroups, each taking every 256th row
    (BF, 57344, 1, 1), (BF, 40960, 100, 100), (BF, 57344, 256, 256), (BF, 57344, 257, 256),
    (BF, 57344, 2048, 256), (F, 28672, 300, 256)])
def test_plain_wide_rows_grid_by_hand(dtype, H, T, want):
    assert S.plan(S.make_key(rn_call(dtype, T, H)), T)[2] == [(S.RN_WIDE, want, 1024)]


def test_wide_rows_grid_of_candidates_by_hand():
    # bf16 rows of 65,536 (8192 vectors) at 2048 rows: plain rows take the
    # 1024-lane form by policy (256 workgroups); residual rows split by
    # policy and have it as a tuning candidate, one workgroup per row
    for call, want in ((rn_call(BF, 2048, 65536), 256), (res_call(BF, 2048, 65536), 2048)):
        key = S.make_key(call)
        wide = [c for c in S.candidates(key) if c.kernels == (S.RN_WIDE,)]
        assert len(wide) == 1
        assert S.cand_plan(key, wide[0], 2048)[2] == [(S.RN_WIDE, want, 1024)]
    # residual rows take the wide form when the split's scratch does not fit
    # (bucket 20), a workgroup per row
    assert S.rn_role(BF, 65536, S.ALIGN | S.CONTIG, 1 << 20, 20) == (S.RN_WIDE, 1 << 20)
    assert S.grid_of(S.RN_WIDE, BF, 2048, 57344) == 2048
    assert S.grid_of(S.RN_WIDE, BF, 2048, 57344, res=False) == 256


def test_split_scratch_layout_by_hand():
    # 3 rows of bf16 65536 (8192 vectors, 4 workgroups each): 8 header words,
    # 12 slots, 3 counters
    assert S.split_slices(BF, 65536) == 4 and S.split_words(3, 4) == 8 + 12 + 3
    assert S.grid_of(S.RN_SPLIT, BF, 3, 65536) == 12
    # f32 16388 = 4097 vectors: 3 workgroups, the last holds one vector
    assert S.split_slices(F, 16388) == 3


@pytest.mark.parametrize("T", [1, 8, 64, 65, 8192])
def test_rmsnorm_policy_does_not_depend_on_tokens(T):
    b = S.bucket(T)
    assert S.rn_role(BF, 4096, S.ALIGN | S.CONTIG, T, b) == (S.RN_BLOCK[2], T)
    assert S.rn_role(F, 256, S.ALIGN | S.CONTIG, T, b) == (S.RN_WAVE[1], -(-T // 4))


def test_unaligned_and_strided_layouts():
    off = elem_offset(BF)
    assert S.plan(S.make_key(rn_call(BF, 2, 4096, off=off)), 2)[0] == S.RN_SCALAR
    # a padded row stride that keeps 16 B alignment stays vectorised
    assert S.plan(S.make_key(rn_call(BF, 2, 4096, pad=64)), 2)[0] == 14
    assert S.plan(S.make_key(sw_call(BF, 2, 11008, pad=64)), 2)[0] == S.SW_ROWS
    assert S.plan(S.make_key(sw_call(BF, 2, 11008, off=off)), 2)[0] == S.SW_SCALAR
    assert S.plan(S.make_key(sw_call(BF, 2, 11003, pad=1)), 2)[0] == S.SW_SCALAR
    assert S.plan(S.make_key(rope_call(BF, 2, 32, 32, 128, off=off)), 2)[0] == S.ROPE_SCALAR
    # hd 96 bf16: 48 pairs = 6 vectors per half, not a power of two
    assert S.plan(S.make_key(rope_call(BF, 2, 4, 4, 96)), 2)[0] == S.ROPE_SCALAR
    c = chain_call(BF, 4, 4096, 11008, 32, 32, 128, sw_pad=64)
    v, roles, launches = S.plan(S.make_key(c), 4)
    assert v == S.CH_SEQ and roles == (14, 31, S.SW_ROWS) and len(launches) == 3


def test_chain_key_keeps_per_role_flags():
    a = chain_call(BF, 4, 4096, 11008, 32, 32, 128, sw_pad=64)
    b = chain_call(BF, 4, 4096, 11008, 32, 32, 128, rope_pad=64)
    assert S.make_key(a) != S.make_key(b)
    assert S.plan(S.make_key(a), 4)[1] != S.plan(S.make_key(b), 4)[1]


def test_swiglu_flat_grid_cap_and_tail():
    # 3 * 5 = 15 f32 elements: 3 whole vectors + a 3-element tail -> 1 block
    assert S.sw_role(F, 5, 3, False, 3) == (S.SW_FLAT, 1)
    # 1 element: no whole vector, still one block for the tail
    assert S.sw_role(F, 1, 3, False, 1) == (S.SW_FLAT, 1)
    assert S.sw_role(BF, 1 << 30, 3, True, 1024) == (S.SW_FLAT_NT, S.GRID_CAP)
    # 65 tokens x 1024 bf16: 8320 vectors -> 33 blocks
    assert S.sw_role(BF, 1024, 3, True, 65) == (S.SW_FLAT_NT, 33)


def test_swiglu_streams_beyond_320_mib():
    # bytes at the top of the bucket: 3 * T * I * 2 for bf16 SwiGLU
    MiB = 1 << 20
    k = S.make_key(sw_call(BF, 2048, 28672))             # 3 * 2048 * 28672 * 2 = 336 MiB
    assert S.call_bytes(k) == 336 * MiB and S.plan(k, 2048)[0] == S.SW_FLAT_NT
    k = S.make_key(sw_call(BF, 1500, 28672))             # same bucket (11): 2048 at the top
    assert S.plan(k, 1500)[0] == S.SW_FLAT_NT
    k = S.make_key(sw_call(BF, 1024, 28672))             # 168 MiB
    assert S.call_bytes(k) == 168 * MiB and S.plan(k, 1024)[0] == S.SW_FLAT
    k = S.make_key(sw_call(BF, 1, 1 << 30))              # one token, 6 GiB: streams
    assert S.plan(k, 1)[0] == S.SW_FLAT_NT
    # the chain counts norm rows, whole Q/K heads and SwiGLU: Llama-7B shapes
    # at 2048 tokens: 2048 * 2 * (4 * 4096 + 2 * 64 * 128 + 3 * 11008) = 263 MiB
    k = S.make_key(chain_call(BF, 2048, 4096, 11008, 32, 32, 128))
    assert S.call_bytes(k) == 2048 * 2 * (4 * 4096 + 2 * 64 * 128 + 3 * 11008)
    assert S.plan(k, 2048)[1][2] == S.SW_FLAT
    k = S.make_key(chain_call(BF, 4096, 4096, 11008, 32, 32, 128))   # 526 MiB
    assert S.plan(k, 4096)[1][2] == S.SW_FLAT_NT


# ---- Algorithm 1 and the three paths ---------------------------------------------
def test_miss_install_hit_and_order():
    m = S.SpecCacheModel()
    a = rn_call(BF, 1, 4096)
    b = rn_call(BF, 3, 4096)          # bucket 2: a different specialization
    assert m.call(a) == S.MISS and m.last.n_launches == 0 and m.launch_count == 0
    assert m.install_last_miss()[0] == S.OK
    assert m.call(a) == S.OK and m.last.version == 0
    assert m.call(b) == S.MISS
    st, rec = m.install_last_miss()
    assert st == S.OK and rec.version == 1
    assert m.call(b) == S.OK and m.last.version == 1
    assert m.call(a) == S.OK and m.last.version == 0
    assert m.versions[0] != m.versions[1]
    s = m.stats
    assert (s.calls, s.hits, s.misses, s.errors, s.installs) == (5, 3, 2, 0, 2)
    assert m.version_hits == [2, 1]


def test_install_is_idempotent_and_needs_a_miss():
    m = S.SpecCacheModel()
    assert m.install_last_miss()[0] == S.E_INVALID
    c = sw_call(F, 4, 688)
    m.call(c)
    m.call(c)
    assert m.install_last_miss()[0] == S.OK
    assert m.install_last_miss()[0] == S.OK
    assert len(m.versions) == 1 and m.stats.installs == 1


def test_capacity_is_enforced():
    m = S.SpecCacheModel(capacity=2)
    for T in (1, 2, 4):
        assert m.call(sw_call(BF, T, 128)) == S.MISS
        st, _ = m.install_last_miss()
    assert st == S.E_FULL and len(m.versions) == 2


def test_errors_never_install_or_launch():
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    bad = [rn_call(BF, 1, 4096, null=("x",)), rn_call(BF, -1, 4096), rn_call(BF, 1, 0),
           rn_call(BF, 1, 4096, eps=float("nan")), rn_call(BF, 1, 4096, eps=-1.0),
           rope_call(BF, 1, 4, 4, 63), rope_call(BF, 1, 4, 4, 64, base=1.0),
           rope_call(BF, 1, 4, 4, 64, pos_off=2), rope_call(BF, 1, 0, 4, 64),
           sw_call(BF, 1, 0), rn_call(7, 1, 4096)]
    for c in bad:
        assert m.call(c) == S.E_INVALID
    assert m.call(rn_call(BF, S.T_MAX + 1, 64)) == S.E_UNSUPPORTED
    assert m.call(rope_call(BF, 1, 4, 4, 1024)) == S.E_UNSUPPORTED
    assert m.call(rn_call(BF, 1, S.H_LIMIT)) == S.E_UNSUPPORTED
    assert m.versions == [] and m.launch_count == 0
    assert m.stats.errors == len(bad) + 3


def test_empty_call_is_ok_and_launches_nothing():
    m = S.SpecCacheModel()
    assert m.call(rn_call(BF, 0, 4096, null=("x", "y"))) == S.OK
    assert m.last.n_launches == 0 and m.stats.empty == 1 and m.versions == []


def test_launch_error_stops_dispatch():
    m = S.SpecCacheModel()
    c = chain_call(BF, 4, 4096, 11008, 32, 32, 128, sw_pad=64)     # three launches
    m.call(c)
    m.install_last_miss()
    m.launch_fails = {1}
    assert m.call(c) == S.E_LAUNCH
    assert m.launch_count == 2                       # the third launch never issued
    assert len(m.versions) == 1 and m.stats.errors == 1 and m.version_hits == [0]


def test_auto_install_counts_one_miss():
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    c = rn_call(BF, 1, 4096)
    assert m.call(c) == S.OK and m.call(c) == S.OK
    s = m.stats
    assert (s.calls, s.hits, s.misses, s.installs) == (2, 1, 1, 1)


def test_stats_invariant_over_mixed_stream():
    import workloads as wl
    m = S.SpecCacheModel()
    for T, dt, layout in wl.mixed_stream(n=2000):
        d = BF if dt == wl.BF16 else F
        off = elem_offset(d) if layout == wl.LAYOUT_UNALIGNED else 0
        pad = wl.MIXED_PAD if layout == wl.LAYOUT_STRIDED else 0
        c = chain_call(d, T, 4096, 11008, 32, 32, 128, res_off=off, rope_off=off,
                       sw_off=off, res_pad=pad, rope_pad=pad, sw_pad=pad)
        if m.call(c) == S.MISS:
            m.install_last_miss()
            assert m.call(c) == S.OK
    s = m.stats
    assert s.calls == s.hits + s.misses + s.errors + s.empty
    assert len(set(m.versions)) == len(m.versions) <= 9 * 2 * 3
    assert s.misses == len(m.versions)


def test_rope_head_slices_worked_by_hand():
    # slices = min(4, ceil(heads * lanes / 256)) for vector RoPE roles at
    # decode sizes (bucket <= 6), else 1
    # bf16 hd 128: 8 lanes per head. 64 + 8 heads -> 576 lanes -> 3.
    assert S.plan(S.make_key(rope_call(BF, 2, 64, 8, 128)), 2)[2] == [(S.ROPE_VEC, 6, 256)]
    # f32 hd 128: 16 lanes per head. 64 + 8 heads -> 1152 lanes -> capped at 4.
    assert S.plan(S.make_key(rope_call(F, 2, 64, 8, 128)), 2)[2] == [(S.ROPE_VEC, 8, 256)]
    # 4 + 4 heads of 64 (bf16: 4 lanes) -> 32 lanes -> 1.
    assert S.plan(S.make_key(rope_call(BF, 3, 4, 4, 64)), 3)[2] == [(S.ROPE_VEC, 3, 256)]
    # beyond decode sizes (T = 65 -> bucket 7): one block per token.
    assert S.plan(S.make_key(rope_call(BF, 65, 64, 8, 128)), 65)[2] == [(S.ROPE_VEC, 65, 256)]
    # scalar roles never split.
    c = rope_call(BF, 2, 64, 8, 128, off=elem_offset(BF))
    assert S.plan(S.make_key(c), 2)[2] == [(S.ROPE_SCALAR, 2, 256)]
