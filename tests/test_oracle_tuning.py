"""Pins for the tuning part of the selection model: the candidate plans of a
key, the choice rule, and the tuning call's operand sizes (CPU only).

The Triton autotuner the paper describes (Sec. 2) times a set of candidate
configurations and keeps the fastest; here a key's candidates are the kernel
variants whose preconditions the key guarantees. Lists below are worked by
hand from the kernels' stated requirements; the property tests restate those
requirements independently of the candidate function.
"""
import pytest

from oracle import selection as S
from tests.selection_calls import (add_call, chain_call, elem_offset, emb_call, mf_call,
                                   qkn_call, res_call, rn_call, rope_call, silu_call, sw_call)

BF, F = S.DT_BF16, S.DT_F32
Cand = S.Cand
Z = (0, 0, 0)


def key_of(call):
    return S.make_key(call)


# ---- candidate lists worked by hand --------------------------------------------------
def test_llama7b_decode_chain_candidates():
    # Policy roles (14 = RN_BLOCK_2, 31 = ROPE_VEC, 41 = SW_FLAT), two head
    # slices (64 heads x 8 lanes = 512 lanes). The norm row (512 vectors) has
    # no other register layout; slices 2, 1, 4; SwiGLU cached then
    # nontemporal; last the three-launch sequence of the policy's roles.
    k = key_of(chain_call(BF, 1, 4096, 11008, 32, 32, 128))
    want = [Cand(50, (14, 31, w), (50,), s) for s in (2, 1, 4) for w in (41, 42)]
    want.append(Cand(51, (14, 31, 41), (14, 31, 41), 2))
    assert S.candidates(k) == want
    # grids at one token: norm 1 + RoPE 1 * slices + SwiGLU 1376 vectors / 256 = 6
    grids = [S.cand_plan(k, c, 1)[2] for c in want]
    assert grids[:6] == [[(50, 9, 256)]] * 2 + [[(50, 8, 256)]] * 2 + [[(50, 11, 256)]] * 2
    assert grids[6] == [(14, 1, 256), (31, 2, 256), (41, 6, 256)]


def test_tiny_f32_chain_candidates():
    # f32, H = 256 -> 64 vectors -> one wavefront per row (11 = RN_WAVE_1), also
    # one workgroup per row (13 = RN_BLOCK_1). hd = 64: 8 heads x 8 lanes = 64
    # lanes -> one slice by policy. 2 x 3 x 2 fused plans + the sequence.
    k = key_of(chain_call(F, 4, 256, 688, 4, 4, 64))
    want = [Cand(50, (r, 31, w), (50,), s) for r in (11, 13) for s in (1, 2, 4)
            for w in (41, 42)]
    want.append(Cand(51, (11, 31, 41), (11, 31, 41), 1))
    assert S.candidates(k) == want
    # T = 4: wavefront rows 4 per workgroup -> 1; workgroup rows -> 4; RoPE
    # 4 x slices; SwiGLU 4 * 688 / 4 = 688 vectors -> 3 workgroups
    assert S.cand_plan(k, want[0], 4)[2] == [(50, 1 + 4 + 3, 256)]
    assert S.cand_plan(k, want[6 + 4], 4)[2] == [(50, 4 + 16 + 3, 256)]


def test_prefill_chain_candidates():
    # Bucket 13: policy RN_BLOCK_4 (15), one token per RoPE workgroup (72
    # heads x 8 lanes fill 576 lanes), SwiGLU nontemporal (42). Geometry
    # options beyond decode sizes: 1, 2, 4 tokens per workgroup, then 2 and 4
    # slices (up to bucket 13).
    k = key_of(chain_call(BF, 8192, 8192, 28672, 64, 8, 128, base=500000.0))
    geo = [(1, 1), (1, 2), (1, 4), (2, 1), (4, 1)]
    want = [Cand(50, (15, 31, w), (50,), s, t) for s, t in geo for w in (42, 41)]
    want.append(Cand(51, (15, 31, 42), (15, 31, 42), 1, 1))
    assert S.candidates(k) == want
    # RoPE grids at 8192 tokens: 8192, 4096, 2048, 16384, 32768
    assert [S.cand_plan(k, c, 8192)[2][0][1] - 8192 - 114688 for c in want[:10:2]] == \
        [8192, 4096, 2048, 16384, 32768]


def test_slices_fixed_beyond_bucket_13():
    k = key_of(chain_call(BF, 8193, 8192, 28672, 64, 8, 128, base=500000.0))
    assert [c.slices for c in S.candidates(k)] == [1] * 7
    assert [c.tokens for c in S.candidates(k)] == [1, 1, 2, 2, 4, 4, 1]
    assert [c.roles[2] for c in S.candidates(k)] == [42, 41, 42, 41, 42, 41, 42]


@pytest.mark.parametrize("nq,nk,hd,dtype,b,want", [
    (8, 1, 128, BF, 13, 4),        # 9 heads x 8 lanes = 72 lanes: 256 / 72 -> 4
    (8, 8, 128, BF, 13, 2),        # 128 lanes -> 2
    (9, 9, 128, BF, 7, 2),         # 144 lanes -> ceil(1.8) = 2
    (16, 16, 128, BF, 7, 1),       # 256 lanes: full
    (64, 8, 128, BF, 13, 1),       # 576 lanes
    (4, 4, 64, F, 9, 4),           # f32 hd 64: 8 heads x 8 lanes = 64 -> 4
    (8, 1, 128, BF, 6, 1),         # decode sizes: one token per workgroup
    (1, 0, 16, BF, 10, 4),         # one head of one vector
])
def test_rope_tokens_worked_by_hand(nq, nk, hd, dtype, b, want):
    T = 1 << b
    f = S.unpack_key(key_of(rope_call(dtype, T, nq, nk, hd)))
    assert f["bucket"] == b
    assert S.rope_tokens(dtype, hd, False, nq + nk, b, S.ROPE_VEC) == want
    assert S.rope_tokens(dtype, hd, False, nq + nk, b, S.ROPE_SCALAR) == 1
    # the RoPE op's grid at T tokens
    assert S.plan(key_of(rope_call(dtype, T, nq, nk, hd)), T)[2] == \
        [(S.ROPE_VEC, -(-T // want), 256)]


def test_tp8_shard_chain_policy():
    # One GPU's share of the 8192-token prefill under 8-way tensor
    # parallelism: norm rows (8192) + RoPE 4 tokens per workgroup (2048) +
    # SwiGLU 8192 * 3584 / 8 / 256 = 14336 workgroups.
    k = key_of(chain_call(BF, 8192, 8192, 3584, 8, 1, 128, base=5e5))
    assert S.plan(k, 8192) == (S.CH_FUSED, (15, 31, 42), [(50, 8192 + 2048 + 14336, 256)])
    # tiny f32 at 512 tokens: wavefront rows 128 + RoPE 128 + cached SwiGLU 344
    # (512 * 4 * (4 * 256 + 2 * 8 * 64 + 3 * 688) bytes: far below 320 MiB)
    k = key_of(chain_call(F, 512, 256, 688, 4, 4, 64))
    assert S.plan(k, 512) == (S.CH_FUSED, (11, 31, 41), [(50, 128 + 128 + 344, 256)])


def test_qwen3_chain_candidates_keep_the_qk_norm_role():
    k = key_of(chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True))
    cands = S.candidates(k)
    assert {c.roles[1] for c in cands} == {34}
    # 40 heads x 8 lanes = 320 lanes -> 2 slices by policy
    assert [c.slices for c in cands] == [2, 2, 1, 1, 4, 4, 2]


def test_unfused_chain_has_one_candidate():
    k = key_of(chain_call(BF, 1, 4096, 11008, 32, 32, 128, res_off=elem_offset(BF)))
    assert S.candidates(k) == [Cand(51, (10, 31, 41), (10, 31, 41), 2)]


@pytest.mark.parametrize("H,dtype,want,plain", [
    (512, BF, [11, 13, 18], None),       # 64 vectors: wavefront, workgroup, loop
    (1024, BF, [12, 13, 18], None),      # 128 vectors: two per lane of a wavefront
    (4096, BF, [14, 18], None),          # 512 vectors: workgroup x 2, loop
    (8200, BF, [16, 19, 18], None),      # 1025 vectors: workgroup x 8, 1024-lane workgroup, loop
    (32768, BF, [17, 19, 20, 18], None),  # 4096 vectors: x 16, 1024 lanes, 2-way split, loop
    # 8192 vectors: 4-way split, 1024-lane workgroup x 8, loop
    (65536, BF, [20, 19, 18], None),
    # 7168 vectors: residual rows 4-way split, 1024-lane workgroup x 7, loop;
    # plain rows the 1024-lane workgroup first, then the split, then the loop
    (57344, BF, [20, 19, 18], [19, 20, 18]),
    (65544, BF, [20, 18], None),         # 8193 vectors: 5-way split, loop (too long for 1024 lanes)
    (32768, F, [20, 19, 18], None),          # 8192 f32 vectors
    (28672, F, [20, 19, 18], [19, 20, 18]),  # 7168 f32 vectors
    (1048584, BF, [18], None),           # 131073 vectors: 65 workgroups is too many -> loop only
    (100, BF, [10], None),               # ragged: scalar only
])
def test_rmsnorm_candidates(H, dtype, want, plain):
    for mk, w in ((rn_call, plain or want), (res_call, want)):
        cands = S.candidates(key_of(mk(dtype, 3, H)))
        assert [c.variant for c in cands] == w
        assert all(c.kernels == (c.variant,) and c.slices == 1 for c in cands)


def test_unaligned_rmsnorm_has_one_candidate():
    assert [c.variant for c in S.candidates(key_of(rn_call(BF, 1, 4096, off=2)))] == [10]


def test_rope_candidates():
    # GQA decode, T = 8: 40 heads x 8 lanes -> 2 slices; then 1, 4; then scalar.
    k = key_of(rope_call(BF, 8, 32, 8, 128, base=500000.0))
    assert S.candidates(k) == [Cand(31, Z, (31,), 2), Cand(31, Z, (31,), 1),
                               Cand(31, Z, (31,), 4), Cand(30, Z, (30,), 1)]
    assert [S.cand_plan(k, c, 8)[2][0][1] for c in S.candidates(k)] == [16, 8, 32, 8]
    # four slices by policy (128 heads x 8 lanes = 1024 lanes)
    k = key_of(rope_call(BF, 1, 64, 64, 128))
    assert [c.slices for c in S.candidates(k)] == [4, 1, 2, 1]
    # QK norm: the scalar alternative is the QK-norm scalar kernel (33)
    k = key_of(qkn_call(BF, 1, 32, 8, 128))
    assert [c.variant for c in S.candidates(k)] == [34, 34, 34, 33]
    # scalar policy (unaligned): nothing else
    k = key_of(rope_call(BF, 1, 32, 32, 128, off=2))
    assert S.candidates(k) == [Cand(30, Z, (30,), 1)]


def test_swiglu_candidates():
    assert [c.variant for c in S.candidates(key_of(sw_call(BF, 1, 11008)))] == [41, 42, 43]
    assert [c.variant for c in S.candidates(key_of(sw_call(BF, 128, 11008)))] == [41, 42, 43]
    # 4096 tokens x 28672: 672 MiB at the top of the bucket, streaming first
    assert [c.variant for c in S.candidates(key_of(sw_call(BF, 4096, 28672)))] == [42, 41, 43]
    # f32 rows of 688 = 172 vectors
    assert [c.variant for c in S.candidates(key_of(sw_call(F, 3, 688)))] == [41, 42, 43]
    # rows of 690 f32 are not 16-byte multiples: element-wise only
    assert [c.variant for c in S.candidates(key_of(sw_call(F, 4, 690)))] == [40]
    # aligned rows with padding: rows only; unaligned: scalar only
    assert [c.variant for c in S.candidates(key_of(sw_call(BF, 4, 4096, pad=8)))] == [43]
    assert [c.variant for c in S.candidates(key_of(sw_call(BF, 4, 4096, off=2)))] == [40]


def test_short_op_candidates():
    assert [c.variant for c in S.candidates(key_of(add_call(BF, 8192, 8192)))] == [62, 61, 63]
    assert [c.variant for c in S.candidates(key_of(silu_call(BF, 1, 4096)))] == [61, 62, 63]
    assert [c.variant for c in S.candidates(key_of(mf_call(BF, 2, 4096)))] == [61, 62, 63]
    assert [c.variant for c in S.candidates(key_of(add_call(BF, 2, 4096, pad=8)))] == [63]
    assert [c.variant for c in S.candidates(key_of(emb_call(BF, 8, 4096, 1000)))] == [71]
    # ELT_FLAT_U2 grid: two vectors per work-item
    k = key_of(add_call(BF, 8192, 8192))
    assert S.cand_plan(k, S.candidates(k)[0], 8192)[2] == [(62, 8192 * 8192 // 8 // 512, 256)]


# ---- properties: every candidate meets its kernels' requirements ---------------------
def _zoo():
    out = []
    for T in (1, 3, 8, 64, 512, 8192, 8193):
        out += [chain_call(BF, T, 4096, 11008, 32, 32, 128),
                chain_call(BF, T, 8192, 28672, 64, 8, 128, base=500000.0),
                chain_call(F, T, 256, 688, 4, 4, 64),
                chain_call(BF, T, 512, 1024, 8, 2, 64, qk_norm=True),
                chain_call(BF, T, 4096, 11008, 32, 32, 128, sw_pad=8),
                rn_call(BF, T, 512), rn_call(F, T, 4096), res_call(BF, T, 8192),
                rope_call(BF, T, 32, 8, 128), rope_call(F, T, 4, 4, 64),
                qkn_call(BF, T, 16, 16, 256), sw_call(BF, T, 14336), sw_call(F, T, 690),
                add_call(BF, T, 4096), silu_call(F, T, 1000), mf_call(BF, T, 64)]
    return out


def _rows_fit(variant, nvec):
    """Register layouts: a wavefront holds 64 vectors per register slot, a
    workgroup 256."""
    for n, v in S.RN_WAVE.items():
        if variant == v:
            return nvec <= 64 * n
    for n, v in S.RN_BLOCK.items():
        if variant == v:
            return nvec <= 256 * n
    return True


@pytest.mark.parametrize("call", _zoo(), ids=lambda c: f"op{c.op}-T{c.T}")
def test_candidates_meet_kernel_requirements(call):
    k = key_of(call)
    f = S.unpack_key(k)
    v = 16 // S.elem_size(f["dtype"])
    cands = S.candidates(k)
    # index 0 is the policy's plan, at every token count of the bucket
    for T in {call.T, 1 << f["bucket"]}:
        assert S.cand_plan(k, cands[0], T) == S.plan(k, T)
    assert len(set(cands)) == len(cands)                       # no duplicates
    for c in cands:
        assert 1 <= c.slices <= 4 and c.tokens in (1, 2, 4)
        assert c.slices == 1 or c.tokens == 1
        if c.tokens > 1:
            assert f["bucket"] > S.DECODE_BUCKET_MAX
        if c.variant == S.CH_FUSED:
            rn, ro, sw = c.roles
            assert f["flags"] & 0x3F == 0x3F
            assert rn in S.RN_WAVE.values() or rn in S.RN_BLOCK.values()
            assert _rows_fit(rn, f["H"] // v) and f["H"] % v == 0
            assert ro in S.ROPE_VEC_ROLES and sw in (S.SW_FLAT, S.SW_FLAT_NT)
        for kv in c.kernels:
            if kv in (S.SW_FLAT, S.SW_FLAT_NT, S.SW_ROWS, S.ELT_FLAT, S.ELT_FLAT_U2,
                      S.ELT_ROWS) or kv in S.ROPE_VEC_ROLES:
                # vector kernels need the aligned guard of their role
                fl = f["flags"]
                if f["op"] == S.OP_CHAIN:
                    fl = (fl >> (2 if kv in S.ROPE_VEC_ROLES else 4)) & 3
                assert fl & S.ALIGN
                if kv in (S.SW_FLAT, S.SW_FLAT_NT, S.ELT_FLAT, S.ELT_FLAT_U2):
                    assert fl & S.CONTIG
                if kv in (S.SW_ROWS, S.ELT_ROWS):
                    width = f["I"] if kv == S.SW_ROWS else f["H"]
                    assert width % v == 0
            if kv in S.RN_WAVE.values() or kv in S.RN_BLOCK.values():
                assert _rows_fit(kv, f["H"] // v)
        if c.slices > 1:
            assert f["bucket"] <= S.SLICE_BUCKET_MAX
            assert (c.variant == S.CH_FUSED and c.roles[1] in S.ROPE_VEC_ROLES) or \
                any(kv in S.ROPE_VEC_ROLES for kv in c.kernels)


def test_candidate_counts_are_bounded():
    worst = 0
    for call in _zoo():
        worst = max(worst, len(S.candidates(key_of(call))))

    # beyond decode sizes: 2 norm layouts x 5 geometries x 2 SwiGLU forms + 1
    assert worst <= 21


# ---- the choice rule -------------------------------------------------------------------
@pytest.mark.parametrize("times,want", [
    ([1.0, 0.5], 1),
    ([1.0, 0.98], 0),              # within the margin: the policy's plan stays
    ([1.0, 0.96], 1),
    ([1.0, 0.5, 0.5], 1),          # first of equals
    ([0.5, 0.4, 0.3], 2),
    ([0.3, 0.4, 0.5], 0),
    ([2.0], 0),
])
def test_tune_choice(times, want):
    assert S.tune_choice(times) == want


# ---- operand bytes of the tuning call ----------------------------------------------------
def test_tune_operand_bytes_worked_by_hand():
    # RMSNorm bf16 H = 4096, one token: x and y rows + the weight.
    assert S.tune_operand_bytes(key_of(rn_call(BF, 1, 4096))) == 2 * 4096 * 2 + 4096 * 2
    # padded rows (aligned, not contiguous): stride = next multiple of 8 above 100
    k = key_of(rn_call(BF, 3, 100, pad=4))
    assert S.unpack_key(k)["flags"] == S.ALIGN
    assert S.tune_operand_bytes(k) == 2 * 4 * 104 * 2 + 100 * 2
    # Llama-7B decode chain, one token: norm 4 rows + weight; q, k, positions;
    # gate, up, out.
    k = key_of(chain_call(BF, 1, 4096, 11008, 32, 32, 128))
    assert S.tune_operand_bytes(k) == (4 * 4096 * 2 + 8192) + (4096 * 2 * 2 + 4) + 3 * 11008 * 2
    # masked_fill: data rows in elements, the mask in bytes; bucket 2 -> 4 tokens
    assert S.tune_operand_bytes(key_of(mf_call(BF, 3, 64))) == 2 * 4 * 64 * 2 + 4 * 64


def test_tune_tokens_is_the_top_of_the_bucket():
    for T, want in ((1, 1), (2, 2), (3, 4), (5, 8), (8192, 8192), (8193, 16384)):
        assert S.tune_tokens(key_of(sw_call(BF, T, 4096))) == want


# ---- the cache model with tuning ---------------------------------------------------------
def _timer(fast):
    """Candidate `fast` takes 1 ms, every other 2 ms."""
    return lambda key, i, c: 1.0 if i == fast else 2.0


def test_model_keeps_the_measured_candidate():
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE, timer=_timer(3))
    c = chain_call(BF, 1, 4096, 11008, 32, 32, 128)
    assert m.call(c) == S.OK
    assert (m.choice, m.tuned) == ([3], [S.TUNE_MEASURED])
    # candidate 3 = fused, one slice, nontemporal SwiGLU: grid 1 + 1 + 6
    assert m.last.roles == (14, 31, 42) and m.last.launch[0] == (50, 8, 256)
    assert m.call(c) == S.OK and m.stats.hits == 1


def test_model_policy_plan_without_tuning_or_within_margin():
    c = chain_call(BF, 1, 4096, 11008, 32, 32, 128)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    m.call(c)
    assert (m.choice, m.tuned) == ([0], [S.TUNE_NONE])
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE,
                         timer=lambda key, i, cand: 1.0 - 0.004 * i)
    m.call(c)
    assert (m.choice, m.tuned) == ([0], [S.TUNE_MEASURED])
    # one candidate: nothing to time
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE, timer=None)
    m.call(emb_call(BF, 8, 4096, 100))
    assert (m.choice, m.tuned) == ([0], [S.TUNE_NONE])


def test_model_skips_tuning_beyond_the_scratch_limit():
    # 2^22 tokens of a 4096-wide SwiGLU: 3 * 2^22 * 4096 * 2 B = 96 GiB
    c = sw_call(BF, 1 << 22, 4096)
    assert S.tune_operand_bytes(key_of(c)) > S.TUNE_SCRATCH_MAX
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_AUTOTUNE, timer=_timer(1))
    m.call(c)
    assert (m.choice, m.tuned) == ([0], [S.TUNE_SKIPPED])


def test_model_install_key_pins_a_candidate():
    k = key_of(rope_call(BF, 8, 32, 8, 128, base=500000.0))
    m = S.SpecCacheModel(flags=S.FLAG_AUTOTUNE, timer=_timer(1))
    assert m.install_key(k, 4) == S.E_INVALID            # 4 candidates
    assert m.install_key(k, -2) == S.E_INVALID
    assert m.install_key(k, 3) == S.OK
    assert (m.choice, m.tuned) == ([3], [S.TUNE_NONE])
    assert m.install_key(k, 1) == S.OK                   # idempotent: no change
    assert m.choice == [3]
    m.call(rope_call(BF, 8, 32, 8, 128, base=500000.0))
    assert m.last.variant == S.ROPE_SCALAR and m.last.launch[0] == (30, 8, 256)
    bad = list(k)
    bad[0] |= 0xF0   # op 0xF3 is not an op
    assert m.install_key(tuple(bad), 0) == S.E_INVALID
