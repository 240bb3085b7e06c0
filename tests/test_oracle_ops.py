"""Pins for the oracle's ops (CPU only).

Each test pins the oracle to something other than its own formula: a
closed form, a library routine (torch.nn.functional, numpy complex
arithmetic, math.pow), brute force, or an invariant of the operation.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ops
from oracle import numerics as nm
import workloads as wl


@pytest.fixture(scope="module")
def golden(golden_dir):
    with open(os.path.join(golden_dir, "closed_forms.json")) as f:
        return {k: v["value"] for k, v in json.load(f).items() if not k.startswith("_")}


def f32(a):
    return np.asarray(a, dtype=np.float32)


def within_ulps_f32(a, b, n=1):
    a, b = f32(a), f32(b)
    ai = a.view(np.int32).astype(np.int64)
    bi = b.view(np.int32).astype(np.int64)
    ai = np.where(ai < 0, -(ai & 0x7FFFFFFF), ai)
    bi = np.where(bi < 0, -(bi & 0x7FFFFFFF), bi)
    return np.abs(ai - bi) <= n


# ---- RMSNorm -----------------------------------------------------------------
@pytest.mark.parametrize("c", [0.75, -3.0, 1e-3, 40.0])
@pytest.mark.parametrize("eps", [0.0, 1e-6, 1.0])
def test_rmsnorm_constant_row(c, eps):
    H = 64
    x = f32(np.full((1, H), c))
    y = ops.rmsnorm(x, f32(np.ones(H)), eps, nm.F32)
    e = float(np.float32(eps))
    c = float(np.float32(c))
    want = c / math.sqrt(c * c + e)
    assert np.all(y == np.float32(want))
    if eps == 0.0:
        assert np.all(y == np.float32(math.copysign(1.0, c)))


@pytest.mark.parametrize("H", [1, 7, 256, 4096])
def test_rmsnorm_one_hot(H):
    x = np.zeros((2, H), np.float32)
    x[0, H // 2] = 2.5
    x[1, 0] = -0.125
    y = ops.rmsnorm(x, f32(np.ones(H)), 0.0, nm.F32)
    assert y[0, H // 2] == np.float32(math.sqrt(H))
    assert y[1, 0] == np.float32(-math.sqrt(H))
    assert np.count_nonzero(y) == 2


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_rmsnorm_matches_torch_rms_norm_fp64(dtype):
    cfg = wl.TINY_F32 if dtype == nm.F32 else wl.GQA_DECODE
    inp = wl.host_inputs(cfg)
    x, w = inp["x"], inp["w"]
    y = ops.rmsnorm(x, w, 1e-6, dtype)
    xt = torch.from_numpy(nm.values(x, dtype))
    wt = torch.from_numpy(nm.values(w, dtype))
    ref = F.rms_norm(xt, (xt.shape[-1],), wt, float(np.float32(1e-6))).numpy()
    want = nm.round_to(ref, dtype)
    if dtype == nm.F32:
        assert within_ulps_f32(y, want).all()
    else:
        assert (nm.bf16_ulp_distance(y, want) <= 1).all()
        assert np.mean(y == want) > 0.999


def test_rmsnorm_scale_invariance_and_unit_rms():
    rng = np.random.Generator(np.random.PCG64(5))
    x = rng.standard_normal((8, 512)).astype(np.float32)
    w = f32(np.ones(512))
    y1 = ops.rmsnorm(x, w, 0.0, nm.F32)
    y2 = ops.rmsnorm(x * np.float32(8.0), w, 0.0, nm.F32)     # exact scaling
    assert np.array_equal(y1, y2)
    ms = np.mean(y1.astype(np.float64) ** 2, axis=-1)
    assert np.allclose(ms, 1.0, rtol=1e-6)


def test_rmsnorm_weight_is_per_column():
    x = f32(np.ones((3, 4)))
    w = f32([1.0, 2.0, -0.5, 0.0])
    y = ops.rmsnorm(x, w, 0.0, nm.F32)
    assert np.array_equal(y, np.tile(w, (3, 1)))


# ---- residual add ---------------------------------------------------------------
def test_residual_add_bf16_matches_torch_fp32_add_then_cast():
    inp = wl.host_inputs(wl.GQA_DECODE)
    h = ops.residual_add(inp["x"], inp["residual"], nm.BF16)
    xt = torch.from_numpy(inp["x"].view(np.int16).copy()).view(torch.bfloat16).float()
    rt = torch.from_numpy(inp["residual"].view(np.int16).copy()).view(torch.bfloat16).float()
    want = (xt + rt).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(h, want)


def test_residual_add_f32_is_ieee_add():
    inp = wl.host_inputs(wl.TINY_F32)
    h = ops.residual_add(inp["x"], inp["residual"], nm.F32)
    assert np.array_equal(h, inp["x"] + inp["residual"])


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_residual_rmsnorm_reduces_to_rmsnorm(dtype):
    cfg = wl.TINY_F32 if dtype == nm.F32 else wl.LLAMA7B_DECODE
    inp = wl.host_inputs(cfg)
    zero = np.zeros_like(inp["x"])
    y, h = ops.residual_rmsnorm(zero, inp["residual"], inp["w"], 1e-6, dtype)
    assert np.array_equal(h, inp["residual"])
    assert np.array_equal(y, ops.rmsnorm(inp["residual"], inp["w"], 1e-6, dtype))
    y2, h2 = ops.residual_rmsnorm(inp["x"], inp["residual"], inp["w"], 1e-6, dtype)
    assert np.array_equal(y2, ops.rmsnorm(h2, inp["w"], 1e-6, dtype))


# ---- RoPE ---------------------------------------------------------------------
@pytest.mark.parametrize("base,hd", [(10000.0, 64), (10000.0, 128), (500000.0, 128),
                                     (10000.0, 96), (123.5, 6)])
def test_inv_freq_is_correctly_rounded(base, hd, golden):
    inv = ops.rope_inv_freq(base, hd)
    assert inv.dtype == np.float32 and inv.shape == (hd // 2,)
    assert inv[0] == np.float32(golden["inv_freq_0"])
    for i in range(hd // 2):
        exact = math.pow(base, -2.0 * i / hd)         # independent evaluation
        v = inv[i]
        lo = np.nextafter(v, np.float32(0))
        hi = np.nextafter(v, np.float32(np.inf))
        err = abs(float(v) - exact)
        # nearest float32: both neighbours are farther (up to math.pow's error)
        assert err <= abs(float(lo) - exact) * (1 + 1e-9)
        assert err <= abs(float(hi) - exact) * (1 + 1e-9)
    assert np.all(np.diff(inv.astype(np.float64)) < 0)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_rope_position_zero_is_identity(dtype):
    rng = np.random.Generator(np.random.PCG64(7))
    q = wl.host_array(rng, (3, 4, 64), dtype)
    k = wl.host_array(rng, (3, 2, 64), dtype)
    qo, ko = ops.rope_qk(q, k, np.zeros(3, np.int32), 10000.0, dtype)
    assert np.array_equal(qo, q) and np.array_equal(ko, k)


def test_rope_unit_angle_one_hot(golden):
    # pair 0 has inv_0 = 1 exactly, so at pos 1 the angle is 1 rad.
    hd = 16
    q = np.zeros((1, 1, hd), np.float32)
    q[0, 0, 0] = 1.0
    qo, _ = ops.rope_qk(q, np.zeros((1, 0, hd), np.float32), np.array([1], np.int32),
                        10000.0, nm.F32)
    assert qo[0, 0, 0] == np.float32(golden["cos_1"])
    assert qo[0, 0, hd // 2] == np.float32(golden["sin_1"])
    q2 = np.zeros((1, 1, hd), np.float32)
    q2[0, 0, hd // 2] = 1.0                       # second half rotates to -sin
    qo2, _ = ops.rope_qk(q2, None, np.array([1], np.int32), 10000.0, nm.F32)
    assert qo2[0, 0, 0] == np.float32(-golden["sin_1"])
    assert qo2[0, 0, hd // 2] == np.float32(golden["cos_1"])
    others = np.delete(qo.ravel(), [0, hd // 2])
    assert not others.any()


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_rope_matches_complex_multiplication(dtype):
    # Rotate-half RoPE is the complex product (v1 + i v2) * exp(i theta).
    cfg = wl.TINY_F32 if dtype == nm.F32 else wl.GQA_DECODE
    inp = wl.host_inputs(cfg)
    q, pos = inp["q"], inp["pos"]
    if dtype == nm.BF16:
        pos = np.array([0, 1, 17, 255, 1023, 4096, 8000, 8191], np.int32)[: q.shape[0]]
    qo, _ = ops.rope_qk(q, None, pos, cfg.base, dtype)
    hd = q.shape[-1]
    half = hd // 2
    inv = np.array([math.pow(cfg.base, -2.0 * i / hd) for i in range(half)])
    theta = (pos.astype(np.float32)[:, None]
             * inv.astype(np.float32)[None, :]).astype(np.float64)
    v = nm.values(q, dtype)
    z = (v[..., :half] + 1j * v[..., half:]) * np.exp(1j * theta)[:, None, :]
    ref = np.concatenate([z.real, z.imag], axis=-1)
    want = nm.round_to(ref, dtype)
    if dtype == nm.F32:
        assert within_ulps_f32(qo, want, 2).all()
    else:
        assert (nm.bf16_ulp_distance(qo, want) <= 1).all()


def test_rope_preserves_pair_norms_and_inverts():
    rng = np.random.Generator(np.random.PCG64(8))
    q = rng.standard_normal((5, 3, 32)).astype(np.float32)
    pos = np.array([1, 10, 100, 1000, 8191], np.int32)
    qo, _ = ops.rope_qk(q, None, pos, 10000.0, nm.F32)
    n0 = q[..., :16].astype(np.float64) ** 2 + q[..., 16:].astype(np.float64) ** 2
    n1 = qo[..., :16].astype(np.float64) ** 2 + qo[..., 16:].astype(np.float64) ** 2
    assert np.allclose(n0, n1, rtol=1e-6, atol=1e-7)
    back, _ = ops.rope_qk(qo, None, -pos, 10000.0, nm.F32)   # angle(-p) = -angle(p)
    assert np.allclose(back, q, rtol=1e-5, atol=1e-6)


def test_rope_relative_position_property():
    rng = np.random.Generator(np.random.PCG64(9))
    hd = 64
    q = rng.standard_normal((1, 1, hd)).astype(np.float32)
    k = rng.standard_normal((1, 1, hd)).astype(np.float32)

    def score(m, n):
        qm, _ = ops.rope_qk(q, None, np.array([m], np.int32), 10000.0, nm.F32)
        kn, _ = ops.rope_qk(k, None, np.array([n], np.int32), 10000.0, nm.F32)
        return float(np.dot(qm.ravel().astype(np.float64), kn.ravel().astype(np.float64)))

    for m, n, d in [(5, 2, 7), (10, 10, 3), (3, 9, 20)]:
        assert abs(score(m, n) - score(m + d, n + d)) < 1e-4


def test_rope_gqa_same_angles_for_every_head():
    inp = wl.host_inputs(wl.GQA_DECODE)
    q, pos = inp["q"], inp["pos"]
    k = q[:, :8].copy()
    qo, ko = ops.rope_qk(q, k, pos, 500000.0, nm.BF16)
    assert np.array_equal(ko, qo[:, :8])


# ---- SwiGLU ---------------------------------------------------------------------
def test_swiglu_closed_forms(golden):
    g = f32([0.0, 1.0, -1.0, 3.0, 200.0, -200.0, 88.0])
    u = f32([5.0, 1.0, 1.0, 0.0, 1.0, 1.0, 1.0])
    out = ops.swiglu(g, u, nm.F32)
    assert out[0] == 0.0
    assert out[1] == np.float32(golden["silu_1"])
    assert out[2] == np.float32(golden["silu_m1"])
    assert out[3] == 0.0
    assert out[4] == np.float32(200.0)            # silu(g) -> g
    assert out[5] == 0.0 and np.signbit(out[5])   # -> -0, never NaN
    assert out[6] == np.float32(88.0)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_swiglu_matches_torch_silu(dtype):
    cfg = wl.TINY_F32 if dtype == nm.F32 else wl.LLAMA7B_DECODE
    inp = wl.host_inputs(cfg)
    out = ops.swiglu(inp["gate"], inp["up"], dtype)
    g = torch.from_numpy(nm.values(inp["gate"], dtype))
    u = torch.from_numpy(nm.values(inp["up"], dtype))
    want = nm.round_to((F.silu(g) * u).numpy(), dtype)
    if dtype == nm.F32:
        assert within_ulps_f32(out, want).all()
    else:
        assert (nm.bf16_ulp_distance(out, want) <= 1).all()


def test_swiglu_gate_is_first_operand():
    g = f32([2.0])
    u = f32([-3.0])
    a = ops.swiglu(g, u, nm.F32)
    b = ops.swiglu(u, g, nm.F32)
    assert a[0] == np.float32(2.0 / (1 + math.exp(-2.0)) * -3.0)
    assert a[0] != b[0]


# ---- chain ---------------------------------------------------------------------
def test_chain_is_the_three_ops():
    inp = wl.host_inputs(wl.TINY_F32)
    out = ops.decode_chain(inp, 1e-6, 10000.0, nm.F32)
    y, h = ops.residual_rmsnorm(inp["x"], inp["residual"], inp["w"], 1e-6, nm.F32)
    q, k = ops.rope_qk(inp["q"], inp["k"], inp["pos"], 10000.0, nm.F32)
    assert np.array_equal(out["y"], y) and np.array_equal(out["res_out"], h)
    assert np.array_equal(out["q"], q) and np.array_equal(out["k"], k)
    assert np.array_equal(out["out"], ops.swiglu(inp["gate"], inp["up"], nm.F32))


# ---- QK-RMSNorm + RoPE ---------------------------------------------------------------
def test_qk_norm_rope_constant_heads_at_position_zero():
    # A head of constant value c with unit weights and eps 0 normalises to
    # sign(c) everywhere; position 0 rotates by nothing.
    q = np.full((2, 3, 64), -2.5, np.float32)
    k = np.full((2, 1, 64), 0.125, np.float32)
    ones = np.ones(64, np.float32)
    qo, ko = ops.qk_norm_rope(q, k, np.zeros(2, np.int32), 1e4, ones, ones, 0.0, nm.F32)
    assert np.all(qo == -1.0) and np.all(ko == 1.0)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_qk_norm_rope_matches_library_norm_and_complex_rotation(dtype):
    cfg = wl.QWEN3_8B_DECODE
    inp = wl.host_inputs(cfg, T=5)
    if dtype == nm.F32:
        inp = {k: (nm.values(v, nm.BF16).astype(np.float32) if v.dtype == np.uint16 else v)
               for k, v in inp.items()}
    q, qw, pos = inp["q"], inp["q_norm_w"], inp["pos"]
    qo, _ = ops.qk_norm_rope(q, None, pos, cfg.base, qw, None, 1e-6, dtype)
    # torch's RMSNorm over the head dimension in float64 (not rounded) ...
    qt = torch.from_numpy(nm.values(q, dtype))
    n = F.rms_norm(qt, (cfg.hd,), torch.from_numpy(nm.values(qw, dtype)),
                   float(np.float32(1e-6))).numpy()
    # ... then the rotation as a complex product, rounded once
    half = cfg.hd // 2
    inv = np.array([math.pow(cfg.base, -2.0 * i / cfg.hd) for i in range(half)])
    theta = (pos.astype(np.float32)[:, None] * inv.astype(np.float32)[None, :]).astype(np.float64)
    z = (n[..., :half] + 1j * n[..., half:]) * np.exp(1j * theta)[:, None, :]
    want = nm.round_to(np.concatenate([z.real, z.imag], axis=-1), dtype)
    if dtype == nm.F32:
        assert within_ulps_f32(qo, want, 2).all()
    else:
        assert (nm.bf16_ulp_distance(qo, want) <= 1).all()


def test_qk_norm_rope_rounds_once():
    # Rounding the normalised head to bf16 before the rotation would be a
    # second rounding; the op keeps it in full precision.
    cfg = wl.QWEN3_8B_DECODE
    inp = wl.host_inputs(cfg, T=3)
    qo, _ = ops.qk_norm_rope(inp["q"], None, inp["pos"], cfg.base, inp["q_norm_w"], None,
                             1e-6, nm.BF16)
    twice, _ = ops.rope_qk(ops.rmsnorm(inp["q"], inp["q_norm_w"], 1e-6, nm.BF16), None,
                           inp["pos"], cfg.base, nm.BF16)
    a = nm.values(qo, nm.BF16)
    b = nm.values(twice, nm.BF16)
    # the two differ only by the intermediate rounding: at most 2^-8 of the
    # head's largest normalised magnitude per element, plus the final roundings
    scale = np.abs(a).max(axis=-1, keepdims=True)
    assert (np.abs(a - b) <= scale * 2.0 ** -7).all()
    assert not np.array_equal(qo, twice)


def test_qk_norm_rope_preserves_head_rms_with_unit_weights():
    rng = np.random.Generator(np.random.PCG64(21))
    q = rng.standard_normal((4, 6, 128)).astype(np.float32) * np.float32(7.0)
    ones = np.ones(128, np.float32)
    qo, _ = ops.qk_norm_rope(q, None, np.array([0, 5, 500, 8000], np.int32), 5e5, ones, None,
                             0.0, nm.F32)
    ms = np.mean(qo.astype(np.float64) ** 2, axis=-1)     # rotation keeps the unit RMS
    assert np.allclose(ms, 1.0, rtol=1e-5)


def test_chain_with_qk_norm_is_norm_then_rope():
    inp = wl.host_inputs(wl.QWEN3_8B_DECODE)
    out = ops.decode_chain(inp, 1e-6, 1e6, nm.BF16)
    q, k = ops.qk_norm_rope(inp["q"], inp["k"], inp["pos"], 1e6, inp["q_norm_w"],
                            inp["k_norm_w"], 1e-6, nm.BF16)
    assert np.array_equal(out["q"], q) and np.array_equal(out["k"], k)
    plain = ops.rope_qk(inp["q"], inp["k"], inp["pos"], 1e6, nm.BF16)
    assert not np.array_equal(out["q"], plain[0])


# ---- short ops: silu, add, masked_fill, embedding --------------------------------
@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_silu_against_torch_float64(dtype):
    r = np.random.Generator(np.random.PCG64(21))
    x = wl.host_array(r, (7, 300), dtype, outliers=True)
    got = ops.silu(x, dtype)
    want = F.silu(torch.from_numpy(nm.values(x, dtype))).numpy()
    assert np.array_equal(got, nm.round_to(want, dtype))
    # closed forms: silu(0) = 0, silu(-200) = -0.0 (overflow branch), silu(+inf) = +inf
    z = nm.round_to(np.array([0.0, -200.0, np.inf, 1.0]), dtype)
    v = nm.values(ops.silu(z, dtype), dtype)
    assert v[0] == 0 and v[1] == 0 and np.signbit(v[1]) and np.isinf(v[2])
    assert v[3] == nm.values(nm.round_to(np.array([1 / (1 + math.exp(-1))]), dtype), dtype)[0]


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_add_rounds_the_exact_sum_like_torch(dtype):
    r = np.random.Generator(np.random.PCG64(22))
    a = wl.host_array(r, (5, 257), dtype, outliers=True)
    b = wl.host_array(r, (5, 257), dtype)
    got = ops.add(a, b, dtype)
    ta, tb = wl.to_torch(a, dtype), wl.to_torch(b, dtype)
    assert np.array_equal(got, wl.from_torch(ta + tb))     # torch: float32 add, one rounding
    # 1 + 2^-8 in bf16 is a tie: rounds to even (1.0); 1 + 3 * 2^-9 rounds up
    if dtype == nm.BF16:
        one = nm.round_to(np.array([1.0, 1.0]), dtype)
        d = nm.round_to(np.array([2.0 ** -8, 3 * 2.0 ** -9]), dtype)
        s = nm.values(ops.add(one, d, dtype), dtype)
        assert s[0] == 1.0 and s[1] == 1.0 + 2.0 ** -7


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_masked_fill_like_torch(dtype):
    r = np.random.Generator(np.random.PCG64(23))
    x = wl.host_array(r, (6, 129), dtype)
    mask = (r.random((6, 129)) < 0.3).astype(np.uint8) * r.integers(1, 256, (6, 129)).astype(np.uint8)
    for value in (-1e4, 0.1, float("-inf"), 3.0e38):
        got = ops.masked_fill(x, mask, value, dtype)
        t = wl.to_torch(x, dtype).masked_fill(torch.from_numpy(mask != 0), value)
        assert np.array_equal(got, wl.from_torch(t))
    assert np.array_equal(ops.masked_fill(x, np.zeros_like(mask), 5.0, dtype), x)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_embedding_like_torch_and_zero_rows(dtype):
    r = np.random.Generator(np.random.PCG64(24))
    table = wl.host_array(r, (50, 64), dtype)
    ids = r.integers(0, 50, size=9).astype(np.int32)
    got = ops.embedding(table, ids, dtype)
    want = F.embedding(torch.from_numpy(ids.astype(np.int64)), wl.to_torch(table, dtype))
    assert np.array_equal(got, wl.from_torch(want))
    bad = np.array([3, -1, 50, 2 ** 40, 49], dtype=np.int64)
    got = ops.embedding(table, bad, dtype)
    assert np.array_equal(got[0], table[3]) and np.array_equal(got[4], table[49])
    assert not got[1:4].any()
