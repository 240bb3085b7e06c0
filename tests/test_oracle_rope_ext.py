"""Pins for the oracle's RoPE variants (CPU only): GPT-J pairs, partial
rotary, int64 positions, Llama-3 frequency scaling and a caller's cos/sin
cache. Each is checked against an independent definition (complex rotation,
mpmath, closed forms worked by hand) or against an already pinned op on a
reduced case."""
import math

import mpmath
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ops as O
import workloads as wl

LLAMA31 = dict(factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0, original_max_pos=8192)


def _inputs(dtype, T=5, nq=4, nk=2, hd=64, seed=3, pos_max=5000):
    r = np.random.Generator(np.random.PCG64(seed))
    q = wl.host_array(r, (T, nq, hd), dtype)
    k = wl.host_array(r, (T, nk, hd), dtype)
    pos = r.integers(0, pos_max, size=T).astype(np.int32)
    return q, k, pos


def _close(a, b, dtype):
    if dtype == nm.F32:
        x, y = nm.values(a, dtype), nm.values(b, dtype)
        return np.all(np.abs(x - y) <= 2e-6 * np.abs(y) + 2e-6)
    return np.all(nm.bf16_ulp_distance(a, b) <= 1)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_defaults_equal_the_pinned_ops_bitwise(dtype):
    q, k, pos = _inputs(dtype)
    a = O.rope_ext(q, k, pos, 1e4, dtype)
    b = O.rope_qk(q, k, pos, 1e4, dtype)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    r = np.random.Generator(np.random.PCG64(9))
    qw, kw = wl.host_weight(r, 64, dtype), wl.host_weight(r, 64, dtype)
    a = O.rope_ext(q, k, pos, 1e4, dtype, q_w=qw, k_w=kw)
    b = O.qk_norm_rope(q, k, pos, 1e4, qw, kw, 1e-6, dtype)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_interleaved_pairs_are_complex_rotation_of_adjacent_elements(dtype):
    q, k, pos = _inputs(dtype, hd=32)
    got, _ = O.rope_ext(q, k, pos, 1e4, dtype, interleaved=True)
    v = nm.values(q, dtype)
    z = v[..., 0::2] + 1j * v[..., 1::2]
    inv = np.array([math.pow(1e4, -2.0 * i / 32) for i in range(16)], dtype=np.float32)
    th = (pos.astype(np.float32)[:, None] * inv[None, :]).astype(np.float64)
    z = z * np.exp(1j * th)[:, None, :]
    want = np.empty_like(v)
    want[..., 0::2], want[..., 1::2] = z.real, z.imag
    assert _close(got, nm.round_to(want, dtype), dtype)


@pytest.mark.parametrize("interleaved", [False, True])
@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_partial_rotary_rotates_a_prefix_and_passes_the_rest(dtype, interleaved):
    q, k, pos = _inputs(dtype, hd=128)
    rd = 32
    gq, gk = O.rope_ext(q, k, pos, 1e4, dtype, rotary_dim=rd, interleaved=interleaved)
    # elements past rd are untouched, bit for bit
    assert np.array_equal(gq[..., rd:], q[..., rd:]) and np.array_equal(gk[..., rd:], k[..., rd:])
    # the prefix is the full op on a head of width rd (inverse frequencies over rd)
    wq, wk = O.rope_ext(np.ascontiguousarray(q[..., :rd]), np.ascontiguousarray(k[..., :rd]),
                        pos, 1e4, dtype, interleaved=interleaved)
    assert np.array_equal(gq[..., :rd], wq) and np.array_equal(gk[..., :rd], wk)
    # and for rotate-half that op is the pinned one
    if not interleaved:
        rq, _ = O.rope_qk(np.ascontiguousarray(q[..., :rd]), None, pos, 1e4, dtype)
        assert np.array_equal(wq, rq)


def test_partial_rotary_with_qk_norm_normalises_the_whole_head():
    dtype = nm.F32
    q, k, pos = _inputs(dtype, hd=64)
    r = np.random.Generator(np.random.PCG64(4))
    qw, kw = wl.host_weight(r, 64, dtype), wl.host_weight(r, 64, dtype)
    gq, _ = O.rope_ext(q, k, pos, 1e4, dtype, rotary_dim=16, q_w=qw, k_w=kw)
    n = O.rmsnorm(q, qw, 1e-6, dtype)          # pass-through part: just the norm
    assert np.array_equal(gq[..., 16:], n[..., 16:])


def test_int64_positions_round_to_nearest_float32():
    inv = O.rope_inv_freq(1e4, 8)
    p = np.array([3, 2 ** 24 + 1, 2 ** 40 + 3, 2 ** 40 + 2 ** 16 + 1, -(2 ** 33) - 1],
                 dtype=np.int64)
    th = O.rope_angles(p, inv)
    # nearest float32 of each integer, worked by hand (spacing 2 at 2^24,
    # 2^17 at 2^40, 2^10 at 2^33): ties and near-ties as stated
    p32 = np.array([3.0, 2.0 ** 24, 2.0 ** 40, 2.0 ** 40 + 2 ** 17, -(2.0 ** 33)],
                   dtype=np.float32)
    assert np.array_equal(th, (p32[:, None] * inv[None, :]).astype(np.float64))
    # small positions: int64 and int32 give the same op
    q, k, pos = _inputs(nm.BF16)
    a = O.rope_ext(q, k, pos.astype(np.int64), 5e5, nm.BF16)
    b = O.rope_ext(q, k, pos, 5e5, nm.BF16)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_llama3_table_regimes_for_llama31_shapes():
    # base 5e5, hd 128, factor 8, low 1, high 4, original length 8192. The
    # wavelength 2 pi / inv_i crosses 8192 / 4 = 2048 between i = 28 and 29
    # (i < 64 ln(2048 / 2pi) / ln(5e5) = 28.2) and 8192 between i = 34 and 35
    # (i > 64 ln(8192 / 2pi) / ln(5e5) = 34.98): i <= 28 keep their frequency,
    # i >= 35 are divided by 8, i = 29..34 interpolate.
    t = O.rope_inv_freq_llama3(5e5, 128, **_args(LLAMA31))
    plain = O.rope_inv_freq(5e5, 128)
    assert np.array_equal(t[:29], plain[:29])
    mpmath.mp.dps = 50
    for i in range(35, 64):
        exact = mpmath.power(mpmath.mpf(500000), mpmath.mpf(-2 * i) / 128) / 8
        assert t[i] == _nearest_f32(exact), i
    for i in range(29, 35):
        assert plain[i] / 8 < t[i] < plain[i], i
    assert np.all(np.diff(t[29:35].astype(np.float64) / plain[29:35]) < 0)


def _args(d):
    return dict(factor=d["factor"], low=d["low_freq_factor"], high=d["high_freq_factor"],
                orig=d["original_max_pos"])


def _nearest_f32(x) -> np.float32:
    f = np.float32(float(x))
    best = None
    for c in (np.nextafter(f, np.float32(0)), f, np.nextafter(f, np.float32(np.inf))):
        err = abs(mpmath.mpf(float(c)) - x)
        if best is None or err < best[0]:
            best = (err, c)
    return np.float32(best[1])


def test_llama3_interpolation_is_continuous_at_both_edges():
    from decimal import Decimal
    L, lo, hi, f = 8192, 1.0, 4.0, 8.0
    pi = O._decimal_pi()
    # inverse frequencies whose wavelength sits just inside each edge of the band
    for wl_edge, want in ((Decimal(L) / Decimal(lo), "divided"), (Decimal(L) / Decimal(hi), "kept")):
        for eps in (Decimal("1e-30"), Decimal("-1e-30")):
            inv = 2 * pi / (wl_edge * (1 + eps))
            got = O.llama3_scale(inv, f, lo, hi, L)
            ref = inv / Decimal(f) if want == "divided" else inv
            assert abs(got - ref) / ref < Decimal("1e-25")


def test_decimal_pi():
    mpmath.mp.dps = 70
    assert abs(mpmath.mpf(str(O._decimal_pi())) - mpmath.pi) < mpmath.mpf("1e-55")


@pytest.mark.parametrize("interleaved", [False, True])
def test_cos_sin_cache_matches_computed_angles_and_clamps(interleaved):
    dtype = nm.BF16
    q, k, pos = _inputs(dtype, hd=64, pos_max=100)
    inv = O.rope_inv_freq(1e4, 64)
    th = O.rope_angles(np.arange(128, dtype=np.int32), inv)
    cache = np.concatenate([np.cos(th), np.sin(th)], axis=1).astype(np.float32)
    a = O.rope_ext(q, k, pos, 0.0, dtype, interleaved=interleaved, cos_sin=cache)
    b = O.rope_ext(q, k, pos, 1e4, dtype, interleaved=interleaved)
    assert _close(a[0], b[0], dtype) and _close(a[1], b[1], dtype)
    # positions past the cache use its last row, negative ones its first
    p2 = pos.copy()
    p2[0], p2[1] = 1000, -5
    c = O.rope_ext(q, k, p2, 0.0, dtype, interleaved=interleaved, cos_sin=cache)
    p3 = p2.copy()
    p3[0], p3[1] = 127, 0
    d = O.rope_ext(q, k, p3, 0.0, dtype, interleaved=interleaved, cos_sin=cache)
    assert np.array_equal(c[0], d[0]) and np.array_equal(c[1], d[1])
