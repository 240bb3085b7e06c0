"""Pins for the oracle's rounding helpers (CPU only)."""
import numpy as np
import pytest
import torch

from oracle import numerics as nm


def _torch_bf16_bits(f32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_rounding_matches_torch_cast_on_float32_inputs():
    # For float32-representable inputs, one RNE step to bf16 is exactly
    # torch's float32 -> bfloat16 conversion (a library special case).
    rng = np.random.Generator(np.random.PCG64(1))
    bits = rng.integers(0, 2**32, size=400_000, dtype=np.uint64).astype(np.uint32)
    f = bits.view(np.float32)
    f = f[np.isfinite(f)]
    # ties: patterns whose low 16 bits are exactly 0x8000, odd and even
    hi = rng.integers(0, 2**16, size=20_000, dtype=np.uint64).astype(np.uint32)
    ties = ((hi << np.uint32(16)) | np.uint32(0x8000)).view(np.float32)
    ties = ties[np.isfinite(ties)]
    specials = np.array([0.0, -0.0, 1e-45, -1e-45, 1.17549435e-38, 3.3895314e38,
                         3.4028235e38, -3.4028235e38, 1.0, -2.0], dtype=np.float32)
    allf = np.concatenate([f, ties, specials])
    got = nm.f64_to_bf16_bits(allf.astype(np.float64))
    want = _torch_bf16_bits(allf)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (allf[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_bf16_rounding_brute_force_nearest():
    # Brute force over every finite bf16 value: the nearest one, ties to the
    # pattern with an even last bit.
    allbits = np.arange(0, 2**16, dtype=np.uint32).astype(np.uint16)
    vals = nm.bf16_bits_to_f64(allbits)
    fin = np.isfinite(vals)
    cand_bits, cand_vals = allbits[fin], vals[fin]
    rng = np.random.Generator(np.random.PCG64(2))
    xs = np.concatenate([rng.uniform(-4, 4, 300), rng.uniform(-1e-38, 1e-38, 100),
                         rng.standard_normal(100) * 1e30])
    got = nm.f64_to_bf16_bits(xs)
    for x, g in zip(xs, got):
        d = np.abs(cand_vals - x)
        m = d.min()
        best = cand_bits[d == m]
        if best.size > 1:
            best = best[(best & 1) == 0]
            if x == 0:
                best = best[:1]
        # +0 and -0 are both nearest to 0; sign follows the input
        gv = nm.bf16_bits_to_f64(np.array([g], np.uint16))[0]
        assert abs(gv - x) == m
        if best.size == 1 and x != 0:
            assert g == best[0], (x, hex(g), hex(best[0]))


def test_bf16_overflow_and_specials():
    big = np.array([3.4e38, 3.3961775e38, 1e39, -1e39, np.inf, -np.inf])
    got = nm.f64_to_bf16_bits(big)
    assert got[0] == 0x7F80 or nm.bf16_bits_to_f64(got[:1])[0] > 3.3e38
    assert got[2] == 0x7F80 and got[3] == 0xFF80
    assert got[4] == 0x7F80 and got[5] == 0xFF80
    assert nm.f64_to_bf16_bits(np.array([np.nan]))[0] & 0x7FC0 == 0x7FC0
    assert nm.f64_to_bf16_bits(np.array([-0.0]))[0] == 0x8000


def test_bf16_upcast_matches_torch():
    allbits = np.arange(0, 2**16, dtype=np.uint32).astype(np.uint16)
    t = torch.from_numpy(allbits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    mine = nm.bf16_bits_to_f64(allbits)
    same = (t == mine) | (np.isnan(t) & np.isnan(mine))
    assert same.all()


def test_f32_rounding_is_ieee():
    x = np.array([1.0 + 2.0**-24, 1.0 + 3 * 2.0**-24, 1.0 + 2.0**-24 + 2.0**-50])
    got = nm.f64_to_f32(x)
    assert got[0] == np.float32(1.0)                    # tie to even
    assert got[1] == np.float32(1.0 + 2.0**-22)        # tie to even (up)
    assert got[2] == np.float32(1.0 + 2.0**-23)        # above the tie


def test_ulp_distance():
    a = np.array([0x3F80, 0x0000, 0x8000, 0x0001, 0x3F80], np.uint16)
    b = np.array([0x3F81, 0x8000, 0x0001, 0x8001, 0xBF80], np.uint16)
    d = nm.bf16_ulp_distance(a, b)
    assert list(d) == [1, 0, 1, 2, 2 * 0x3F80]


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_round_trip_values(dtype):
    rng = np.random.Generator(np.random.PCG64(3))
    x = rng.standard_normal(1000)
    r = nm.round_to(x, dtype)
    assert np.array_equal(nm.round_to(nm.values(r, dtype), dtype), r)


def test_f32_ulp_distance_and_error_stats():
    from tests.parity import error_stats, f32_ulp_distance
    one = np.float32(1.0)
    a = np.array([one, 0.0, -0.0, np.nextafter(np.float32(0), one), one], np.float32)
    b = np.array([np.nextafter(one, np.float32(2)), -0.0, np.nextafter(np.float32(0), one),
                  -np.nextafter(np.float32(0), one), -one], np.float32)
    assert list(f32_ulp_distance(a, b)) == [1, 0, 1, 2, 2 * 0x3F800000]
    got = np.array([1.0, 2.0, 0.0], np.float32)
    want = np.array([np.nextafter(one, np.float32(2)), 2.0, 0.0], np.float32)
    s = error_stats(got, want, nm.F32)
    assert s["n"] == 3 and s["max_ulp"] == 1 and s["exact"] == pytest.approx(2 / 3)
    assert s["max_abs"] == pytest.approx(2.0**-23)
    assert s["max_rel"] == pytest.approx(2.0**-23 / (1 + 2.0**-23))
    sb = error_stats(np.array([0x3F80, 0x4000], np.uint16), np.array([0x3F81, 0x4000], np.uint16),
                     nm.BF16)
    assert sb["max_ulp"] == 1 and sb["exact"] == 0.5 and sb["max_abs"] == 2.0**-7
