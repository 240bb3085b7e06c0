"""Degenerate inputs: zero rows, infinities, NaNs and extreme magnitudes
through every op, against the oracle (NaN where the oracle has NaN, the same
infinities, the usual tolerance elsewhere). Magnitudes stay where a row's or
head's sum of squares is finite in float32, the GPU's accumulation type
(beyond that float32 and the oracle's float64 legitimately differ).

Each case prints its name before touching the GPU. Inputs are built here
from the seeded generators plus planted special values; expected values
only from `oracle`.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
import workloads as wl

# the oracle meets inf - inf and 0 * inf on purpose here
pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::RuntimeWarning")]
DEV = "cuda:0"
INF, NAN = float("inf"), float("nan")


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


@pytest.fixture
def cache(tri):
    c = tri.SpecCache(auto_install=True)
    yield c
    torch.cuda.synchronize()
    c.close()


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def bits(a, dtype):
    """float values -> the host representation of `dtype` (one rounding)."""
    return nm.round_to(np.asarray(a, dtype=np.float64), dtype)


def dev(a, dtype):
    return wl.to_torch(a, dtype, DEV)


def host(t):
    return wl.from_torch(t)


def check_special(name, got, want, dtype):
    g, o = nm.values(got, dtype), nm.values(want, dtype)
    assert g.shape == o.shape
    assert np.array_equal(np.isnan(g), np.isnan(o)), f"{name}: NaN positions differ"
    inf = np.isinf(o)
    assert np.array_equal(g[inf], o[inf]), f"{name}: infinities differ"
    fin = np.isfinite(o)
    assert np.isfinite(g[fin]).all(), f"{name}: non-finite where the oracle is finite"
    if dtype == nm.F32:
        ok = np.abs(g[fin] - o[fin]) <= 1e-5 * np.abs(o[fin]) + 1e-6
    else:
        ok = (np.abs(g[fin] - o[fin]) <= 2e-2) | \
            (nm.bf16_ulp_distance(np.asarray(got)[fin], np.asarray(want)[fin]) <= 1)
    assert ok.all(), f"{name}: {int((~ok).sum())} finite values outside tolerance"


DTYPES = [nm.F32, nm.BF16]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("res", [False, True], ids=["rmsnorm", "residual"])
def test_norm_special_rows(cache, dtype, res):
    print(f"special: norm {dtype} residual={res}", flush=True)
    H = 1024
    r = rng(1)
    x = r.standard_normal((8, H))
    x[0] = 0.0                                  # zero row: zeros (eps > 0)
    x[1, 7] = INF                               # +inf: NaN there, signed zeros elsewhere
    x[2, 9] = -INF
    x[3, 100] = NAN                             # NaN: the whole row NaN
    x[4] = 1e-30                                # tiny row: eps dominates
    x[5, :] = 3.0                               # constant row: w exactly (up to rounding)
    x[6, 5] = 1e4                               # one large element
    rr = np.zeros((8, H)) if res else None
    w = r.uniform(0.5, 1.5, H)
    xb, wb = bits(x, dtype), bits(w, dtype)
    xd, wd = dev(xb, dtype), dev(wb, dtype)
    if res:
        rb = bits(rr, dtype)
        y, ro = cache.residual_rmsnorm(xd, dev(rb, dtype), wd, 1e-6)
        torch.cuda.synchronize()
        wy, wh = O.residual_rmsnorm(xb, rb, wb, 1e-6, dtype)
        check_special("res_out", host(ro), wh, dtype)
    else:
        y = cache.rmsnorm(xd, wd, 1e-6)
        torch.cuda.synchronize()
        wy = O.rmsnorm(xb, wb, 1e-6, dtype)
    check_special("y", host(y), wy, dtype)


@pytest.mark.parametrize("dtype", DTYPES)
def test_norm_zero_row_without_eps_is_nan(cache, dtype):
    print(f"special: norm eps 0 {dtype}", flush=True)
    x = np.zeros((2, 256))
    x[1] = 1.0
    w = np.ones(256)
    xb, wb = bits(x, dtype), bits(w, dtype)
    y = cache.rmsnorm(dev(xb, dtype), dev(wb, dtype), 0.0)
    torch.cuda.synchronize()
    want = O.rmsnorm(xb, wb, 0.0, dtype)
    assert np.isnan(nm.values(want, dtype)[0]).all()
    check_special("y", host(y), want, dtype)


@pytest.mark.parametrize("dtype", DTYPES)
def test_swiglu_special_values(cache, dtype):
    print(f"special: swiglu {dtype}", flush=True)
    g = np.array([INF, -INF, NAN, 1e30, -1e30, 0.0, 0.0, INF, -0.0, 88.0, -88.0, 1.0] * 4,
                 dtype=np.float64)[None, :]
    u = np.array([1.0, 1.0, 1.0, 1.0, 1.0, INF, NAN, 0.0, 5.0, 1.0, 1.0, -INF] * 4,
                 dtype=np.float64)[None, :]
    gb, ub = bits(g, dtype), bits(u, dtype)
    out = cache.swiglu(dev(gb, dtype), dev(ub, dtype))
    torch.cuda.synchronize()
    check_special("out", host(out), O.swiglu(gb, ub, dtype), dtype)


@pytest.mark.parametrize("dtype", DTYPES)
def test_silu_add_masked_fill_special_values(cache, dtype):
    print(f"special: short ops {dtype}", flush=True)
    a = np.array([INF, -INF, NAN, 1e30, -1e30, 0.0, -0.0, 3.0] * 8, dtype=np.float64)[None, :]
    b = np.array([-INF, 1.0, 1.0, 1e30, -1e30, -0.0, -0.0, NAN] * 8, dtype=np.float64)[None, :]
    ab, bb = bits(a, dtype), bits(b, dtype)
    ad, bd = dev(ab, dtype), dev(bb, dtype)
    out = cache.silu(ad)
    torch.cuda.synchronize()
    check_special("silu", host(out), O.silu(ab, dtype), dtype)
    out = cache.add(ad, bd)
    torch.cuda.synchronize()
    check_special("add", host(out), O.add(ab, bb, dtype), dtype)
    mask = (np.arange(a.size) % 3 == 0).astype(np.uint8)[None, :]
    for value in (NAN, INF, -INF, 0.0):
        out = cache.masked_fill(ad, torch.from_numpy(mask).to(DEV), value)
        torch.cuda.synchronize()
        check_special(f"masked_fill {value}", host(out), O.masked_fill(ab, mask, value, dtype),
                      dtype)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("qkn", [False, True], ids=["rope", "qk_norm_rope"])
def test_rope_special_values_and_positions(tri, cache, dtype, qkn):
    print(f"special: rope {dtype} qkn={qkn}", flush=True)
    T, nq, nk, hd = 6, 4, 2, 128
    r = rng(3)
    q = r.standard_normal((T, nq, hd))
    k = r.standard_normal((T, nk, hd))
    q[0, 0, 3] = INF                      # an infinite element at position 0 (cos 1, sin 0)
    q[1, 1, 70] = NAN
    k[2, 0, :] = 0.0                      # a zero head (QK norm: zeros with eps > 0)
    k[3, 1, 5] = 1e18                     # large, square still finite in float32
    # positions: 0, the largest exactly representable in float32, huge, and ordinary ones
    pos = np.array([0, (1 << 24) - 1, 2_000_000_000, 5, 4095, 1], dtype=np.int32)
    qb, kb = bits(q, dtype), bits(k, dtype)
    qd, kd = dev(qb, dtype), dev(kb, dtype)
    pd = torch.from_numpy(pos).to(DEV)
    if qkn:
        w = bits(r.uniform(0.5, 1.5, hd), dtype)
        wk = bits(r.uniform(0.5, 1.5, hd), dtype)
        cache.qk_norm_rope(qd, kd, pd, dev(w, dtype), dev(wk, dtype), 1e6, 1e-6)
        wq, wkk = O.qk_norm_rope(qb, kb, pos, 1e6, w, wk, 1e-6, dtype)
    else:
        cache.rope_qk(qd, kd, pd, 1e6)
        wq, wkk = O.rope_qk(qb, kb, pos, 1e6, dtype)
    torch.cuda.synchronize()
    check_special("q", host(qd), wq, dtype)
    check_special("k", host(kd), wkk, dtype)


def test_embedding_copies_special_rows_bit_for_bit(cache):
    print("special: embedding", flush=True)
    table = np.arange(16 * 64, dtype=np.float64).reshape(16, 64)
    table[3, :8] = [INF, -INF, NAN, -0.0, 1e30, -1e30, 1e-30, 0.0]
    tb = bits(table, nm.BF16)
    ids = np.array([3, 3, -1, 16, 0, 15], dtype=np.int32)
    out = cache.embedding(dev(tb, nm.BF16), torch.from_numpy(ids).to(DEV))
    torch.cuda.synchronize()
    got, want = host(out), O.embedding(tb, ids, nm.BF16)
    assert np.array_equal(got.view(np.uint16), np.asarray(want).view(np.uint16))


@pytest.mark.parametrize("dtype", DTYPES)
def test_silu_negative_tail_keeps_its_value(cache, dtype):
    """Gates from -60 to -104 (past the float32 overflow of exp(-g) at
    -88.7): SwiGLU and silu stay within one bf16 ulp of the oracle, and
    within float32's relative tolerance wherever the oracle's value is a
    normal float32 (an absolute 1e-42 covers the subnormal range)."""
    print(f"special: silu tail {dtype}", flush=True)
    g = -np.linspace(60.0, 104.0, 4096)[None, :]
    u = rng(6).uniform(0.5, 2.0, g.shape)
    gb, ub = bits(g, dtype), bits(u, dtype)
    gd, ud = dev(gb, dtype), dev(ub, dtype)
    for name, got, want in (("swiglu", cache.swiglu(gd, ud), O.swiglu(gb, ub, dtype)),
                            ("silu", cache.silu(gd), O.silu(gb, dtype))):
        torch.cuda.synchronize()
        got = host(got)
        if dtype == nm.BF16:
            assert nm.bf16_ulp_distance(got, want).max() <= 1, name
        else:
            gv, ov = nm.values(got, dtype), nm.values(want, dtype)
            assert (np.abs(gv - ov) <= 1e-5 * np.abs(ov) + 1e-42).all(), name
        gv, ov = nm.values(got, dtype), nm.values(want, dtype)
        assert (gv[np.abs(ov) >= 2.0**-126] != 0).all(), name     # no flush to zero
