"""Randomised calls through the native entry points against the selection
model (CPU, recording backend): every status, selection record, statistic
and launch count must agree, including for malformed arguments.

Complements the systematic call zoo of test_host_cache with random
combinations of sizes, pointer offsets, paddings, epsilons, bases and RoPE
variants (hypothesis, derandomized so every run draws the same calls).
"""
import ctypes as C

import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import (CACHE_ADDR, add_call, chain_call, emb_call, mf_call, qkn_call,
                                   res_call, rn_call, rope_call, silu_call, sw_call)
from tests.test_host_cache import run_both

BF, F = S.DT_BF16, S.DT_F32
SETTINGS = settings(max_examples=300, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@pytest.fixture(scope="module")
def lib():
    return load_fake()


def _guards(lib, h):
    from paper_2609_37241_amd._lib import Stats, VersionInfo
    st_ = Stats()
    lib.tri_spec_stats(h, C.byref(st_))
    out = []
    for i in range(st_.n_versions):
        v = VersionInfo()
        assert lib.tri_spec_version_info(h, i, C.byref(v)) == 0
        out.append((v.b_lo, v.b_hi, v.h_lo, v.h_hi, v.h_mod))
    return out


def _check(lib, calls, flags=0):
    lib.trifake_reset()
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), S.MAX_CAPACITY, flags) == 0
    try:
        m = S.SpecCacheModel(capacity=S.MAX_CAPACITY, flags=flags)
        for c in calls:
            run_both(lib, h, m, c)
        assert _guards(lib, h) == [(g.b_lo, g.b_hi, g.h_lo, g.h_hi, g.h_mod) for g in m.guards]
    finally:
        lib.tri_spec_cache_destroy(h)


dtypes = st.sampled_from([F, F, BF, BF, BF, 7])
tokens = st.sampled_from([-1, 0, 1, 2, 3, 5, 8, 9, 63, 64, 65, 128, 513, 8192, 8193,
                          S.T_MAX, S.T_MAX + 1])
offs = st.sampled_from([0, 0, 0, 1, 2, 4, 8, 16])
pads = st.sampled_from([0, 0, 0, -1, 1, 3, 8, 64])
epss = st.sampled_from([1e-6, 1e-6, 0.0, -1e-6, float("nan"), float("inf"), 1e39, 1e-30])
bases = st.sampled_from([1e4, 5e5, 1e6, 1.0, 0.5, 1.0001, float("nan"), float("inf"), 3e38])
widths = st.sampled_from([0, 1, 2, 7, 8, 64, 100, 256, 520, 688, 1001, 4096, 8192, 11008, 40000,
                          S.H_LIMIT - 1, S.H_LIMIT])
heads = st.sampled_from([0, 1, 2, 3, 4, 8, 32, 64, 4096, 4097, -1])
hds = st.sampled_from([0, 1, 2, 63, 64, 96, 128, 256, 512, 514, 1024])
exts = st.one_of(
    st.none(),
    st.fixed_dictionaries({
        "rotary_dim": st.sampled_from([0, 0, 2, 3, 32, 64, 66, 96, 128, -2]),
        "interleaved": st.sampled_from([0, 1, 2]),
        "pos_int64": st.sampled_from([0, 1, 3]),
    }),
    st.fixed_dictionaries({
        "scaling": st.sampled_from([S.SCALING_LLAMA3, S.SCALING_LLAMA3, 2]),
        "factor": st.sampled_from([8.0, 0.0, -1.0, float("inf")]),
        "low_freq_factor": st.sampled_from([1.0, 0.0, float("nan")]),
        "high_freq_factor": st.sampled_from([4.0, 1.0, 0.5]),
        "original_max_pos": st.sampled_from([8192, 0, -5]),
    }),
    st.fixed_dictionaries({
        "cos_sin": st.sampled_from([CACHE_ADDR, CACHE_ADDR + 2, CACHE_ADDR + 4]),
        "cos_sin_len": st.sampled_from([0, 1, 4096]),
        "interleaved": st.sampled_from([0, 1]),
    }),
)


@st.composite
def norm_calls(draw):
    mk = draw(st.sampled_from([rn_call, res_call]))
    return mk(draw(dtypes), draw(tokens), draw(widths), eps=draw(epss), off=draw(offs),
              pad=draw(pads))


@st.composite
def rope_calls(draw):
    qkn = draw(st.booleans())
    d, T, nq, nk, hd = draw(dtypes), draw(tokens), draw(heads), draw(heads), draw(hds)
    ext = draw(exts)
    if qkn:
        return qkn_call(d, T, nq, nk, hd, base=draw(bases), eps=draw(epss), off=draw(offs),
                        pad=draw(pads), w_off=draw(offs), ext=ext)
    return rope_call(d, T, nq, nk, hd, base=draw(bases), off=draw(offs), pad=draw(pads),
                     pos_off=draw(st.sampled_from([0, 0, 2, 4])), ext=ext)


@st.composite
def short_calls(draw):
    d, T, W = draw(dtypes), draw(tokens), draw(widths)
    kind = draw(st.sampled_from(["sw", "silu", "add", "mf", "emb"]))
    if kind == "sw":
        return sw_call(d, T, W, off=draw(offs), pad=draw(pads))
    if kind == "silu":
        return silu_call(d, T, W, off=draw(offs), pad=draw(pads))
    if kind == "add":
        return add_call(d, T, W, off=draw(offs), b_off=draw(offs), pad=draw(pads))
    if kind == "mf":
        return mf_call(d, T, W, off=draw(offs), m_off=draw(offs), pad=draw(pads),
                       m_pad=draw(pads),
                       value=draw(st.sampled_from([-1e4, float("-inf"), float("nan"), 0.0])))
    return emb_call(d, T, W, draw(st.sampled_from([0, 1, 5, 128256])),
                    ids64=draw(st.sampled_from([0, 1, 2])), off=draw(offs), pad=draw(pads),
                    ids_off=draw(st.sampled_from([0, 0, 2, 4])))


@st.composite
def chain_calls(draw):
    d, T = draw(dtypes), draw(tokens)
    H = draw(st.sampled_from([1, 64, 256, 520, 4096, 8192, 40000]))
    I = draw(st.sampled_from([1, 688, 690, 11008, 14336]))
    nq, nk = draw(st.sampled_from([(4, 4), (32, 32), (32, 8), (8, 1), (4, 0), (64, 8)]))
    hd = draw(st.sampled_from([64, 96, 128, 256]))
    return chain_call(d, T, H, I, nq, nk, hd, base=draw(bases), eps=draw(epss),
                      res_off=draw(offs), res_pad=draw(pads), rope_off=draw(offs),
                      rope_pad=draw(pads), sw_off=draw(offs), sw_pad=draw(pads),
                      qk_norm=draw(st.booleans()), qk_eps=draw(epss), w_off=draw(offs),
                      ext=draw(exts))


@SETTINGS
@given(st.lists(norm_calls(), min_size=1, max_size=6))
def test_random_norm_calls(lib, calls):
    _check(lib, calls)


@SETTINGS
@given(st.lists(rope_calls(), min_size=1, max_size=6))
def test_random_rope_calls(lib, calls):
    _check(lib, calls)


@SETTINGS
@given(st.lists(short_calls(), min_size=1, max_size=6))
def test_random_short_op_calls(lib, calls):
    _check(lib, calls)


@SETTINGS
@given(st.lists(chain_calls(), min_size=1, max_size=4), st.sampled_from([0, 1]))
def test_random_chain_calls(lib, calls, auto):
    _check(lib, calls, flags=S.FLAG_AUTO_INSTALL if auto else 0)


# Generic (range-guarded) versions: longer call lists, so that later calls
# land in the runs and row-length ranges of earlier versions.
GENERIC = S.FLAG_GENERIC | S.FLAG_AUTO_INSTALL


@SETTINGS
@given(st.lists(norm_calls(), min_size=2, max_size=12))
def test_random_norm_calls_generic(lib, calls):
    _check(lib, calls, flags=GENERIC)


@SETTINGS
@given(st.lists(chain_calls(), min_size=2, max_size=8))
def test_random_chain_calls_generic(lib, calls):
    _check(lib, calls, flags=GENERIC)


@SETTINGS
@given(st.lists(st.one_of(rope_calls(), short_calls()), min_size=2, max_size=10))
def test_random_rope_and_short_calls_generic(lib, calls):
    _check(lib, calls, flags=GENERIC)
