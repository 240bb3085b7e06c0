"""The native cache core on the CPU, against the recording launch backend.

Checks the library's guards, ordered dispatch (Algorithm 1, Sec. 3.2), the
miss / install / error paths (Sec. 3.5), argument preparation and the
selection records -- bit for bit against the oracle's selection model.
"""
import collections
import ctypes as C
import math
import struct

import numpy as np
import pytest

from oracle import ops as O
from oracle import selection as S
from tests.native_libs import load_fake
from tests.selection_calls import (CACHE_ADDR, add_call, chain_call, elem_offset, emb_call,
                                   mf_call, qkn_call, res_call, rn_call, rope_call, silu_call,
                                   sw_call)
import workloads as wl

BF, F = S.DT_BF16, S.DT_F32


@pytest.fixture(scope="module")
def lib():
    return load_fake()


@pytest.fixture
def fresh(lib):
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


def c_call(lib, cache, c: S.Call, stream=None):
    from paper_2609_37241_amd._lib import ChainArgs
    p, s = c.ptr, c.stride
    if c.op == S.OP_RMSNORM:
        return lib.tri_rmsnorm(cache, c.dtype, p.get("x"), s["x"], p.get("w"), p.get("y"),
                               s["y"], c.T, c.H, c.eps, stream)
    if c.op == S.OP_RES_RMSNORM:
        return lib.tri_residual_rmsnorm(cache, c.dtype, p.get("x"), s["x"], p.get("res"),
                                        s["res"], p.get("w"), p.get("y"), s["y"],
                                        p.get("res_out"), s["res_out"], c.T, c.H, c.eps, stream)
    if c.op in (S.OP_ROPE_QK, S.OP_QK_NORM_ROPE) and c.ext is not None:
        return lib.tri_rope_qk_ext(cache, c.dtype, p.get("q"), s["q"], p.get("k"), s["k"],
                                   p.get("pos"), c.T, c.nq, c.nk, c.hd, c.base,
                                   C.byref(c_ext(c.ext)), p.get("q_w") if c.op == 6 else None,
                                   p.get("k_w"), c.eps, stream)
    if c.op == S.OP_ROPE_QK:
        return lib.tri_rope_qk(cache, c.dtype, p.get("q"), s["q"], p.get("k"), s["k"],
                               p.get("pos"), c.T, c.nq, c.nk, c.hd, c.base, stream)
    if c.op == S.OP_QK_NORM_ROPE:
        return lib.tri_qk_norm_rope(cache, c.dtype, p.get("q"), s["q"], p.get("k"), s["k"],
                                    p.get("pos"), c.T, c.nq, c.nk, c.hd, c.base, p.get("q_w"),
                                    p.get("k_w"), c.eps, stream)
    if c.op == S.OP_SILU:
        return lib.tri_silu(cache, c.dtype, p.get("a"), s["a"], p.get("out"), s["out"], c.T,
                            c.H, stream)
    if c.op == S.OP_ADD:
        return lib.tri_add(cache, c.dtype, p.get("a"), s["a"], p.get("b"), s["b"], p.get("out"),
                           s["out"], c.T, c.H, stream)
    if c.op == S.OP_MASKED_FILL:
        return lib.tri_masked_fill(cache, c.dtype, p.get("a"), s["a"], p.get("b"), s["b"],
                                   c.value, p.get("out"), s["out"], c.T, c.H, stream)
    if c.op == S.OP_EMBEDDING:
        return lib.tri_embedding(cache, c.dtype, p.get("table"), s["table"], c.n_rows,
                                 p.get("ids"), c.ids64, p.get("out"), s["out"], c.T, c.H, stream)
    if c.op == S.OP_SWIGLU:
        return lib.tri_swiglu(cache, c.dtype, p.get("gate"), s["gate"], p.get("up"), s["up"],
                              p.get("out"), s["out"], c.T, c.I, stream)
    a = ChainArgs()
    a.dtype, a.nq, a.nk, a.hd = c.dtype, c.nq, c.nk, c.hd
    a.T, a.H, a.I, a.eps, a.base = c.T, c.H, c.I, c.eps, c.base
    a.x, a.x_rs = p.get("x"), s["x"]
    a.res, a.res_rs = p.get("res"), s["res"]
    a.w = p.get("w")
    a.y, a.y_rs = p.get("y"), s["y"]
    a.res_out, a.ro_rs = p.get("res_out"), s["res_out"]
    a.q, a.q_ts = p.get("q"), s["q"]
    a.k, a.k_ts = p.get("k"), s["k"]
    a.pos = p.get("pos")
    a.gate, a.g_rs = p.get("gate"), s["gate"]
    a.up, a.u_rs = p.get("up"), s["up"]
    a.out, a.o_rs = p.get("out"), s["out"]
    a.q_norm_w, a.k_norm_w, a.qk_eps = p.get("q_w"), p.get("k_w"), c.qk_eps
    if c.ext is not None:
        x = c_ext(c.ext)
        a.rope_ext = C.pointer(x)
    return lib.tri_decode_chain(cache, C.byref(a), stream)


def c_ext(ext):
    from paper_2609_37241_amd._lib import RopeExt
    x = RopeExt()
    full = dict(S.PLAIN_EXT)
    full.update(ext)
    for n, _ in RopeExt._fields_:
        setattr(x, n, full[n] if full[n] is not None else 0)
    return x


def c_record(lib, cache):
    from paper_2609_37241_amd._lib import Selection
    sel = Selection()
    assert lib.tri_spec_last_selection(cache, C.byref(sel)) == 0
    return sel.as_tuple()


def c_stats(lib, cache):
    from paper_2609_37241_amd._lib import Stats
    st = Stats()
    lib.tri_spec_stats(cache, C.byref(st))
    return (st.calls, st.hits, st.misses, st.errors, st.empty, st.installs, st.n_versions)


def m_stats(m):
    s = m.stats
    return (s.calls, s.hits, s.misses, s.errors, s.empty, s.installs, len(m.versions))


def c_install(lib, cache):
    from paper_2609_37241_amd._lib import Selection
    sel = Selection()
    st = lib.tri_spec_install_last_miss(cache, C.byref(sel))
    return st, (sel.as_tuple() if st == 0 else None)


def run_both(lib, cache, m, c, install=True):
    """Call both sides (installing on a miss) and compare every observable."""
    st_c = c_call(lib, cache, c)
    st_m = m.call(c)
    assert st_c == st_m, (c, st_c, st_m)
    assert c_record(lib, cache) == m.last.as_tuple(), c
    if st_c == S.MISS and install:
        ic, rc = c_install(lib, cache)
        im, rm = m.install_last_miss()
        assert ic == im
        if ic == 0:
            assert rc == rm.as_tuple()
            st_c = c_call(lib, cache, c)
            st_m = m.call(c)
            assert st_c == st_m == S.OK
            assert c_record(lib, cache) == m.last.as_tuple()
    assert c_stats(lib, cache) == m_stats(m)
    assert lib.trifake_launch_count() == m.launch_count
    return st_c


LLAMA3 = dict(scaling=S.SCALING_LLAMA3, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0,
              original_max_pos=8192)
ROPE_EXTS = [dict(rotary_dim=64), dict(rotary_dim=32), dict(rotary_dim=96), dict(interleaved=1),
             dict(interleaved=1, rotary_dim=64), dict(pos_int64=1), LLAMA3,
             dict(LLAMA3, rotary_dim=64, interleaved=1, pos_int64=1),
             dict(cos_sin=CACHE_ADDR, cos_sin_len=4096),
             dict(cos_sin=CACHE_ADDR, cos_sin_len=1, interleaved=1, pos_int64=1),
             dict(rotary_dim=0, interleaved=0, pos_int64=0, scaling=0)]


def call_zoo():
    """Calls over every op, dtype, size class, layout and error kind."""
    calls = []
    for d in (F, BF):
        off = elem_offset(d)
        for T in (0, 1, 2, 3, 4, 5, 8, 9, 64, 65, 512, 8192):
            for H in (64, 256, 520, 4096, 8192, 16384, 40000, 100):
                calls.append(rn_call(d, T, H))
                calls.append(res_call(d, T, H))
            calls.append(rn_call(d, T, 4096, off=off))
            calls.append(res_call(d, T, 4096, pad=64))
            for nq, nk, hd in ((4, 4, 64), (32, 32, 128), (32, 8, 128), (64, 8, 128),
                               (4, 0, 64), (2, 2, 96), (1, 1, 2), (8, 8, 512)):
                calls.append(rope_call(d, T, nq, nk, hd))
            calls.append(rope_call(d, T, 32, 8, 128, base=500000.0, off=off))
            calls.append(rope_call(d, T, 32, 8, 128, pad=64))
            for nq, nk, hd in ((32, 8, 128), (4, 0, 64), (2, 2, 96), (8, 8, 512), (1, 1, 2)):
                calls.append(qkn_call(d, T, nq, nk, hd, base=1e6))
            calls.append(qkn_call(d, T, 32, 8, 128, w_off=off))
            calls.append(qkn_call(d, T, 32, 8, 128, off=off))
            calls.append(qkn_call(d, T, 32, 8, 128, pad=64))
            for ext in ROPE_EXTS:
                calls.append(rope_call(d, T, 32, 8, 128, base=5e5, ext=ext))
                calls.append(qkn_call(d, T, 8, 2, 64, base=5e5, ext=ext))
            calls.append(rope_call(d, T, 4, 4, 64, off=off, ext=dict(interleaved=1)))
            calls.append(rope_call(d, T, 4, 4, 96, ext=dict(rotary_dim=32, interleaved=1)))
            calls.append(rope_call(d, T, 4, 4, 2, ext=dict(interleaved=1)))
            calls.append(rope_call(d, T, 2, 2, 512, ext=dict(interleaved=1)))
            calls.append(qkn_call(d, T, 2, 2, 512, ext=dict(interleaved=1)))
            for I in (688, 11008, 14336, 28672, 11003, 1):
                calls.append(sw_call(d, T, I))
            calls.append(sw_call(d, T, 11008, off=off))
            calls.append(sw_call(d, T, 11008, pad=64))
            calls.append(sw_call(d, T, 11003, pad=1))
            calls.append(chain_call(d, T, 4096, 11008, 32, 32, 128))
            for W in (4096, 11008, 1001, 8, 1):
                calls.append(silu_call(d, T, W))
                calls.append(add_call(d, T, W))
                calls.append(mf_call(d, T, W))
                calls.append(emb_call(d, T, W, 32000))
            calls.append(silu_call(d, T, 4096, pad=64))
            calls.append(add_call(d, T, 4096, b_off=off))
            calls.append(add_call(d, T, 4096, off=off))
            calls.append(mf_call(d, T, 4096, m_off=4))
            calls.append(mf_call(d, T, 4096, m_off=8, m_pad=8))
            calls.append(mf_call(d, T, 4096, m_pad=3))
            calls.append(emb_call(d, T, 4096, 128256, ids64=1))
            calls.append(emb_call(d, T, 4096, 5, pad=64))
            calls.append(emb_call(d, T, 4096, 5, off=off))
            calls.append(chain_call(d, T, 8192, 28672, 64, 8, 128, base=500000.0))
            calls.append(chain_call(d, T, 256, 688, 4, 4, 64))
            calls.append(chain_call(d, T, 4096, 14336, 32, 8, 128, sw_pad=64))
            calls.append(chain_call(d, T, 4096, 14336, 32, 8, 128, rope_off=off))
            calls.append(chain_call(d, T, 40000, 11008, 32, 32, 128))
            calls.append(chain_call(d, T, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True))
            calls.append(chain_call(d, T, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True,
                                    w_off=off))
            calls.append(chain_call(d, T, 256, 688, 4, 0, 64, qk_norm=True))
            for ext in ROPE_EXTS[::2]:
                calls.append(chain_call(d, T, 4096, 14336, 32, 8, 128, base=5e5, ext=ext))
                calls.append(chain_call(d, T, 4096, 12288, 32, 8, 128, base=1e6, ext=ext,
                                        qk_norm=True))
    # errors
    calls += [rn_call(BF, 1, 4096, null=("x",)), rn_call(BF, -1, 4096), rn_call(BF, 1, 0),
              rn_call(BF, 1, 4096, eps=float("nan")), rn_call(BF, 1, 4096, eps=-1.0),
              rn_call(BF, 1, 4096, eps=float("inf")), rn_call(BF, 1, 4096, eps=1e39),
              rn_call(BF, 1, 4096, off=1), rn_call(7, 1, 4096), rn_call(BF, S.T_MAX + 1, 64),
              rn_call(BF, S.T_MAX, 64), rn_call(BF, 1, S.H_LIMIT), rn_call(BF, 1, S.H_LIMIT - 1),
              res_call(BF, 2, 4096, null=("res_out",)), res_call(F, 2, 64, pad=-1),
              rope_call(BF, 1, 4, 4, 63), rope_call(BF, 1, 4, 4, 0), rope_call(BF, 1, 4, 4, 1024),
              rope_call(BF, 1, 4, 4, 64, base=1.0), rope_call(BF, 1, 4, 4, 64, base=float("nan")),
              rope_call(BF, 1, 4, 4, 64, pos_off=2), rope_call(BF, 1, 0, 4, 64),
              rope_call(BF, 1, 4, -1, 64), rope_call(BF, 1, 5000, 4, 64),
              rope_call(BF, 1, 4, 4, 64, null=("k",)), rope_call(BF, 1, 4, 0, 64, null=("k",)),
              rope_call(BF, 1, 4, 4, 64, null=("pos",)), rope_call(BF, 1, 4, 4, 64, off=1),
              rope_call(BF, 1, 4, 4, 64, pad=-1),
              qkn_call(BF, 1, 4, 4, 64, null=("q_w",)), qkn_call(BF, 1, 4, 4, 64, null=("k_w",)),
              qkn_call(BF, 1, 4, 0, 64, null=("k_w", "k")), qkn_call(BF, 1, 4, 4, 64, w_off=1),
              qkn_call(BF, 1, 4, 4, 64, eps=float("nan")), qkn_call(BF, 1, 4, 4, 64, eps=-1.0),
              qkn_call(BF, 1, 4, 4, 63, null=("q_w",)), qkn_call(BF, 1, 4, 4, 64, base=0.5),
              chain_call(BF, 1, 4096, 12288, 32, 8, 128, qk_norm=True, null=("k_w",)),
              chain_call(BF, 1, 4096, 12288, 32, 8, 128, qk_norm=True, qk_eps=float("inf")),
              chain_call(BF, 1, 4096, 12288, 32, 8, 128, qk_norm=True, w_off=1),
              chain_call(BF, 1, 4096, 12288, 32, 8, 128, qk_eps=float("nan")),
              rope_call(BF, 1, 4, 4, 64, ext=dict(rotary_dim=3)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(rotary_dim=66)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(rotary_dim=-2)),
              rope_call(BF, 1, 4, 4, 1024, ext=dict(rotary_dim=3)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(interleaved=2)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(pos_int64=3)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(scaling=2)),
              rope_call(BF, 1, 4, 4, 64, pos_off=4, ext=dict(pos_int64=1)),
              rope_call(BF, 1, 4, 4, 64, pos_off=4),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR + 2, cos_sin_len=8)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=0)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=8,
                                                  **LLAMA3)),
              rope_call(BF, 1, 4, 4, 64, base=1.0, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=8)),
              rope_call(BF, 1, 4, 4, 64, base=float("nan"),
                        ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=8)),
              rope_call(BF, 1, 4, 4, 64, base=1.0, ext=LLAMA3),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, factor=0.0)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, factor=float("inf"))),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, low_freq_factor=-1.0)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, high_freq_factor=1.0)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, high_freq_factor=float("nan"))),
              rope_call(BF, 1, 4, 4, 64, ext=dict(LLAMA3, original_max_pos=0)),
              qkn_call(BF, 1, 4, 4, 64, ext=dict(rotary_dim=80)),
              qkn_call(BF, 1, 4, 4, 64, null=("k_w",), ext=dict(interleaved=1)),
              chain_call(BF, 1, 4096, 11008, 32, 32, 128, ext=dict(rotary_dim=130)),
              chain_call(BF, 1, 4096, 11008, 32, 32, 128, ext=dict(LLAMA3, factor=-8.0)),
              silu_call(BF, 1, 0), silu_call(BF, 1, S.I_LIMIT), silu_call(BF, 1, 64, null=("a",)),
              silu_call(BF, 1, 64, off=1), silu_call(BF, 3, 64, pad=-1),
              add_call(BF, 1, 64, null=("b",)), add_call(BF, 1, 64, b_off=1),
              add_call(F, 1, 64, null=("out",)), add_call(F, 2, 64, pad=-1),
              mf_call(BF, 1, 64, null=("b",)), mf_call(BF, 1, 64, m_off=1),
              mf_call(BF, 2, 64, m_pad=-1), mf_call(BF, 1, 64, off=1),
              mf_call(F, 1, 64, value=float("nan")), mf_call(F, 1, 64, value=float("inf")),
              emb_call(BF, 1, 0, 10), emb_call(BF, 1, 64, 0), emb_call(BF, 1, 64, 10, ids64=2),
              emb_call(BF, 1, S.I_LIMIT, 10), emb_call(BF, 1, 64, 10, null=("ids",)),
              emb_call(BF, 1, 64, 10, ids_off=2), emb_call(BF, 1, 64, 10, ids64=1, ids_off=4),
              emb_call(BF, 1, 64, 10, off=1), emb_call(BF, 2, 64, 10, pad=-1),
              emb_call(F, 0, 64, 0),
              sw_call(BF, 1, 0), sw_call(BF, 1, S.I_LIMIT), sw_call(BF, 1, 64, null=("up",)),
              sw_call(BF, 1, 64, off=1), sw_call(BF, 3, 64, pad=-1)]
    # operand extents: rows spanning exactly 2^47 bytes pass, one element
    # more (or any stride that would wrap the kernels' offsets) is INVALID;
    # with one row the stride is never used
    span = 2 ** 46                                  # bf16 elements in 2^47 bytes
    calls += [rn_call(BF, 2, 4096, pad=span - 8192), rn_call(BF, 2, 4096, pad=span - 8191),
              rn_call(F, 3, 64, pad=2 ** 60), rn_call(BF, 1, 4096, pad=2 ** 62),
              res_call(BF, 2, 4096, pad=2 ** 50), res_call(BF, 9, 1024, pad=2 ** 43),
              rope_call(BF, 2, 4, 4, 64, pad=2 ** 50), rope_call(BF, 1, 4, 4, 64, pad=2 ** 62),
              rope_call(BF, 2, 4, 4, 64, pad=span - 512), rope_call(BF, 2, 4, 4, 64,
                                                                    pad=span - 511),
              qkn_call(BF, 3, 4, 4, 64, pad=2 ** 61),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=2 ** 39)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=2 ** 39 + 1)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=2 ** 62)),
              rope_call(BF, 1, 4, 4, 64, ext=dict(rotary_dim=32, cos_sin=CACHE_ADDR,
                                                  cos_sin_len=2 ** 40)),
              sw_call(BF, 2, 64, pad=2 ** 50), sw_call(F, 2, 64, pad=2 ** 45 - 128),
              sw_call(F, 2, 64, pad=2 ** 45 - 127),
              silu_call(BF, 2, 64, pad=2 ** 50), add_call(BF, 2, 64, pad=2 ** 50),
              mf_call(BF, 2, 64, m_pad=2 ** 47 - 128), mf_call(BF, 2, 64, m_pad=2 ** 47 - 127),
              emb_call(BF, 1, 64, 2 ** 40), emb_call(BF, 1, 64, 2 ** 40 + 1),
              emb_call(BF, 2, 64, 10, pad=2 ** 50),
              chain_call(BF, 2, 4096, 11008, 32, 32, 128, sw_pad=2 ** 50),
              chain_call(BF, 2, 4096, 11008, 32, 32, 128, res_pad=2 ** 50),
              chain_call(BF, 2, 4096, 11008, 32, 32, 128, rope_pad=2 ** 50)]
    return calls


def test_selection_parity_over_call_zoo(lib, fresh):
    cache = fresh(capacity=4096)
    m = S.SpecCacheModel(capacity=4096)
    for c in call_zoo():
        run_both(lib, cache, m, c)
    # second pass: everything installed now hits (or errors) identically
    for c in call_zoo():
        st = run_both(lib, cache, m, c)
        assert st != S.MISS


def test_selection_parity_mixed_stream(lib, fresh):
    # The full mixed-shape stream: 10,000 chain calls with token counts from
    # 1..512, 90 % bf16, 5 % unaligned or padded layouts.
    cache = fresh()
    m = S.SpecCacheModel()
    for T, dt, layout in wl.mixed_stream():
        d = BF if dt == wl.BF16 else F
        off = elem_offset(d) if layout == wl.LAYOUT_UNALIGNED else 0
        pad = wl.MIXED_PAD if layout == wl.LAYOUT_STRIDED else 0
        c = chain_call(d, T, wl.MIXED_H, wl.MIXED_I, wl.MIXED_NQ, wl.MIXED_NK, wl.MIXED_HD,
                       res_off=off, rope_off=off, sw_off=off, res_pad=pad, rope_pad=pad,
                       sw_pad=pad)
        run_both(lib, cache, m, c)
    # one miss per distinct key: 9 token buckets x 2 dtypes x 3 layouts at most
    assert m.stats.misses == len(m.versions) <= 54
    assert m.stats.hits == wl.MIXED_CALLS


def test_auto_install_parity(lib, fresh):
    cache = fresh(flags=1)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL)
    for c in call_zoo()[:400]:
        run_both(lib, cache, m, c, install=False)


def test_capacity_full(lib, fresh):
    cache = fresh(capacity=2)
    m = S.SpecCacheModel(capacity=2)
    for T in (1, 2, 4, 8):
        run_both(lib, cache, m, sw_call(BF, T, 128))
    assert c_install(lib, cache)[0] == S.E_FULL
    cache2 = fresh(capacity=1, flags=1)
    m2 = S.SpecCacheModel(capacity=1, flags=S.FLAG_AUTO_INSTALL)
    for T in (1, 2):
        run_both(lib, cache2, m2, sw_call(BF, T, 128), install=False)
    assert c_record(lib, cache2)[1] == S.E_FULL


@pytest.mark.parametrize("fail_at", [0, 1, 2])
def test_launch_failure_stops_dispatch(lib, fresh, fail_at):
    cache = fresh()
    m = S.SpecCacheModel()
    c = chain_call(BF, 4, 4096, 11008, 32, 32, 128, sw_pad=64)    # three launches
    run_both(lib, cache, m, c)
    base = lib.trifake_launch_count()
    lib.trifake_fail_at(base + fail_at)
    m.launch_fails = {base + fail_at}
    assert run_both(lib, cache, m, c) == S.E_LAUNCH
    assert lib.trifake_launch_count() == base + fail_at + 1
    # the version is kept and the next call hits
    lib.trifake_fail_at(-1)
    m.launch_fails = set()
    assert run_both(lib, cache, m, c) == S.OK


def test_install_needs_a_miss_and_is_idempotent(lib, fresh):
    cache = fresh()
    assert c_install(lib, cache)[0] == S.E_INVALID
    c = rope_call(BF, 1, 32, 32, 128)
    assert c_call(lib, cache, c) == S.MISS
    assert c_call(lib, cache, c) == S.MISS
    assert c_install(lib, cache)[0] == 0
    assert c_install(lib, cache)[0] == 0
    assert c_stats(lib, cache)[-1] == 1
    assert lib.trifake_upload_count() == 1


def test_create_errors(lib):
    h = C.c_void_p()
    assert lib.tri_spec_cache_create(C.byref(h), 4097, 0) == S.E_INVALID
    assert lib.tri_spec_cache_create(C.byref(h), 0, 32) == S.E_INVALID
    assert lib.tri_spec_cache_create(C.byref(h), 0, 3) == S.OK      # auto-install + JIT
    lib.tri_spec_cache_destroy(h)
    assert lib.tri_spec_cache_create(None, 0, 0) == S.E_INVALID
    lib.trifake_init_status(S.E_RUNTIME)
    assert lib.tri_spec_cache_create(C.byref(h), 0, 0) == S.E_RUNTIME
    lib.trifake_reset()
    assert lib.tri_rmsnorm(None, 1, 1, 1, 1, 1, 1, 1, 1, 1e-6, None) == S.E_INVALID
    assert lib.tri_decode_chain(None, None, None) == S.E_INVALID


def test_chain_null_args(lib, fresh):
    cache = fresh()
    assert lib.tri_decode_chain(cache, None, None) == S.E_INVALID
    assert c_stats(lib, cache)[3] == 1


def test_status_strings(lib):
    assert lib.tri_status_str(1) == b"TRI_MISS"
    assert lib.tri_status_str(-5) == b"TRI_E_LAUNCH"
    assert lib.tri_status_str(42) == b"TRI_UNKNOWN"


# ---- several chains per entry call ------------------------------------------------------
def c_layers(lib, cache, calls, stream=None):
    from paper_2609_37241_amd._lib import ChainArgs
    arr = (ChainArgs * max(1, len(calls)))()
    keep = []
    for i, c in enumerate(calls):
        a = _chain_struct(c, keep)
        arr[i] = a
    return lib.tri_decode_chain_layers(cache, arr, len(calls), stream)


def _chain_struct(c, keep):
    from paper_2609_37241_amd._lib import ChainArgs
    p, s = c.ptr, c.stride
    a = ChainArgs()
    a.dtype, a.nq, a.nk, a.hd = c.dtype, c.nq, c.nk, c.hd
    a.T, a.H, a.I, a.eps, a.base = c.T, c.H, c.I, c.eps, c.base
    a.x, a.x_rs = p.get("x"), s["x"]
    a.res, a.res_rs = p.get("res"), s["res"]
    a.w = p.get("w")
    a.y, a.y_rs = p.get("y"), s["y"]
    a.res_out, a.ro_rs = p.get("res_out"), s["res_out"]
    a.q, a.q_ts = p.get("q"), s["q"]
    a.k, a.k_ts = p.get("k"), s["k"]
    a.pos = p.get("pos")
    a.gate, a.g_rs = p.get("gate"), s["gate"]
    a.up, a.u_rs = p.get("up"), s["up"]
    a.out, a.o_rs = p.get("out"), s["out"]
    a.q_norm_w, a.k_norm_w, a.qk_eps = p.get("q_w"), p.get("k_w"), c.qk_eps
    if c.ext is not None:
        x = c_ext(c.ext)
        keep.append(x)
        a.rope_ext = C.pointer(x)
    return a


def run_layers_both(lib, cache, m, calls):
    st_c = c_layers(lib, cache, calls)
    st_m = m.call_layers(calls)
    assert st_c == st_m, (st_c, st_m)
    assert c_record(lib, cache) == m.last.as_tuple()
    assert c_stats(lib, cache) == m_stats(m)
    assert lib.trifake_launch_count() == m.launch_count
    return st_c


def _layer_lists():
    g = lambda T, **kw: chain_call(BF, T, 4096, 14336, 32, 8, 128, base=5e5, **kw)
    off = elem_offset(BF)
    return [
        [g(1)] * 32,                                           # one version, 32 layers
        [g(1), g(8), g(1, rope_off=off), g(0), g(3)],          # fused + three-launch layers
        [g(0), g(0)],                                          # all empty
        [],                                                    # no layers
        [g(1), g(-1), g(1)],                                   # invalid layer: nothing runs
        [g(1), chain_call(BF, 1, 4096, 14336, 32, 8, 127)],    # invalid head_dim
        [g(1, qk_norm=True), g(1, ext=dict(interleaved=1)), g(2, qk_norm=True)],
        [chain_call(F, 5, 256, 688, 4, 4, 64), g(1), chain_call(F, 5, 256, 688, 4, 4, 64)],
    ]


@pytest.mark.parametrize("auto", [0, 1, S.FLAG_GENERIC, S.FLAG_GENERIC | 1],
                         ids=["exact", "exact-auto", "generic", "generic-auto"])
def test_layers_parity_with_model(lib, fresh, auto):
    cache = fresh(flags=auto)
    m = S.SpecCacheModel(flags=auto)
    for calls in _layer_lists() * 2:
        st = run_layers_both(lib, cache, m, calls)
        if st == S.MISS:
            while st == S.MISS:        # install the recorded miss, retry the whole list
                ic, rc = c_install(lib, cache)
                im, rm = m.install_last_miss()
                assert ic == im == 0 and rc == rm.as_tuple()
                st = run_layers_both(lib, cache, m, calls)
    from paper_2609_37241_amd._lib import VersionInfo
    got = []
    for i in range(len(m.versions)):
        v = VersionInfo()
        assert lib.tri_spec_version_info(cache, i, C.byref(v)) == 0
        got.append((v.b_lo, v.b_hi, v.h_lo, v.h_hi, v.h_mod))
    assert got == [(g.b_lo, g.b_hi, g.h_lo, g.h_hi, g.h_mod) for g in m.guards]
    if auto & S.FLAG_GENERIC:
        assert any(g.b_lo >= 0 for g in m.guards)


@pytest.mark.parametrize("fail_at", [0, 1, 5, 9])
def test_layers_launch_failure_stops_and_counts_once(lib, fresh, fail_at):
    cache = fresh(flags=1)
    m = S.SpecCacheModel(flags=1)
    off = elem_offset(BF)
    calls = [chain_call(BF, 2, 4096, 14336, 32, 8, 128, rope_off=off * (i % 2)) for i in range(6)]
    run_layers_both(lib, cache, m, calls)          # installs both versions
    lib.trifake_fail_at(lib.trifake_launch_count() + fail_at)
    m.launch_fails = {m.launch_count + fail_at}
    assert run_layers_both(lib, cache, m, calls) == S.E_LAUNCH


def test_layers_limit(lib, fresh):
    cache = fresh(flags=1)
    m = S.SpecCacheModel(flags=1)
    c = chain_call(BF, 1, 256, 688, 4, 4, 64)
    assert run_layers_both(lib, cache, m, [c] * S.MAX_LAYERS) == S.OK
    assert run_layers_both(lib, cache, m, [c] * (S.MAX_LAYERS + 1)) == S.E_INVALID
    assert lib.tri_decode_chain_layers(cache, None, 2, None) == S.E_INVALID


def test_graph_build_records_the_layer_launches_once(lib, fresh):
    cache = fresh(flags=1)
    m = S.SpecCacheModel(flags=1)
    off = elem_offset(BF)
    calls = [chain_call(BF, 1, 4096, 14336, 32, 8, 128, rope_off=off * (i == 2)) for i in range(4)]
    keep = []
    from paper_2609_37241_amd._lib import ChainArgs
    arr = (ChainArgs * 4)(*[_chain_struct(c, keep) for c in calls])
    g = C.c_void_p()
    n0 = lib.trifake_launch_count()
    assert lib.tri_graph_build_layers(cache, arr, 4, C.byref(g)) == 0
    # the model: the same one entry call
    assert m.call_layers(calls) == S.OK
    assert c_record(lib, cache) == m.last.as_tuple()
    assert c_stats(lib, cache) == m_stats(m)
    # fused, fused, three launches, fused; all on the capture stream
    assert lib.tri_graph_launch_count(g) == 6 == lib.trifake_launch_count() - n0
    streams = {_launch_at(lib, i)[5] for i in range(n0, n0 + 6)}
    assert len(streams) == 1 and streams.pop() >= 0xCA000000
    for _ in range(3):
        assert lib.tri_graph_launch(g, None) == 0
    assert lib.trifake_graph_launches() == 3
    assert lib.trifake_launch_count() - n0 == 6          # replays launch nothing new
    assert c_stats(lib, cache) == m_stats(m)              # nor touch the statistics
    lib.tri_graph_destroy(g)
    assert lib.trifake_graph_destroys() == 1


def test_graph_build_miss_and_errors_make_no_graph(lib, fresh):
    cache = fresh()
    calls = [chain_call(BF, 1, 256, 688, 4, 4, 64)]
    keep = []
    from paper_2609_37241_amd._lib import ChainArgs
    arr = (ChainArgs * 1)(*[_chain_struct(c, keep) for c in calls])
    g = C.c_void_p(123)
    assert lib.tri_graph_build_layers(cache, arr, 1, C.byref(g)) == S.MISS and not g.value
    bad = (ChainArgs * 1)(*[_chain_struct(chain_call(BF, 1, 256, 688, 4, 4, 63), keep)])
    assert lib.tri_graph_build_layers(cache, bad, 1, C.byref(g)) == S.E_INVALID and not g.value
    assert lib.tri_graph_build_layers(cache, arr, 1, None) == S.E_INVALID
    lib.trifake_capture_fail(1)
    c_install(lib, cache)
    assert lib.tri_graph_build_layers(cache, arr, 1, C.byref(g)) == S.E_RUNTIME and not g.value
    assert lib.tri_graph_launch(None, None) == S.E_INVALID


def _launch_at(lib, i, nbytes=16):
    kv, dt, sub = C.c_int32(), C.c_int32(), C.c_int32()
    grid, block = C.c_uint32(), C.c_uint32()
    stream = C.c_void_p()
    buf = C.create_string_buffer(nbytes)
    lib.trifake_get(i, C.byref(kv), C.byref(dt), C.byref(sub), C.byref(grid), C.byref(block),
                    C.byref(stream), buf, nbytes)
    return kv.value, dt.value, sub.value, grid.value, block.value, stream.value or 0


# ---- runtime-compiled specializations and key import / export ------------------------------
def test_jit_cache_makes_the_same_selections(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    m = S.SpecCacheModel(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    for c in call_zoo():
        run_both(lib, cache, m, c)
    # one compiled kernel per launch of every installed version
    n_launch = sum(len(S.plan(k, 1)[2]) for k in m.versions)
    assert lib.trifake_jit_count() == n_launch


def jit_sources(lib):
    out = []
    for i in range(lib.trifake_jit_count()):
        n = lib.trifake_jit_source(i, None, 0)
        buf = C.create_string_buffer(n + 1)
        lib.trifake_jit_source(i, buf, n + 1)
        out.append(buf.raw[:n].decode())
    return out


def _kernel_part(src):
    return src[src.rindex('extern "C"'):]


def test_jit_source_fixes_the_key_shape(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    # fused: RN_BLOCK_2 norm role, QK-norm GPT-J RoPE role, cached SwiGLU;
    # mode = GPT-J pairs | 3 workgroups per token (40 heads x 16 lanes / 256) << 8
    c = chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True,
                   ext=dict(interleaved=1))
    assert S.plan(S.make_key(c), 1)[0] == S.CH_FUSED
    assert c_call(lib, cache, c) == 0
    (src,) = jit_sources(lib)
    k = _kernel_part(src)
    assert "tri_jit_kernel(tri::ChainArgs a)" in k
    for frag in ("a.rn.H = 4096;", "a.rope.hd = 128;", "a.rope.rd = 128;", "a.rope.nq = 32;",
                 "a.rope.nk = 8;", "a.rope.mode = 769u;", "a.sw.I = 12288;",
                 "body_chain<1, false, 2, false, true, true>(a, gridDim.x)"):
        assert frag in k, frag
    assert src.startswith("// Kernel argument blocks")     # the embedded prelude
    assert "#include <hip/" not in src and '#include "../kernargs.h"' not in src
    # three launches (partial rotary with the QK norm takes the scalar role):
    # one specialization per role kernel, each with its own fields fixed
    c = chain_call(F, 2, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True,
                   ext=dict(rotary_dim=64, pos_int64=1))
    assert c_call(lib, cache, c) == 0
    rn, rope, sw = (_kernel_part(x) for x in jit_sources(lib)[1:])
    assert "tri::RnArgs a" in rn and "a.H = 4096;" in rn and "body_rn_block<0, 4, true>" in rn
    assert ("a.rd = 64;" in rope and "a.mode = 2u;" in rope
            and "body_rope_scalar<0, true>" in rope)
    assert "a.I = 12288;" in sw and "body_sw_flat<0, 1, false>" in sw


def test_code_directory_shares_compiled_objects(lib, fresh, tmp_path):
    from paper_2609_37241_amd._lib import VersionInfo
    calls = [chain_call(BF, 1, 4096, 11008, 32, 32, 128),
             chain_call(BF, 2, 4096, 14336, 32, 8, 128, rope_off=elem_offset(BF)),   # 3 launches
             rn_call(F, 3, 4096)]
    a = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    assert lib.tri_spec_set_code_dir(a, str(tmp_path).encode()) == 0
    for c in calls:
        assert c_call(lib, a, c) == 0
    assert lib.trifake_compile_count() == 5
    files = sorted(p.name for p in tmp_path.iterdir())
    assert len(files) == 5 and all(f.startswith("tri-") and f.endswith(".co") for f in files)
    v = VersionInfo()
    assert lib.tri_spec_version_info(a, 0, C.byref(v)) == 0 and v.jit == 1
    srcs_a = jit_sources(lib)
    # a second cache with the same directory loads every object, compiles none
    # (creating a cache here also resets the recording backend's counters)
    b = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    assert lib.tri_spec_set_code_dir(b, str(tmp_path).encode()) == 0
    for c in calls:
        assert c_call(lib, b, c) == 0
    assert lib.trifake_compile_count() == 0
    for i in range(3):
        assert lib.tri_spec_version_info(b, i, C.byref(v)) == 0 and v.jit == 2
    assert jit_sources(lib) == srcs_a                 # the same kernels, loaded
    # a corrupt object is recompiled and replaced
    (tmp_path / files[0]).write_bytes(b"garbage")
    c2 = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    lib.tri_spec_set_code_dir(c2, str(tmp_path).encode())
    for c in calls:
        assert c_call(lib, c2, c) == 0
    assert lib.trifake_compile_count() == 1
    assert (tmp_path / files[0]).read_bytes()[:4] == b"CO1:"
    # path limits
    assert lib.tri_spec_set_code_dir(c2, b"x" * 1024) == S.E_INVALID
    assert lib.tri_spec_set_code_dir(c2, None) == 0


def test_jit_failure_installs_nothing(lib, fresh):
    cache = fresh(flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    lib.trifake_jit_fail(1)
    assert c_call(lib, cache, chain_call(BF, 1, 256, 688, 4, 4, 64)) == S.E_RUNTIME
    assert c_stats(lib, cache)[5:] == (0, 0)
    lib.trifake_jit_fail(0)
    assert c_call(lib, cache, chain_call(BF, 1, 256, 688, 4, 4, 64)) == 0
    assert c_stats(lib, cache)[5:] == (1, 1)


def _hiprtc():
    h = C.CDLL("/opt/rocm/lib/libhiprtc.so")
    h.hiprtcCreateProgram.argtypes = [C.POINTER(C.c_void_p), C.c_char_p, C.c_char_p, C.c_int,
                                      C.c_void_p, C.c_void_p]
    h.hiprtcCompileProgram.argtypes = [C.c_void_p, C.c_int, C.POINTER(C.c_char_p)]
    h.hiprtcGetProgramLogSize.argtypes = [C.c_void_p, C.POINTER(C.c_size_t)]
    h.hiprtcGetProgramLog.argtypes = [C.c_void_p, C.c_char_p]
    h.hiprtcGetCodeSize.argtypes = [C.c_void_p, C.POINTER(C.c_size_t)]
    h.hiprtcDestroyProgram.argtypes = [C.POINTER(C.c_void_p)]
    return h


def _compile(h, src):
    prog = C.c_void_p()
    assert h.hiprtcCreateProgram(C.byref(prog), src.encode(), b"t.hip", 0, None, None) == 0
    opts = [b"--offload-arch=gfx950", b"-O3", b"-std=c++17", b"-ffp-contract=off", b"-Xclang",
            b"-target-feature", b"-Xclang", b"-packed-fp32-ops"]
    arr = (C.c_char_p * len(opts))(*opts)
    rc = h.hiprtcCompileProgram(prog, len(opts), arr)
    n = C.c_size_t()
    h.hiprtcGetProgramLogSize(prog, C.byref(n))
    log = C.create_string_buffer(n.value + 1)
    h.hiprtcGetProgramLog(prog, log)
    size = C.c_size_t()
    h.hiprtcGetCodeSize(prog, C.byref(size))
    h.hiprtcDestroyProgram(C.byref(prog))
    return rc, log.value.decode(errors="replace"), size.value


def test_every_kind_of_generated_source_compiles(lib, fresh):
    """hipRTC (it needs no GPU) compiles one source for every kernel body
    and template form the zoo's versions produce."""
    import os
    import re
    if not os.path.exists("/opt/rocm/lib/libhiprtc.so"):
        pytest.skip("hipRTC not installed")
    cache = fresh(capacity=S.MAX_CAPACITY, flags=S.FLAG_AUTO_INSTALL | S.FLAG_JIT)
    for c in call_zoo():
        c_call(lib, cache, c)
    forms = {}
    for src in jit_sources(lib):
        body = re.search(r"tri::dev::(\w+<[^>]*>)", _kernel_part(src)).group(1)
        forms.setdefault(body, src)
    assert len(forms) >= 30
    h = _hiprtc()
    for body, src in sorted(forms.items()):
        rc, log, size = _compile(h, src)
        assert rc == 0 and size > 0, (body, log[-2000:])


def test_export_import_prewarms_a_cache(lib, fresh):
    a = fresh(capacity=S.MAX_CAPACITY, flags=S.FLAG_AUTO_INSTALL)
    for c in call_zoo():
        c_call(lib, a, c)
    n = C.c_uint32()
    assert lib.tri_spec_export_keys(a, None, 0, C.byref(n)) == 0
    buf = (C.c_uint64 * (6 * n.value))()
    assert lib.tri_spec_export_keys(a, buf, n.value, C.byref(n)) == 0
    keys = [tuple(buf[6 * i: 6 * i + 6]) for i in range(n.value)]
    assert all(S.key_valid(k) for k in keys)
    assert 256 < n.value < S.MAX_CAPACITY
    b = fresh(capacity=S.MAX_CAPACITY)
    m = S.SpecCacheModel(capacity=S.MAX_CAPACITY)
    done = C.c_uint32()
    assert lib.tri_spec_import_keys(b, buf, n.value, C.byref(done)) == 0 and done.value == n.value
    assert m.import_keys(keys) == (S.OK, len(keys))
    for c in call_zoo():                     # no misses after the pre-warm
        assert run_both(lib, b, m, c, install=False) != S.MISS
    assert m.stats.misses == 0


def _mutations(key):
    k = list(key)
    out = []
    for word, shift, width in ((0, 0, 8), (0, 8, 8), (0, 16, 8), (0, 24, 8), (0, 32, 32),
                               (1, 0, 32), (1, 32, 32), (2, 0, 16), (2, 16, 16), (2, 32, 16),
                               (2, 48, 16), (3, 0, 16), (3, 16, 8), (3, 24, 8), (3, 32, 32),
                               (4, 0, 32), (4, 32, 32), (5, 0, 32), (5, 32, 32)):
        for val in (0, 1, 2, 3, 7, 0x7F, 0xFF, 0x7F800000, 0x3F800000, 0x4F000000, (1 << width) - 1):
            val &= (1 << width) - 1
            m = list(k)
            m[word] = (m[word] & ~(((1 << width) - 1) << shift)) | (val << shift)
            out.append(tuple(m))
    return out


def test_imported_keys_are_checked_like_the_model(lib, fresh):
    base_keys = [S.make_key(c) for c in (
        chain_call(BF, 8, 4096, 14336, 32, 8, 128, base=5e5),
        chain_call(F, 1, 256, 688, 4, 4, 64, qk_norm=True, ext=dict(interleaved=1, rotary_dim=32)),
        rope_call(BF, 3, 8, 2, 128, ext=dict(LLAMA3)),
        rope_call(BF, 3, 8, 2, 128, ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=7)),
        rn_call(F, 5, 4096), sw_call(BF, 9, 11008), qkn_call(BF, 1, 32, 8, 128))]
    seen = set()
    n_bad = 0
    for key in base_keys:
        for mk in [key] + _mutations(key):
            if mk in seen:
                continue
            seen.add(mk)
            cache = fresh()
            buf = (C.c_uint64 * 6)(*mk)
            done = C.c_uint32()
            st = lib.tri_spec_import_keys(cache, buf, 1, C.byref(done))
            want = S.key_valid(mk)
            assert (st == 0) == want, (hex(mk[0]), [hex(x) for x in mk], st)
            n_bad += not want
    assert n_bad > 100


# ---- argument preparation ----------------------------------------------------------
# Argument struct sizes the kernels take (RnArgs, RopeArgs, SwArgs, ChainArgs).
ARG_SIZES = {"rn": 88, "rope": 112, "sw": 80, "chain": 288}
RopeBlock = collections.namedtuple(
    "RopeBlock", "q k pos inv qw kw cos_sin q_ts k_ts T cs_len nq nk hd rd eps mode")


def rope_block(raw, off=0):
    return RopeBlock(*struct.unpack_from("<7Q4q4ifI", raw, off))


def _last_launch(lib, nbytes=512, size=None):
    i = lib.trifake_launch_count() - 1
    kv, dt, sub = C.c_int32(), C.c_int32(), C.c_int32()
    grid, block = C.c_uint32(), C.c_uint32()
    stream = C.c_void_p()
    buf = C.create_string_buffer(nbytes)
    n = lib.trifake_get(i, C.byref(kv), C.byref(dt), C.byref(sub), C.byref(grid),
                        C.byref(block), C.byref(stream), buf, nbytes)
    assert n >= 0
    if size is not None:
        assert n == ARG_SIZES[size]
    return kv.value, dt.value, sub.value, grid.value, block.value, stream.value, buf.raw


def test_long_rows_launch_split_wide_and_loop_forms(lib, fresh):
    """Residual rows beyond 4096 vectors are split over S = ceil(vectors /
    2048) workgroups of 256 (standalone, and as the norm launch of a
    three-launch chain), plain rows beyond 7168 vectors too (up to 256 rows); plain rows of
    4097..7168 vectors take one 1024-work-item workgroup, and so do rows of
    up to 8192 vectors where the split's scratch for the key's bucket would
    be too large; longer rows make two passes. Launches and records match
    the model's plan."""
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    cases = [(rn_call(BF, 3, 65536), [S.RN_SPLIT]), (rn_call(BF, 3, 57344), [S.RN_WIDE]),
             (res_call(BF, 3, 65536), [S.RN_SPLIT]),
             (res_call(F, 2, 20480), [S.RN_SPLIT]), (rn_call(F, 2, 20480), [S.RN_WIDE]),
             (rn_call(BF, 3, 65544), [S.RN_SPLIT]), (rn_call(BF, 3, 32768), [S.RN_BLOCK[16]]),
             (rn_call(BF, 3, 1048584), [S.RN_LOOP]),
             (res_call(BF, (1 << 19) + 1, 32776), [S.RN_WIDE]),
             (chain_call(BF, 2, 40960, 11008, 32, 32, 128), [S.RN_SPLIT, S.ROPE_VEC, S.SW_FLAT])]
    for c, kinds in cases:
        n0 = lib.trifake_launch_count()
        assert c_call(lib, cache, c) == 0
        got = [(l[0], l[3], l[4]) for l in (_launch_at(lib, i)
                                             for i in range(n0, lib.trifake_launch_count()))]
        want = [tuple(l) for l in S.plan(S.make_key(c), c.T)[2]]
        assert got == want and [g[0] for g in got] == kinds, (c.op, c.H, got)
        assert [g[2] for g in got] == [1024 if k == S.RN_WIDE else 256 for k in kinds]
        assert [tuple(l) for l in c_record(lib, cache)[6][:len(want)]] == want


@pytest.mark.parametrize("dtype,H", [(BF, 57344), (BF, 65536), (F, 32768), (BF, 32776)])
def test_plain_wide_rows_launch_at_most_256_workgroups(lib, fresh, dtype, H):
    """Plain rows of 4097..8192 vectors on the 1024-work-item form launch
    one workgroup per row up to 256 rows and 256 workgroups beyond (each
    taking every 256th row); rows of 7169..8192 vectors split up to 256
    rows. Launch and record against the model's plan at the edges."""
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    for T in (1, 255, 256, 257, 700, 2048, 4096):
        c = rn_call(dtype, T, H)
        n0 = lib.trifake_launch_count()
        assert c_call(lib, cache, c) == 0
        got = [(l[0], l[3], l[4]) for l in (_launch_at(lib, i)
                                             for i in range(n0, lib.trifake_launch_count()))]
        want = [tuple(l) for l in S.plan(S.make_key(c), T)[2]]
        assert got == want, (H, T, got, want)
        if T > 256:
            assert got == [(S.RN_WIDE, 256, 1024)]
        elif H // (16 // S.elem_size(dtype)) <= S.WIDE_PLAIN_VECS:
            assert got == [(S.RN_WIDE, T, 1024)]
        else:
            assert got[0][0] == S.RN_SPLIT


def test_split_rows_carry_the_version_scratch(lib, fresh):
    """A split version owns a zeroed scratch sized for the top of its token
    bucket (8 header words, S slots and one counter per row, 8 bytes each),
    allocated at install; every launch of the version passes its address
    after the row arguments (a 96-byte argument block); versions of other
    forms allocate none; the cache frees it."""
    import ctypes as C
    lib.trifake_zero_allocs.argtypes = [C.POINTER(C.c_int64)]
    counts = (C.c_int64 * 2)()
    cache = fresh(flags=S.FLAG_AUTO_INSTALL)
    lib.trifake_zero_allocs(counts)
    base = list(counts)
    c = res_call(BF, 3, 65536)                  # bucket 2 -> 4 rows, S = 4
    ptrs = []
    for _ in range(2):
        assert c_call(lib, cache, c) == 0
        kv, dt, sub, grid, block, stream, raw = _last_launch(lib)
        assert (kv, grid, block, sub) == (S.RN_SPLIT, 12, 256, 1)
        ptrs.append(int.from_bytes(raw[88:96], "little"))
    assert ptrs[0] == ptrs[1] != 0
    lib.trifake_zero_allocs(counts)
    assert (counts[0] - base[0], counts[1] - base[1]) == (1, 8 * (8 + 4 * 5))
    assert c_call(lib, cache, rn_call(BF, 3, 32768)) == 0      # RN_BLOCK[16]: none
    lib.trifake_zero_allocs(counts)
    assert counts[0] - base[0] == 1


def test_rmsnorm_argument_block_and_stream(lib, fresh):
    cache = fresh(flags=1)
    c = res_call(BF, 5, 4096, pad=64)
    assert c_call(lib, cache, c, stream=0xABC0) == 0
    kv, dt, sub, grid, block, stream, raw = _last_launch(lib, size="rn")
    assert (kv, dt, sub, grid, block, stream) == (S.RN_BLOCK[2], BF, 1, 5, 256, 0xABC0)
    f = struct.unpack_from("<5Q4qqif", raw)
    p = c.ptr
    assert f[:5] == (p["x"], p["res"], p["w"], p["y"], p["res_out"])
    assert f[5:9] == (4160,) * 4 and f[9:11] == (5, 4096)
    assert f[11] == np.float32(1e-6)


def test_chain_argument_block(lib, fresh):
    cache = fresh(flags=1)
    c = chain_call(BF, 8, 4096, 14336, 32, 8, 128, base=500000.0)
    assert c_call(lib, cache, c) == 0
    kv, dt, sub, grid, block, _, raw = _last_launch(lib, size="chain")
    # fused kernel: RN_BLOCK_2 (norm role index 3), plain RoPE, cached one-vector SwiGLU;
    # RoPE: 40 heads x 8 lanes = 320 > 256 -> two workgroups per token
    assert (kv, dt, sub, grid, block) == (50, BF, 3 * 8, 8 + 16 + 56, 256)
    rope = rope_block(raw, 88)
    assert (rope.q, rope.k, rope.pos) == (c.ptr["q"], c.ptr["k"], c.ptr["pos"])
    assert (rope.qw, rope.kw, rope.cos_sin, rope.eps, rope.mode) == (0, 0, 0, 0.0, 2 << 8)
    assert (rope.q_ts, rope.k_ts, rope.T, rope.cs_len) == (32 * 128, 8 * 128, 8, 0)
    assert (rope.nq, rope.nk, rope.hd, rope.rd) == (32, 8, 128, 128)
    sw = struct.unpack_from("<3Q7q", raw, 200)
    assert sw[:3] == (c.ptr["gate"], c.ptr["up"], c.ptr["out"])
    assert sw[3:] == (14336, 14336, 14336, 8, 14336, 8 * 14336 // 8, 8 * 14336)
    assert struct.unpack_from("<2I", raw, 280) == (8, 16)
    # the RoPE table pointer is this version's uploaded constants
    assert rope.inv != 0


def test_qk_norm_chain_argument_block(lib, fresh):
    cache = fresh(flags=1)
    c = chain_call(BF, 1, 4096, 12288, 32, 8, 128, base=1e6, qk_norm=True, qk_eps=1e-5)
    assert c_call(lib, cache, c) == 0
    kv, dt, sub, grid, block, _, raw = _last_launch(lib, size="chain")
    # RN_BLOCK_2 with the QK-norm RoPE role and cached SwiGLU
    assert (kv, dt, sub, grid, block) == (50, BF, 3 * 8 + 2, 1 + 2 + 6, 256)
    rope = rope_block(raw, 88)
    assert (rope.qw, rope.kw) == (c.ptr["q_w"], c.ptr["k_w"])
    assert rope.eps == np.float32(1e-5)
    assert S.unpack_key(S.make_key(c))["flags"] == 0x7F
    # the standalone op launches the same role body with the same block
    c2 = qkn_call(BF, 1, 32, 8, 128, base=1e6, eps=1e-5)
    assert c_call(lib, cache, c2) == 0
    kv2, _, _, grid2, _, _, raw2 = _last_launch(lib, size="rope")
    assert (kv2, grid2) == (S.ROPE_QKN_VEC, 2)
    assert rope_block(raw2)[4:] == rope[4:]   # all but the per-version table


def test_qk_norm_without_k_heads_passes_no_k_weight(lib, fresh):
    cache = fresh(flags=1)
    c = qkn_call(F, 2, 4, 0, 64)
    assert c_call(lib, cache, c) == 0
    rope = rope_block(_last_launch(lib, size="rope")[6])
    assert rope.k == 0 and rope.qw == c.ptr["q_w"] and rope.kw == 0


@pytest.mark.parametrize("base,hd", [(10000.0, 64), (10000.0, 128), (500000.0, 128),
                                     (10000.0, 96), (10000.0, 512), (1234.5, 2),
                                     (1e6, 256), (2.0, 128)])
def test_rope_table_matches_oracle_exactly(lib, fresh, base, hd):
    cache = fresh(flags=1)
    assert c_call(lib, cache, rope_call(BF, 3, 4, 2, hd, base=base)) == 0
    n = C.c_uint32()
    buf = (C.c_float * 256)()
    assert lib.tri_spec_version_constants(cache, 0, buf, 256, C.byref(n)) == 0
    got = np.array(buf[: n.value], dtype=np.float32)
    want = O.rope_inv_freq(base, hd)
    assert n.value == hd // 2
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("base,hd,rd", [(5e5, 128, 128), (5e5, 128, 64), (1e4, 64, 32),
                                        (5e5, 256, 256), (1e6, 128, 96)])
def test_llama3_table_matches_oracle_exactly(lib, fresh, base, hd, rd):
    cache = fresh(flags=1)
    assert c_call(lib, cache, rope_call(BF, 3, 4, 2, hd, base=base,
                                        ext=dict(LLAMA3, rotary_dim=rd))) == 0
    n = C.c_uint32()
    buf = (C.c_float * 256)()
    assert lib.tri_spec_version_constants(cache, 0, buf, 256, C.byref(n)) == 0
    got = np.array(buf[: n.value], dtype=np.float32)
    want = O.rope_inv_freq_llama3(base, rd, 8.0, 1.0, 4.0, 8192)
    assert n.value == rd // 2
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_partial_rotary_table_and_cache_mode_constants(lib, fresh):
    cache = fresh(flags=1)
    assert c_call(lib, cache, rope_call(F, 2, 4, 2, 128, ext=dict(rotary_dim=32))) == 0
    assert c_call(lib, cache, rope_call(F, 2, 4, 2, 128,
                                        ext=dict(cos_sin=CACHE_ADDR, cos_sin_len=9))) == 0
    n = C.c_uint32()
    buf = (C.c_float * 256)()
    assert lib.tri_spec_version_constants(cache, 0, buf, 256, C.byref(n)) == 0
    assert np.array_equal(np.array(buf[:n.value], dtype=np.float32), O.rope_inv_freq(1e4, 32))
    assert lib.tri_spec_version_constants(cache, 1, buf, 256, C.byref(n)) == 0
    assert n.value == 0
    rope = rope_block(_last_launch(lib, size="rope")[6])
    assert (rope.inv, rope.cos_sin, rope.cs_len, rope.mode) == (0, CACHE_ADDR, 9, 4)


def test_rope_ext_argument_block(lib, fresh):
    cache = fresh(flags=1)
    c = rope_call(BF, 3, 8, 2, 128, ext=dict(rotary_dim=64, interleaved=1, pos_int64=1))
    assert c_call(lib, cache, c) == 0
    kv, _, _, grid, _, _, raw = _last_launch(lib, size="rope")
    assert (kv, grid) == (S.ROPE_VEC_I, 3)
    rope = rope_block(raw)
    assert (rope.hd, rope.rd, rope.mode, rope.pos) == (128, 64, 1 | 2, c.ptr["pos"])


def test_plain_ext_shares_versions_with_the_plain_entry(lib, fresh):
    # A zeroed variant struct and the plain entry point make the same key.
    cache = fresh()
    m = S.SpecCacheModel()
    run_both(lib, cache, m, rope_call(BF, 1, 32, 8, 128))
    run_both(lib, cache, m, rope_call(BF, 1, 32, 8, 128, ext={}))
    run_both(lib, cache, m, rope_call(BF, 1, 32, 8, 128, ext=dict(rotary_dim=128)))
    assert m.stats.installs == 1 and m.stats.hits == 3


def test_version_info(lib, fresh):
    from paper_2609_37241_amd._lib import VersionInfo
    cache = fresh(flags=1)
    c = chain_call(F, 4, 256, 688, 4, 4, 64)
    for _ in range(3):
        c_call(lib, cache, c)
    v = VersionInfo()
    assert lib.tri_spec_version_info(cache, 0, C.byref(v)) == 0
    assert (v.variant, tuple(v.roles), v.hits) == (50, (11, 31, 41), 2)
    assert tuple(v.key) == S.make_key(c)
    assert lib.tri_spec_version_info(cache, 1, C.byref(v)) == S.E_INVALID
