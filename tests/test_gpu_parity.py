"""GPU parity: the HIP path through the C ABI vs the CPU oracle.

Every case prints its name (pytest -v) before touching the GPU. Inputs come
from the seeded generators in `workloads`; expected values only from
`oracle`. Selection records are compared with the oracle's selection model.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from oracle import selection as S
from tests.parity import (binding_rope_ext, check, expected_record, model_chain_call,
                          oracle_rope_kw)
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


@pytest.fixture
def cache(tri):
    c = tri.SpecCache()
    yield c
    torch.cuda.synchronize()
    c.close()


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def place(a: np.ndarray, dtype: str, layout: str = "plain", pad: int = 64):
    """Host array [T, W] or [T, nh, hd] -> device tensor with the given layout."""
    src = wl.to_torch(a, dtype, DEV)
    shape = src.shape
    T = shape[0]
    W = int(np.prod(shape[1:]))
    td = src.dtype
    if layout == "plain":
        return src.contiguous()
    if layout == "strided":
        buf = torch.zeros((T, W + pad), dtype=td, device=DEV)
        rs = W + pad
    elif layout == "unaligned":
        buf = torch.zeros(T * W + 1, dtype=td, device=DEV)
        rs = W
    else:
        raise ValueError(layout)
    strides = (rs,) + tuple(int(np.prod(shape[i + 1:])) for i in range(1, len(shape)))
    off = 1 if layout == "unaligned" else 0
    view = torch.as_strided(buf, size=shape, stride=strides, storage_offset=off)
    view.copy_(src)
    return view


def empty_like_layout(t):
    """Output tensor with the same layout (strides, 16-byte phase) as t."""
    buf = torch.zeros(t.untyped_storage().nbytes() // t.element_size(), dtype=t.dtype,
                      device=DEV)
    return torch.as_strided(buf, size=t.shape, stride=t.stride(),
                            storage_offset=t.storage_offset())


def host(t):
    return wl.from_torch(t)


# ---- the configured chains ---------------------------------------------------------
TINY_QKN_F32 = wl.ChainConfig("tiny_qkn_f32", wl.F32, T=3, H=256, nq=4, nk=2, hd=64, I=688,
                              base=1e6, pos_mode="uniform", pos_max=4095, qk_norm=True)
CHAIN_CFGS = [wl.TINY_F32, wl.LLAMA7B_DECODE, wl.GQA_DECODE, wl.QWEN3_8B_DECODE, TINY_QKN_F32,
              wl.LLAMA31_8B_DECODE, wl.GPTJ_DECODE]


def run_chain(cache, cfg, d):
    """decode_chain over device tensors d (head-norm weights when present)."""
    import paper_2609_37241_amd as tri
    rope = binding_rope_ext(tri, cfg.rope_ext) if cfg.rope_ext else None
    cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"], d["gate"],
                       d["up"], cfg.eps, cfg.base, y=d["y"], residual_out=d["res_out"],
                       out=d["out"], q_norm_w=d.get("q_norm_w"), k_norm_w=d.get("k_norm_w"),
                       rope=rope)


def chain_oracle(inp, cfg):
    if cfg.rope_ext:
        inp = dict(inp, rope_ext=oracle_rope_kw(cfg.rope_ext))
    return O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)


@pytest.mark.parametrize("cfg", CHAIN_CFGS, ids=lambda c: c.name)
def test_chain_config(tri, cache, cfg):
    inp = wl.host_inputs(cfg)
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    d["y"] = torch.empty_like(d["x"])
    d["res_out"] = torch.empty_like(d["x"])
    d["out"] = torch.empty_like(d["gate"])
    run_chain(cache, cfg, d)
    torch.cuda.synchronize()
    want = chain_oracle(inp, cfg)
    check("y", host(d["y"]), want["y"], cfg.dtype)
    check("res_out", host(d["res_out"]), want["res_out"], cfg.dtype, exact=True)
    check("q", host(d["q"]), want["q"], cfg.dtype)
    check("k", host(d["k"]), want["k"], cfg.dtype)
    check("out", host(d["out"]), want["out"], cfg.dtype)
    rec = cache.last_selection().as_tuple()
    assert rec == expected_record(model_chain_call(d, cfg.eps, cfg.base, ext=cfg.rope_ext), 0)
    assert rec[3] == S.CH_FUSED


@pytest.mark.parametrize("cfg", CHAIN_CFGS, ids=lambda c: c.name)
def test_fused_chain_equals_separate_ops_bitwise(tri, cache, cfg):
    inp = wl.host_inputs(cfg)
    a = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    b = {k: v.clone() for k, v in a.items()}
    rope = binding_rope_ext(tri, cfg.rope_ext) if cfg.rope_ext else None
    y, ro, out = cache.decode_chain(a["x"], a["residual"], a["w"], a["q"], a["k"], a["pos"],
                                    a["gate"], a["up"], cfg.eps, cfg.base,
                                    q_norm_w=a.get("q_norm_w"), k_norm_w=a.get("k_norm_w"),
                                    rope=rope)
    assert cache.last_selection().variant == S.CH_FUSED
    y2, ro2 = cache.residual_rmsnorm(b["x"], b["residual"], b["w"], cfg.eps)
    if cfg.rope_ext:
        cache.rope(b["q"], b["k"], b["pos"], cfg.base, rope, q_w=b.get("q_norm_w"),
                   k_w=b.get("k_norm_w"), eps=cfg.eps)
    elif cfg.qk_norm:
        cache.qk_norm_rope(b["q"], b["k"], b["pos"], b["q_norm_w"], b["k_norm_w"], cfg.base,
                           cfg.eps)
    else:
        cache.rope_qk(b["q"], b["k"], b["pos"], cfg.base)
    out2 = cache.swiglu(b["gate"], b["up"])
    torch.cuda.synchronize()
    for n, g, h in (("y", y, y2), ("res_out", ro, ro2), ("q", a["q"], b["q"]),
                    ("k", a["k"], b["k"]), ("out", out, out2)):
        check(n, host(g), host(h), cfg.dtype, exact=True)


# ---- RMSNorm / residual RMSNorm: every variant ------------------------------------------
RN_CASES = [
    # dtype, T, H, layout -> variant (by the policy table)
    (nm.F32, 5, 64, "plain"), (nm.F32, 5, 100, "plain"), (nm.F32, 37, 520, "plain"),
    (nm.F32, 6, 4096, "plain"), (nm.F32, 3, 8192, "plain"), (nm.F32, 3, 16384, "plain"),
    (nm.F32, 2, 65536, "plain"), (nm.F32, 5, 4097, "plain"), (nm.F32, 7, 4096, "unaligned"),
    (nm.F32, 7, 4096, "strided"),
    (nm.BF16, 1, 4096, "plain"), (nm.BF16, 9, 256, "plain"), (nm.BF16, 9, 520, "plain"),
    (nm.BF16, 6, 4096, "plain"), (nm.BF16, 5, 8192, "plain"), (nm.BF16, 3, 32768, "plain"),
    (nm.BF16, 2, 65536, "plain"), (nm.BF16, 4, 100, "plain"), (nm.BF16, 7, 4096, "unaligned"),
    (nm.BF16, 7, 4096, "strided"), (nm.BF16, 3, 1, "plain"),
    # more rows and short rows (a wavefront per row, 4 rows per block)
    (nm.BF16, 130, 4096, "plain"), (nm.F32, 100, 256, "plain"), (nm.BF16, 70, 8192, "plain"),
    (nm.F32, 65, 4096, "unaligned"), (nm.BF16, 66, 4096, "strided"), (nm.F32, 67, 16384, "plain"),
    (nm.BF16, 13, 1024, "plain"), (nm.BF16, 13, 1032, "plain"), (nm.F32, 7, 512, "plain"),
    # rows beyond 4096 vectors: residual rows (and plain rows beyond 8192
    # vectors) split over ceil(vectors / 2048) workgroups (3..16 here, a
    # ragged last slice at 8193 vectors), plain rows of up to 8192 vectors
    # in one 1024-lane workgroup (4097 vectors: one lane group holds the
    # last vector), two passes beyond 64 slices
    (nm.BF16, 3, 32776, "plain"), (nm.F32, 4, 16388, "strided"), (nm.BF16, 9, 32776, "unaligned"),
    (nm.BF16, 5, 40960, "plain"), (nm.BF16, 3, 65536, "strided"), (nm.BF16, 67, 49152, "plain"),
    (nm.BF16, 2, 65544, "plain"), (nm.F32, 4, 20480, "plain"), (nm.F32, 3, 32768, "plain"),
    (nm.F32, 2, 32772, "plain"), (nm.F32, 2, 131072, "plain"), (nm.BF16, 5, 40960, "unaligned"),
    (nm.BF16, 300, 65536, "plain"), (nm.BF16, 3, 1048576, "plain"), (nm.F32, 2, 524288, "plain"),
    (nm.BF16, 2, 1048584, "plain"), (nm.F32, 2, 524292, "plain"),
    # plain rows of 4097..7168 vectors beyond 256 rows: 256 workgroups, each
    # taking every 256th row (1 to 4 rows; an odd and an even count end the
    # two-buffer loop on either buffer); a ragged 4097-vector row, strided
    (nm.BF16, 257, 57344, "plain"), (nm.F32, 600, 20480, "plain"),
    (nm.BF16, 513, 32776, "strided"), (nm.BF16, 1000, 49152, "plain"),
]


@pytest.mark.parametrize("res", [False, True], ids=["rmsnorm", "residual"])
@pytest.mark.parametrize("dtype,T,H,layout", RN_CASES)
def test_rmsnorm_variants(tri, cache, dtype, T, H, layout, res):
    r = rng(T * 131 + H)
    x = wl.host_array(r, (T, H), dtype)
    rr = wl.host_array(r, (T, H), dtype)
    w = wl.host_weight(r, H, dtype)
    xd = place(x, dtype, layout)
    wd = wl.to_torch(w, dtype, DEV)
    yd = empty_like_layout(xd)
    if res:
        rd = place(rr, dtype, layout)
        rod = empty_like_layout(xd)
        cache.residual_rmsnorm(xd, rd, wd, 1e-6, out=yd, residual_out=rod)
        want_y, want_h = O.residual_rmsnorm(x, rr, w, 1e-6, dtype)
    else:
        cache.rmsnorm(xd, wd, 1e-6, out=yd)
        want_y = O.rmsnorm(x, w, 1e-6, dtype)
    torch.cuda.synchronize()
    check("y", host(yd), want_y, dtype)
    if res:
        check("res_out", host(rod), want_h, dtype, exact=True)
    sel = cache.last_selection()
    es = 4 if dtype == nm.F32 else 2
    flags = S.ALIGN if (xd.data_ptr() % 16 == 0 and (xd.stride(0) * es) % 16 == 0) else 0
    assert (sel.variant, sel.launch[0].grid_x) == S.rn_role(
        S.DT_F32 if dtype == nm.F32 else S.DT_BF16, H, flags, T, S.bucket(T), res)


@pytest.mark.parametrize("dtype,H", [(nm.BF16, 57344), (nm.F32, 20480), (nm.BF16, 32776)])
def test_plain_wide_rows_same_bits_at_any_row_count(tri, cache, dtype, H):
    """Plain rows of 4097..7168 vectors: one call of 600 rows (256 workgroups
    that take 2-3 rows each, the next row requested before the current
    row's reduction) gives every row the same bits as calls of at most 256
    rows (one row per workgroup), and the oracle's values."""
    r = rng(H + 600)
    T = 600
    x = wl.host_array(r, (T, H), dtype)
    w = wl.host_weight(r, H, dtype)
    xd, wd = wl.to_torch(x, dtype, DEV), wl.to_torch(w, dtype, DEV)
    whole = cache.rmsnorm(xd, wd, 1e-6)
    sel = cache.last_selection()
    assert (sel.variant, sel.launch[0].grid_x) == (S.RN_WIDE, 256)
    parts = []
    for lo in range(0, T, 256):
        parts.append(cache.rmsnorm(xd[lo:lo + 256], wd, 1e-6))
        sel = cache.last_selection()
        assert (sel.variant, sel.launch[0].grid_x) == (S.RN_WIDE, min(256, T - lo))
    torch.cuda.synchronize()
    check("600 rows vs chunks", host(whole), host(torch.cat(parts)), dtype, exact=True)
    check("600 rows vs oracle", host(whole), O.rmsnorm(x, w, 1e-6, dtype), dtype)


def test_split_rows_reuse_their_scratch(tri, cache):
    """A split version's scratch is cleared by each call's last readers, so
    back-to-back calls of one version (different data, fewer rows within the
    bucket, the plain and the residual form, and calls of other versions in
    between) each match the oracle; every row is checked."""
    r = rng(17)
    H = 65536                                   # bf16: 8192 vectors, 4 workgroups per row
    w = wl.host_weight(r, H, nm.BF16)
    wd = wl.to_torch(w, nm.BF16, DEV)
    for step, T in enumerate((7, 8, 5, 8, 1)):  # bucket 3 for all but the last
        x = wl.host_array(r, (T, H), nm.BF16)
        res = wl.host_array(r, (T, H), nm.BF16)
        xd, rd = wl.to_torch(x, nm.BF16, DEV), wl.to_torch(res, nm.BF16, DEV)
        y = cache.rmsnorm(xd, wd, 1e-6)
        y2, ro = cache.residual_rmsnorm(xd, rd, wd, 1e-6)
        z = cache.rmsnorm(xd[:, :4096].contiguous(), wd[:4096].contiguous(), 1e-6)
        torch.cuda.synchronize()
        assert cache.last_selection().variant != S.RN_SPLIT
        check(f"{step} y", host(y), O.rmsnorm(x, w, 1e-6, nm.BF16), nm.BF16)
        wy, wh = O.residual_rmsnorm(x, res, w, 1e-6, nm.BF16)
        check(f"{step} residual y", host(y2), wy, nm.BF16)
        check(f"{step} res_out", host(ro), wh, nm.BF16, exact=True)
        check(f"{step} short rows", host(z), O.rmsnorm(x[:, :4096], w[:4096], 1e-6, nm.BF16),
              nm.BF16)
    kinds = {cache.version_info(i).variant for i in range(cache.stats()["n_versions"])}
    assert S.RN_SPLIT in kinds


def test_generic_split_version_across_buckets(tri):
    """One generic split version of residual bf16 rows of 65536 (4
    workgroups per row) serves calls of 1 to 700 rows, buckets 0 to 10,
    through one scratch sized for the top of its run; plain rows of 65536
    split up to 256 rows (buckets 0-8, one generic version) and take a
    second generic version on 256 1024-lane workgroups beyond (the 700-row
    call); plain rows of 57344 (7168 vectors) take one generic 1024-lane
    version over every bucket and their row class; every row of every call
    against the oracle."""
    r = rng(19)
    H = 65536
    w = wl.host_weight(r, H, nm.BF16)
    wd = wl.to_torch(w, nm.BF16, DEV)
    c = tri.SpecCache(auto_install=True, generic=True)
    try:
        for step, T in enumerate((3, 700, 1, 64, 129, 2)):
            print(f"generic split: call {step}, {T} rows", flush=True)
            x = wl.host_array(r, (T, H), nm.BF16)
            res = wl.host_array(r, (T, H), nm.BF16)
            xd, rd = wl.to_torch(x, nm.BF16, DEV), wl.to_torch(res, nm.BF16, DEV)
            y = c.rmsnorm(xd, wd, 1e-6)
            sel = c.last_selection()
            y2, ro = c.residual_rmsnorm(xd, rd, wd, 1e-6)
            sel2 = c.last_selection()
            y3 = c.rmsnorm(xd[:, :57344], wd[:57344], 1e-6)
            sel3 = c.last_selection()
            torch.cuda.synchronize()
            assert (sel.variant, sel.launch[0].grid_x) == (
                (S.RN_SPLIT, 4 * T) if T <= 256 else (S.RN_WIDE, 256))
            assert sel2.variant == S.RN_SPLIT and sel2.launch[0].grid_x == 4 * T
            assert sel3.variant == S.RN_WIDE and sel3.launch[0].grid_x == min(T, 256)
            check(f"{step} y", host(y), O.rmsnorm(x, w, 1e-6, nm.BF16), nm.BF16)
            check(f"{step} y 57344", host(y3), O.rmsnorm(x[:, :57344], w[:57344], 1e-6, nm.BF16),
                  nm.BF16)
            wy, wh = O.residual_rmsnorm(x, res, w, 1e-6, nm.BF16)
            check(f"{step} residual y", host(y2), wy, nm.BF16)
            check(f"{step} res_out", host(ro), wh, nm.BF16, exact=True)
        st = c.stats()
        # plain, residual, plain 57344 (first call); plain 700 rows (second)
        assert st["n_versions"] == 4 and st["misses"] == 4
        guards = [(c.version_info(i).variant, c.version_info(i).b_lo, c.version_info(i).b_hi,
                   c.version_info(i).h_lo, c.version_info(i).h_hi) for i in range(4)]
        assert guards == [(S.RN_SPLIT, 0, 8, 0, 0), (S.RN_SPLIT, 0, 19, 0, 0),
                          (S.RN_WIDE, 0, 22, 32776, 57344), (S.RN_WIDE, 9, 22, 0, 0)]
    finally:
        torch.cuda.synchronize()
        c.close()


def test_rmsnorm_in_place(tri, cache):
    r = rng(3)
    x = wl.host_array(r, (6, 4096), nm.BF16)
    w = wl.host_weight(r, 4096, nm.BF16)
    xd = wl.to_torch(x, nm.BF16, DEV)
    cache.rmsnorm(xd, wl.to_torch(w, nm.BF16, DEV), 1e-6, out=xd)
    torch.cuda.synchronize()
    check("y", host(xd), O.rmsnorm(x, w, 1e-6, nm.BF16), nm.BF16)


# ---- RoPE: every variant ---------------------------------------------------------------
ROPE_CASES = [
    # dtype, T, nq, nk, hd, base, layout
    (nm.BF16, 1, 32, 32, 128, 1e4, "plain"), (nm.BF16, 8, 32, 8, 128, 5e5, "plain"),
    (nm.BF16, 37, 32, 8, 128, 5e5, "plain"), (nm.F32, 4, 4, 4, 64, 1e4, "plain"),
    (nm.F32, 19, 4, 4, 64, 1e4, "plain"), (nm.BF16, 5, 2, 2, 96, 1e4, "plain"),
    (nm.F32, 3, 3, 0, 128, 1e4, "plain"), (nm.BF16, 6, 4, 4, 512, 1e4, "plain"),
    (nm.F32, 6, 2, 3, 512, 1e4, "plain"), (nm.F32, 2, 2, 2, 2, 1e4, "plain"),
    (nm.BF16, 9, 8, 2, 128, 5e5, "unaligned"), (nm.F32, 9, 8, 2, 128, 5e5, "strided"),
    (nm.BF16, 17, 64, 8, 128, 5e5, "plain"),
]


@pytest.mark.parametrize("dtype,T,nq,nk,hd,base,layout", ROPE_CASES)
def test_rope_variants(tri, cache, dtype, T, nq, nk, hd, base, layout):
    r = rng(T * 7 + nq * 13 + hd)
    q = wl.host_array(r, (T, nq, hd), dtype)
    k = wl.host_array(r, (T, nk, hd), dtype)
    pos = r.integers(0, 8192, size=T).astype(np.int32)
    qd = place(q, dtype, layout)
    kd = place(k, dtype, layout) if nk else None
    cache.rope_qk(qd, kd, wl.to_torch(pos, dtype, DEV), base)
    torch.cuda.synchronize()
    wq, wk = O.rope_qk(q, k, pos, base, dtype)
    check("q", host(qd), wq, dtype)
    if nk:
        check("k", host(kd), wk, dtype)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_rope_position_zero_is_exact_identity(tri, cache, dtype):
    r = rng(11)
    q = wl.host_array(r, (12, 8, 128), dtype)
    k = wl.host_array(r, (12, 2, 128), dtype)
    qd, kd = wl.to_torch(q, dtype, DEV), wl.to_torch(k, dtype, DEV)
    cache.rope_qk(qd, kd, torch.zeros(12, dtype=torch.int32, device=DEV), 5e5)
    torch.cuda.synchronize()
    check("q", host(qd), q, dtype, exact=True)
    check("k", host(kd), k, dtype, exact=True)


# ---- QK-RMSNorm + RoPE: every variant ------------------------------------------------
QKN_CASES = [
    # dtype, T, nq, nk, hd, layout, weight offset (elements); vector cases cover
    # every lane-group width of the head reduction (hd/2 / V = 1 .. 64 lanes)
    (nm.BF16, 1, 32, 8, 128, "plain", 0), (nm.BF16, 8, 32, 8, 128, "plain", 0),
    (nm.BF16, 37, 64, 8, 128, "plain", 0), (nm.BF16, 5, 8, 8, 16, "plain", 0),
    (nm.BF16, 5, 8, 4, 32, "plain", 0), (nm.BF16, 5, 8, 4, 64, "plain", 0),
    (nm.BF16, 5, 8, 4, 256, "plain", 0), (nm.BF16, 3, 4, 4, 512, "plain", 0),
    (nm.F32, 5, 8, 8, 8, "plain", 0), (nm.F32, 5, 8, 4, 16, "plain", 0),
    (nm.F32, 5, 8, 4, 32, "plain", 0), (nm.F32, 5, 8, 4, 64, "plain", 0),
    (nm.F32, 19, 64, 8, 128, "plain", 0), (nm.F32, 5, 8, 4, 256, "plain", 0),
    (nm.F32, 3, 2, 3, 512, "plain", 0), (nm.F32, 4, 3, 0, 128, "plain", 0),
    (nm.BF16, 9, 8, 2, 128, "strided", 0),
    # scalar role: unaligned operands or weights, half-heads not a power of two
    # of vectors, head counts beyond one 256-head slice
    (nm.BF16, 9, 8, 2, 128, "unaligned", 0), (nm.F32, 9, 8, 2, 128, "plain", 1),
    (nm.BF16, 5, 2, 2, 96, "plain", 0), (nm.F32, 2, 2, 2, 2, "plain", 0),
    (nm.BF16, 3, 300, 20, 64, "unaligned", 0), (nm.F32, 3, 5, 0, 64, "unaligned", 0),
]


def place_weight(w: np.ndarray, dtype: str, off: int):
    """A head-norm weight [hd] on the device, `off` elements past 16 B."""
    src = wl.to_torch(w, dtype, DEV)
    buf = torch.zeros(w.shape[0] + 8, dtype=src.dtype, device=DEV)
    view = buf[off:off + w.shape[0]]
    view.copy_(src)
    return view


@pytest.mark.parametrize("dtype,T,nq,nk,hd,layout,w_off", QKN_CASES)
def test_qk_norm_rope_variants(tri, cache, dtype, T, nq, nk, hd, layout, w_off):
    r = rng(T * 5 + nq * 11 + hd + w_off)
    q = wl.host_array(r, (T, nq, hd), dtype)
    k = wl.host_array(r, (T, nk, hd), dtype)
    qw, kw = wl.host_weight(r, hd, dtype), wl.host_weight(r, hd, dtype)
    pos = r.integers(0, 8192, size=T).astype(np.int32)
    qd = place(q, dtype, layout)
    kd = place(k, dtype, layout) if nk else None
    qwd, kwd = place_weight(qw, dtype, w_off), place_weight(kw, dtype, w_off)
    cache.qk_norm_rope(qd, kd, wl.to_torch(pos, dtype, DEV), qwd, kwd if nk else None, 1e6,
                       1e-6)
    torch.cuda.synchronize()
    wq, wk = O.qk_norm_rope(q, k, pos, 1e6, qw, kw, 1e-6, dtype)
    check("q", host(qd), wq, dtype)
    if nk:
        check("k", host(kd), wk, dtype)
    c = S.Call(S.OP_QK_NORM_ROPE, S.DT_F32 if dtype == nm.F32 else S.DT_BF16, T, hd=hd,
               nq=nq, nk=nk, base=1e6, eps=1e-6,
               ptr=dict(q=qd.data_ptr(), k=kd.data_ptr() if nk else None, pos=0,
                        q_w=qwd.data_ptr(), k_w=kwd.data_ptr() if nk else None),
               stride=dict(q=qd.stride(0) if T > 1 else nq * hd,
                           k=(kd.stride(0) if T > 1 else nk * hd) if nk else 0))
    assert cache.last_selection().variant == S.plan(S.make_key(c), T)[0]


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_qk_norm_rope_zero_heads_and_position_zero(tri, cache, dtype):
    # A zero head normalises to zero (eps > 0); at position 0 the rotation is
    # the identity, so the op is exactly a per-head RMSNorm.
    r = rng(23)
    q = wl.host_array(r, (6, 8, 128), dtype)
    k = wl.host_array(r, (6, 2, 128), dtype)
    q[2, 3] = 0
    k[4, 1] = 0
    qw, kw = wl.host_weight(r, 128, dtype), wl.host_weight(r, 128, dtype)
    qd, kd = wl.to_torch(q, dtype, DEV), wl.to_torch(k, dtype, DEV)
    cache.qk_norm_rope(qd, kd, torch.zeros(6, dtype=torch.int32, device=DEV),
                       wl.to_torch(qw, dtype, DEV), wl.to_torch(kw, dtype, DEV), 1e4, 1e-6)
    torch.cuda.synchronize()
    gq, gk = host(qd), host(kd)
    assert not nm.values(gq[2, 3], dtype).any() and not nm.values(gk[4, 1], dtype).any()
    check("q", gq, O.rmsnorm(q, qw, 1e-6, dtype), dtype)
    check("k", gk, O.rmsnorm(k, kw, 1e-6, dtype), dtype)


# ---- RoPE variants ----------------------------------------------------------------------
LLAMA3 = dict(scaling=S.SCALING_LLAMA3, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0,
              original_max_pos=8192)
EXT_CASES = [
    # dtype, T, nq, nk, hd, variant, QK norm, layout
    (nm.BF16, 5, 8, 2, 128, dict(rotary_dim=64), False, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(rotary_dim=96), False, "plain"),
    (nm.F32, 5, 8, 2, 128, dict(rotary_dim=32), False, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(interleaved=1), False, "plain"),
    (nm.F32, 9, 8, 2, 64, dict(interleaved=1), False, "plain"),
    (nm.F32, 3, 2, 2, 512, dict(interleaved=1), False, "plain"),
    (nm.BF16, 3, 2, 2, 512, dict(interleaved=1), True, "plain"),
    (nm.F32, 3, 2, 2, 512, dict(interleaved=1), True, "plain"),
    (nm.BF16, 7, 8, 2, 128, dict(interleaved=1, rotary_dim=64), False, "plain"),
    (nm.BF16, 7, 8, 2, 96, dict(interleaved=1), False, "plain"),
    (nm.BF16, 6, 8, 2, 128, dict(pos_int64=1), False, "plain"),
    (nm.F32, 6, 8, 2, 128, LLAMA3, False, "plain"),
    (nm.BF16, 6, 32, 8, 128, dict(LLAMA3, rotary_dim=64, interleaved=1, pos_int64=1), False,
     "plain"),
    (nm.BF16, 6, 8, 2, 128, dict(cache=1), False, "plain"),
    (nm.F32, 6, 8, 2, 64, dict(cache=1, interleaved=1, pos_int64=1), False, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(rotary_dim=64), True, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(interleaved=1), True, "plain"),
    (nm.F32, 5, 8, 2, 128, dict(interleaved=1, cache=1), True, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(interleaved=1), False, "unaligned"),
    (nm.F32, 4, 300, 20, 64, dict(interleaved=1, rotary_dim=48), True, "unaligned"),
]


@pytest.mark.parametrize("dtype,T,nq,nk,hd,ext,qkn,layout", EXT_CASES)
def test_rope_variant_cases(tri, cache, dtype, T, nq, nk, hd, ext, qkn, layout):
    r = rng(T * 3 + nq * 7 + hd + 5 * len(ext) + qkn)
    q = wl.host_array(r, (T, nq, hd), dtype)
    k = wl.host_array(r, (T, nk, hd), dtype)
    qw, kw = wl.host_weight(r, hd, dtype), wl.host_weight(r, hd, dtype)
    ext = dict(ext)
    rd = ext.get("rotary_dim") or hd
    table = None
    if ext.pop("cache", 0):
        table = wl.cos_sin_table(r, 300, rd)
        pos = r.integers(-20, 320, size=T)              # some clamp at either end
    elif ext.get("pos_int64"):
        pos = r.integers(0, 1 << 40, size=T)
    else:
        pos = r.integers(0, 131072, size=T)
    pos = pos.astype(np.int64 if ext.get("pos_int64") else np.int32)
    qd = place(q, dtype, layout)
    kd = place(k, dtype, layout)
    td = torch.from_numpy(table).to(DEV) if table is not None else None
    x = binding_rope_ext(tri, ext, td)
    cache.rope(qd, kd, torch.from_numpy(pos).to(DEV), 5e5, x,
               q_w=wl.to_torch(qw, dtype, DEV) if qkn else None,
               k_w=wl.to_torch(kw, dtype, DEV) if qkn else None, eps=1e-6)
    torch.cuda.synchronize()
    wq, wk = O.rope_ext(q, k, pos, 5e5, dtype, q_w=qw if qkn else None, k_w=kw if qkn else None,
                        eps=1e-6, **oracle_rope_kw(ext, table))
    check("q", host(qd), wq, dtype)
    check("k", host(kd), wk, dtype)
    mext = dict(ext, cos_sin=td.data_ptr() if td is not None else None,
                cos_sin_len=300 if td is not None else 0)
    c = S.Call(S.OP_QK_NORM_ROPE if qkn else S.OP_ROPE_QK,
               S.DT_F32 if dtype == nm.F32 else S.DT_BF16, T, hd=hd, nq=nq, nk=nk, base=5e5,
               ptr=dict(q=qd.data_ptr(), k=kd.data_ptr(), pos=0, q_w=0, k_w=0),
               stride=dict(q=qd.stride(0), k=kd.stride(0)), ext=mext)
    assert cache.last_selection().variant == S.plan(S.make_key(c), T)[0]
    if not qkn and rd < hd:          # elements past the rotary span are untouched
        check("q tail", host(qd)[..., rd:], q[..., rd:], dtype, exact=True)


# ---- short ops: silu, add, masked_fill, embedding -------------------------------------------
SHORT_CASES = [
    # op, dtype, T, W, layout
    ("silu", nm.BF16, 1, 11008, "plain"), ("silu", nm.F32, 130, 1000, "plain"),
    ("silu", nm.BF16, 5, 11008, "strided"), ("silu", nm.F32, 5, 1001, "unaligned"),
    ("silu", nm.BF16, 3, 1001, "plain"),
    ("add", nm.BF16, 1, 4096, "plain"), ("add", nm.F32, 100, 4096, "plain"),
    ("add", nm.BF16, 7, 4096, "strided"), ("add", nm.BF16, 7, 1003, "unaligned"),
    ("add", nm.F32, 3, 1001, "plain"),
    ("masked_fill", nm.BF16, 1, 4096, "plain"), ("masked_fill", nm.F32, 130, 1000, "plain"),
    ("masked_fill", nm.BF16, 9, 4096, "strided"), ("masked_fill", nm.F32, 9, 999, "unaligned"),
    ("masked_fill", nm.BF16, 3, 1001, "plain"),
]


@pytest.mark.parametrize("op,dtype,T,W,layout", SHORT_CASES)
def test_short_op_variants(tri, cache, op, dtype, T, W, layout):
    r = rng(T * 17 + W + len(op))
    a = wl.host_array(r, (T, W), dtype, outliers=True)
    b = wl.host_array(r, (T, W), dtype)
    ad, bd = place(a, dtype, layout), place(b, dtype, layout)
    out = empty_like_layout(ad)
    if op == "silu":
        cache.silu(ad, out=out)
        want = O.silu(a, dtype)
    elif op == "add":
        cache.add(ad, bd, out=out)
        want = O.add(a, b, dtype)
    else:
        mask = (r.random((T, W)) < 0.3).astype(np.uint8) * np.uint8(7)
        md = torch.from_numpy(mask).to(DEV)
        if layout == "strided":           # padded mask rows too
            buf = torch.zeros((T, W + 64), dtype=torch.uint8, device=DEV)
            buf[:, :W] = md
            md = buf[:, :W]
        cache.masked_fill(ad, md, float("-inf") if dtype == nm.BF16 else -1e4, out=out)
        want = O.masked_fill(a, mask, float("-inf") if dtype == nm.BF16 else -1e4, dtype)
    torch.cuda.synchronize()
    check(op, host(out), want, dtype, exact=op != "silu")


EMB_CASES = [
    # dtype, T, H, n_rows, int64 ids, layout
    (nm.BF16, 1, 4096, 32000, False, "plain"), (nm.F32, 9, 4096, 1000, True, "plain"),
    (nm.BF16, 70, 1001, 50, False, "plain"), (nm.F32, 5, 4096, 10, False, "strided"),
    (nm.BF16, 6, 4096, 20, True, "unaligned"), (nm.BF16, 300, 128, 7, False, "plain"),
]


@pytest.mark.parametrize("dtype,T,H,n_rows,ids64,layout", EMB_CASES)
def test_embedding_variants(tri, cache, dtype, T, H, n_rows, ids64, layout):
    r = rng(T + H + n_rows)
    table = wl.host_array(r, (n_rows, H), dtype)
    ids = r.integers(-2, n_rows + 2, size=T)           # some out of range on both sides
    if ids64:
        ids[0] = 1 << 40
    ids = ids.astype(np.int64 if ids64 else np.int32)
    td = place(table, dtype, layout)
    out = place(np.zeros((T, H), dtype=table.dtype), dtype, layout)
    cache.embedding(td, torch.from_numpy(ids).to(DEV), out=out)
    torch.cuda.synchronize()
    check("embedding", host(out), O.embedding(table, ids, dtype), dtype, exact=True)


# ---- SwiGLU: every variant ---------------------------------------------------------------
SW_CASES = [
    # dtype, T, I, layout
    (nm.BF16, 1, 11008, "plain"), (nm.BF16, 8, 14336, "plain"), (nm.BF16, 300, 688, "plain"),
    (nm.F32, 4, 688, "plain"), (nm.F32, 130, 1000, "plain"), (nm.F32, 3, 11003, "plain"),
    (nm.BF16, 3, 11003, "plain"), (nm.BF16, 1, 5, "plain"), (nm.F32, 1, 1, "plain"),
    (nm.BF16, 5, 11008, "strided"), (nm.F32, 5, 11008, "strided"),
    (nm.BF16, 5, 11008, "unaligned"), (nm.F32, 5, 1001, "unaligned"),
]


@pytest.mark.parametrize("dtype,T,I,layout", SW_CASES)
def test_swiglu_variants(tri, cache, dtype, T, I, layout):
    r = rng(T * 3 + I)
    g = wl.host_array(r, (T, I), dtype)
    u = wl.host_array(r, (T, I), dtype)
    gd, ud = place(g, dtype, layout), place(u, dtype, layout)
    od = empty_like_layout(gd)
    cache.swiglu(gd, ud, out=od)
    torch.cuda.synchronize()
    check("out", host(od), O.swiglu(g, u, dtype), dtype)


@pytest.mark.parametrize("dtype", [nm.F32, nm.BF16])
def test_swiglu_extremes(tri, cache, dtype):
    g = np.array([[0.0, 1.0, -1.0, 88.0, -88.0, 200.0, -200.0, 3.0] * 4], np.float32)
    u = np.array([[5.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 0.0] * 4], np.float32)
    if dtype == nm.BF16:
        g, u = nm.round_to(g, nm.BF16), nm.round_to(u, nm.BF16)
    gd, ud = wl.to_torch(g, dtype, DEV), wl.to_torch(u, dtype, DEV)
    od = cache.swiglu(gd, ud)
    torch.cuda.synchronize()
    got = host(od)
    check("out", got, O.swiglu(g, u, dtype), dtype)
    v = nm.values(got, dtype)
    assert not np.isnan(v).any()
    assert v[0, 6] == 0.0 and np.signbit(v[0, 6])


def test_swiglu_in_place(tri, cache):
    r = rng(5)
    g = wl.host_array(r, (4, 11008), nm.BF16)
    u = wl.host_array(r, (4, 11008), nm.BF16)
    gd, ud = wl.to_torch(g, nm.BF16, DEV), wl.to_torch(u, nm.BF16, DEV)
    cache.swiglu(gd, ud, out=gd)
    torch.cuda.synchronize()
    check("out", host(gd), O.swiglu(g, u, nm.BF16), nm.BF16)


MEDIUM = [wl.ChainConfig("medium_bf16", wl.BF16, T=100, H=4096, nq=32, nk=8, hd=128, I=11008,
                         base=500000.0, pos_mode="uniform", pos_max=8191),
          wl.ChainConfig("medium_f32", wl.F32, T=70, H=256, nq=4, nk=4, hd=64, I=690,
                         pos_mode="uniform", pos_max=4095),
          wl.ChainConfig("ragged_bf16", wl.BF16, T=65, H=2048, nq=7, nk=3, hd=64, I=1001,
                         pos_mode="uniform", pos_max=100000),
          wl.ChainConfig("medium_qkn_bf16", wl.BF16, T=100, H=4096, nq=32, nk=8, hd=128,
                         I=12288, base=1e6, pos_mode="uniform", pos_max=8191, qk_norm=True),
          wl.ChainConfig("ragged_qkn_f32", wl.F32, T=67, H=512, nq=5, nk=3, hd=128, I=1001,
                         base=1e6, pos_mode="uniform", pos_max=100000, qk_norm=True),
          wl.ChainConfig("medium_gptj_bf16", wl.BF16, T=100, H=4096, nq=16, nk=16, hd=256,
                         I=16384, pos_mode="uniform", pos_max=2047,
                         rope=(("rotary_dim", 64), ("interleaved", 1))),
          wl.ChainConfig("medium_llama31_qkn_bf16", wl.BF16, T=90, H=4096, nq=32, nk=8, hd=128,
                         I=14336, base=5e5, pos_mode="uniform", pos_max=131071, qk_norm=True,
                         rope=wl.LLAMA3_SCALING + (("interleaved", 1),)),
          # few heads per token: four tokens per RoPE workgroup, ragged last block
          wl.ChainConfig("tp8_shard_bf16", wl.BF16, T=301, H=8192, nq=8, nk=1, hd=128, I=3584,
                         base=5e5, pos_mode="uniform", pos_max=8191, outliers=True),
          wl.ChainConfig("tp8_shard_qkn_f32", wl.F32, T=130, H=1024, nq=4, nk=1, hd=128, I=704,
                         base=1e6, pos_mode="uniform", pos_max=8191, qk_norm=True)]


@pytest.mark.parametrize("cfg", MEDIUM, ids=lambda c: c.name)
def test_chain_beyond_decode_sizes(tri, cache, cfg):
    """Fused chain with the workgroup-per-row norm role and the streaming
    4-vector SwiGLU role (ragged tails included)."""
    inp = wl.host_inputs(cfg)
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    d["y"], d["res_out"], d["out"] = (torch.empty_like(d["x"]), torch.empty_like(d["x"]),
                                      torch.empty_like(d["gate"]))
    run_chain(cache, cfg, d)
    torch.cuda.synchronize()
    want = chain_oracle(inp, cfg)
    for n in ("y", "q", "k", "out"):
        check(n, host(d[n]), want[n], cfg.dtype)
    check("res_out", host(d["res_out"]), want["res_out"], cfg.dtype, exact=True)
    rec = cache.last_selection().as_tuple()
    assert rec == expected_record(model_chain_call(d, cfg.eps, cfg.base, ext=cfg.rope_ext), 0)


# ---- several chains per entry call ---------------------------------------------------------
def test_chain_layers_run_in_order(tri, cache):
    """Six layers where layer l + 1 adds layer l's residual output: the result
    is only right if the launches run in layer order. One layer is unaligned
    (three launches) and one is empty."""
    cfg = wl.GQA_DECODE
    n = 6
    host_layers, dev_layers, args = [], [], []
    prev_ro = None
    for l in range(n):
        inp = wl.host_inputs(cfg, seed=100 + l)
        layout = "unaligned" if l == 3 else "plain"
        d = {k: place(v, cfg.dtype, layout) if k not in ("w", "pos") else
             wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
        d["y"], d["res_out"], d["out"] = (empty_like_layout(d["x"]), empty_like_layout(d["x"]),
                                          empty_like_layout(d["gate"]))
        if prev_ro is not None:
            d["residual"] = prev_ro                     # consumes the previous layer
        a, _ = cache.chain_args(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                d["gate"], d["up"], cfg.eps, cfg.base, y=d["y"],
                                residual_out=d["res_out"], out=d["out"])
        if l == 4:
            a.T = 0                                     # an empty layer is skipped
        host_layers.append(inp)
        dev_layers.append(d)
        args.append(a)
        prev_ro = d["res_out"]
    cache.decode_chain_layers(args)
    torch.cuda.synchronize()
    rec = cache.last_selection()
    assert rec.op == 7 and rec.n_launches == 1 + 1 + 1 + 3 + 1
    res = None
    for l in range(n):
        inp = dict(host_layers[l])
        if res is not None:
            inp["residual"] = res
        if l == 4:                                      # skipped: outputs untouched, so
            res = np.zeros_like(inp["x"])               # layer 5 reads a zero residual
            continue
        want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
        d = dev_layers[l]
        check(f"res_out[{l}]", host(d["res_out"]), want["res_out"], cfg.dtype, exact=True)
        for nme in ("y", "q", "k", "out"):
            check(f"{nme}[{l}]", host(d[nme]), want[nme], cfg.dtype)
        res = want["res_out"]
    # layer 5 consumed layer 4's residual output, which was never written
    assert host(dev_layers[4]["res_out"]).view(np.uint16).max() == 0


def test_graph_of_layers_replays_match_direct_calls(tri, cache):
    """A captured step of four dependent layers (one three-launch layer),
    replayed three times with new input data between replays (same
    pointers): every replay equals a direct tri_decode_chain_layers call on
    the same data, bit for bit, and the oracle within tolerance."""
    cfg = wl.GQA_DECODE
    n = 4

    def make(seed_base):
        layers, args = [], []
        prev = None
        for l in range(n):
            inp = wl.host_inputs(cfg, seed=seed_base + l)
            layout = "unaligned" if l == 2 else "plain"
            d = {k: place(v, cfg.dtype, layout) if k not in ("w", "pos") else
                 wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
            d["y"], d["res_out"], d["out"] = (empty_like_layout(d["x"]),
                                              empty_like_layout(d["x"]),
                                              empty_like_layout(d["gate"]))
            if prev is not None:
                d["residual"] = prev
            a, _ = cache.chain_args(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                    d["gate"], d["up"], cfg.eps, cfg.base, y=d["y"],
                                    residual_out=d["res_out"], out=d["out"])
            layers.append((inp, d))
            args.append(a)
            prev = d["res_out"]
        return layers, args

    gl, gargs = make(200)            # buffers the graph is built on
    dl, dargs = make(200)            # twin buffers for direct calls
    graph = cache.build_graph(gargs)
    # layer 2 is unaligned, and so is layer 3, whose residual is layer 2's output
    assert graph.launch_count == 1 + 1 + 3 + 3
    try:
        for rep in range(3):
            # new data, same pointers: refill layer inputs of both twins
            for l in range(n):
                fresh = wl.host_inputs(cfg, seed=300 + 10 * rep + l)
                for k in ("x", "q", "k", "gate", "up") + (("residual",) if l == 0 else ()):
                    src = wl.to_torch(fresh[k], cfg.dtype, DEV)
                    gl[l][1][k].copy_(src)
                    dl[l][1][k].copy_(src)
            torch.cuda.synchronize()
            graph.launch()
            cache.decode_chain_layers(dargs)
            torch.cuda.synchronize()
            for l in range(n):
                for nme in ("y", "res_out", "out", "q", "k"):
                    check(f"rep{rep} {nme}[{l}]", host(gl[l][1][nme]), host(dl[l][1][nme]),
                          cfg.dtype, exact=True)
            want = O.decode_chain({k: host(v) for k, v in gl[0][1].items()
                                   if k in ("x", "residual", "w", "pos", "gate", "up")}
                                  | {"q": wl.host_inputs(cfg, seed=300 + 10 * rep)["q"],
                                     "k": wl.host_inputs(cfg, seed=300 + 10 * rep)["k"]},
                                  cfg.eps, cfg.base, cfg.dtype)
            check(f"rep{rep} out[0] vs oracle", host(gl[0][1]["out"]), want["out"], cfg.dtype)
            check(f"rep{rep} q[0] vs oracle", host(gl[0][1]["q"]), want["q"], cfg.dtype)
    finally:
        torch.cuda.synchronize()
        graph.close()


# ---- chain layouts, degenerate calls, miss path ----------------------------------------------
@pytest.mark.parametrize("layout", ["strided", "unaligned"])
def test_chain_three_launch_variant(tri, cache, layout):
    cfg = wl.GQA_DECODE
    inp = wl.host_inputs(cfg)
    d = {k: place(v, cfg.dtype, layout) if k not in ("w", "pos") else
         wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    d["y"], d["res_out"], d["out"] = (empty_like_layout(d["x"]), empty_like_layout(d["x"]),
                                      empty_like_layout(d["gate"]))
    cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"], d["gate"],
                       d["up"], cfg.eps, cfg.base, y=d["y"], residual_out=d["res_out"],
                       out=d["out"])
    torch.cuda.synchronize()
    want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
    for n in ("y", "q", "k", "out"):
        check(n, host(d[n]), want[n], cfg.dtype)
    check("res_out", host(d["res_out"]), want["res_out"], cfg.dtype, exact=True)
    rec = cache.last_selection().as_tuple()
    assert rec == expected_record(model_chain_call(d, cfg.eps, cfg.base), 0)
    assert rec[3] == S.CH_SEQ and rec[4] == 3


def test_empty_calls_launch_nothing(tri, cache):
    x = torch.zeros((0, 4096), dtype=torch.bfloat16, device=DEV)
    w = torch.ones(4096, dtype=torch.bfloat16, device=DEV)
    cache.rmsnorm(x, w)
    g = torch.zeros((0, 128), dtype=torch.float32, device=DEV)
    cache.swiglu(g, g)
    s = cache.stats()
    assert s["empty"] == 2 and s["n_versions"] == 0 and s["errors"] == 0


def test_miss_then_hit_and_stats(tri, cache):
    r = rng(1)
    x = wl.to_torch(wl.host_array(r, (2, 4096), nm.BF16), nm.BF16, DEV)
    w = wl.to_torch(wl.host_weight(r, 4096, nm.BF16), nm.BF16, DEV)
    for _ in range(5):
        cache.rmsnorm(x, w)
    torch.cuda.synchronize()
    s = cache.stats()
    assert (s["calls"], s["hits"], s["misses"], s["installs"]) == (6, 5, 1, 1)
    assert cache.version_info(0).hits == 5


def test_empty_kernel_launch(tri, cache):
    for _ in range(10):
        cache.launch_empty()
    torch.cuda.synchronize()


def test_invalid_arguments_raise_and_launch_nothing(tri, cache):
    x = torch.zeros((2, 64), dtype=torch.float32, device=DEV)
    w = torch.ones(64, dtype=torch.float32, device=DEV)
    with pytest.raises(tri.TriError) as e:
        cache.rmsnorm(x, w, eps=float("nan"))
    assert e.value.status == tri.E_INVALID
    assert cache.stats()["n_versions"] == 0


def test_binding_rejects_mismatched_shapes_before_any_call(tri, cache):
    """The C entry points see pointers and strides only; the binding checks
    that every tensor has the shape and dtype the call implies (outputs with
    too few rows, short or strided weights, mismatched operands) and raises
    before calling the library."""
    f32, bf16, i32 = torch.float32, torch.bfloat16, torch.int32
    x = torch.zeros((4, 64), dtype=f32, device=DEV)
    w = torch.ones(64, dtype=f32, device=DEV)
    q = torch.zeros((4, 2, 64), dtype=f32, device=DEV)
    k = torch.zeros((4, 1, 64), dtype=f32, device=DEV)
    pos = torch.zeros(4, dtype=i32, device=DEV)
    bad = [
        lambda: cache.rmsnorm(x, w, out=torch.empty((3, 64), dtype=f32, device=DEV)),
        lambda: cache.rmsnorm(x, torch.ones(32, dtype=f32, device=DEV)),
        lambda: cache.rmsnorm(x, torch.ones(128, dtype=f32, device=DEV)[::2]),
        lambda: cache.rmsnorm(x, w.to(bf16)),
        lambda: cache.rmsnorm(x[0], w),
        lambda: cache.residual_rmsnorm(x, x[:3], w),
        lambda: cache.residual_rmsnorm(x, x, w, residual_out=torch.empty((4, 32), dtype=f32,
                                                                          device=DEV)),
        lambda: cache.swiglu(x, torch.zeros((4, 32), dtype=f32, device=DEV)),
        lambda: cache.swiglu(x, x, out=torch.empty((2, 64), dtype=f32, device=DEV)),
        lambda: cache.add(x, x, out=torch.empty((4, 64), dtype=bf16, device=DEV)),
        lambda: cache.silu(x, out=torch.empty((5, 64), dtype=f32, device=DEV)),
        lambda: cache.masked_fill(x, torch.zeros((4, 32), dtype=torch.uint8, device=DEV), 0.0),
        lambda: cache.embedding(x, pos, out=torch.empty((3, 64), dtype=f32, device=DEV)),
        lambda: cache.rope_qk(q, k, pos[:3]),
        lambda: cache.rope_qk(q, k[:2], pos),
        lambda: cache.rope_qk(q, torch.zeros((4, 1, 32), dtype=f32, device=DEV), pos),
        lambda: cache.rope_qk(q, k, pos.to(torch.int64)),
        lambda: cache.qk_norm_rope(q, k, pos, torch.ones(32, dtype=f32, device=DEV)),
        lambda: cache.decode_chain(x, x, w, q, k, pos, x, x[:2]),
        lambda: cache.decode_chain(x, x, w, q[:2], k[:2], pos[:2], x, x),
    ]
    for i, fn in enumerate(bad):
        with pytest.raises((ValueError, TypeError)):
            fn()
    st = cache.stats()
    assert st["calls"] == 0 and st["n_versions"] == 0


def test_binding_rejects_host_tensors_and_narrow_cos_sin_tables(tri, cache):
    """Every tensor must live on the cache's device (a kernel handed a host
    address would fault), and a cos/sin table must be exactly rotary_dim
    floats wide (a narrower one would be read past its end): the binding
    raises before any native call."""
    f32, i32 = torch.float32, torch.int32
    x = torch.zeros((4, 64), dtype=f32, device=DEV)
    w = torch.ones(64, dtype=f32, device=DEV)
    q = torch.zeros((4, 2, 64), dtype=f32, device=DEV)
    k = torch.zeros((4, 1, 64), dtype=f32, device=DEV)
    pos = torch.zeros(4, dtype=i32, device=DEV)
    m = torch.zeros((4, 64), dtype=torch.uint8, device=DEV)
    cpu = lambda t: t.cpu()                                          # noqa: E731
    narrow = tri.rope_ext(cos_sin=torch.zeros((16, 32), dtype=f32, device=DEV))
    host_tab = tri.rope_ext(cos_sin=torch.zeros((16, 64), dtype=f32))
    bad = [
        lambda: cache.rmsnorm(cpu(x), w),
        lambda: cache.rmsnorm(x, cpu(w)),
        lambda: cache.rmsnorm(x, w, out=cpu(x)),
        lambda: cache.residual_rmsnorm(x, cpu(x), w),
        lambda: cache.swiglu(x, cpu(x)),
        lambda: cache.silu(cpu(x)),
        lambda: cache.add(x, cpu(x)),
        lambda: cache.masked_fill(x, cpu(m), 1.0),
        lambda: cache.embedding(x, cpu(pos)),
        lambda: cache.rope_qk(q, k, cpu(pos)),
        lambda: cache.rope_qk(q, cpu(k), pos),
        lambda: cache.qk_norm_rope(q, k, pos, cpu(w)),
        lambda: cache.rope(q, k, pos, ext=narrow),
        lambda: cache.rope(q, k, pos, ext=host_tab),
        lambda: cache.decode_chain(x, x, w, q, k, cpu(pos), x, x),
        lambda: cache.decode_chain(x, x, w, q, k, pos, x, x, rope=narrow),
    ]
    for i, fn in enumerate(bad):
        with pytest.raises(ValueError):
            fn()
    st = cache.stats()
    assert st["calls"] == 0 and st["n_versions"] == 0


def test_chain_args_keep_their_tensors_alive(tri, cache):
    """A prebuilt argument struct holds bare addresses; it keeps every tensor
    behind them alive (the outputs it allocated included), so a later call
    through it never writes into memory the allocator has handed out again."""
    import gc
    import weakref
    cfg = wl.TINY_F32
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in wl.host_inputs(cfg).items()}
    args, outs = cache.chain_args(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                  d["gate"], d["up"], cfg.eps, cfg.base)
    refs = [weakref.ref(t) for t in list(d.values()) + list(outs)]
    del d, outs
    gc.collect()
    assert all(r() is not None for r in refs)
    cache.decode_chain_args(args)
    torch.cuda.synchronize()
    y, ro, out = (r() for r in refs[-3:])
    inp = {k: wl.from_torch(r()) for k, r in zip(("x", "residual", "w"), refs[:3])}
    wy, wh = O.residual_rmsnorm(inp["x"], inp["residual"], inp["w"], cfg.eps, cfg.dtype)
    check("y", host(y), wy, cfg.dtype)
    check("res_out", host(ro), wh, cfg.dtype, exact=True)
    del args, y, ro, out
    gc.collect()
    assert all(r() is None for r in refs)


# ---- full-size prefill chain, every row --------------------------------------------------
@pytest.mark.parametrize("cfg,grid", [(wl.PREFILL_8K, 8192 + 8192 + 114688),
                                      (wl.PREFILL_8K_TP8, 8192 + 2048 + 14336)],
                         ids=lambda c: c.name if hasattr(c, "name") else str(c))
def test_prefill_chain_full_size_all_rows(tri, cache, cfg, grid):
    """The 8192-token chains in the benchmark's launch configuration; every
    row of every output against the oracle, 512 rows at a time."""
    d = wl.device_inputs(cfg, DEV)
    src = {k: v.clone() for k, v in d.items() if k in ("q", "k")}
    y, ro, out = cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                    d["gate"], d["up"], cfg.eps, cfg.base)
    torch.cuda.synchronize()
    rec = cache.last_selection()
    assert rec.variant == S.CH_FUSED and rec.launch[0].grid_x == grid
    w = host(d["w"])
    for r0 in range(0, cfg.T, 512):
        sl = slice(r0, min(cfg.T, r0 + 512))
        wy, wh = O.residual_rmsnorm(host(d["x"][sl]), host(d["residual"][sl]), w, cfg.eps,
                                    cfg.dtype)
        check(f"y {sl}", host(y[sl]), wy, cfg.dtype)
        check(f"res_out {sl}", host(ro[sl]), wh, cfg.dtype, exact=True)
        wq, wk = O.rope_qk(host(src["q"][sl]), host(src["k"][sl]), host(d["pos"][sl]),
                           cfg.base, cfg.dtype)
        check(f"q {sl}", host(d["q"][sl]), wq, cfg.dtype)
        check(f"k {sl}", host(d["k"][sl]), wk, cfg.dtype)
        check(f"out {sl}", host(out[sl]),
              O.swiglu(host(d["gate"][sl]), host(d["up"][sl]), cfg.dtype), cfg.dtype)


# ---- mixed-shape stream -----------------------------------------------------------------------
def _mixed_stream_on_gpu(tri, cache, model, exact_before=(), exact_at=None, check_every=50):
    """The 10,000-call mixed stream on real buffers: every selection record
    against the model's, outputs against the oracle every `check_every`-th
    call and on every miss. `exact_before` keys are installed exactly before
    the stream, `exact_at` = (call index, keys) installs more midway."""
    Tmax = max(wl.MIXED_T_CHOICES)
    H, I, nq, nk, hd = wl.MIXED_H, wl.MIXED_I, wl.MIXED_NQ, wl.MIXED_NK, wl.MIXED_HD
    bufs = {}
    for k in exact_before:
        cache.install_key(k)
        assert model.install_key(k) == S.OK
    stream = wl.mixed_stream()
    assert len(stream) == wl.MIXED_CALLS
    for n, (T, dt, layout) in enumerate(stream):
        if n % 1000 == 0:
            print(f"mixed stream: call {n}", flush=True)
        if exact_at is not None and n == exact_at[0]:
            for k in exact_at[1]:
                cache.install_key(k)
                assert model.install_key(k) == S.OK
        key = (dt, layout)
        if key not in bufs:
            r = rng(len(bufs) + 1)
            h = dict(x=wl.host_array(r, (Tmax, H), dt), residual=wl.host_array(r, (Tmax, H), dt),
                     q=wl.host_array(r, (Tmax, nq, hd), dt), k=wl.host_array(r, (Tmax, nk, hd), dt),
                     gate=wl.host_array(r, (Tmax, I), dt), up=wl.host_array(r, (Tmax, I), dt))
            dd = {k: place(v, dt, layout, pad=wl.MIXED_PAD) for k, v in h.items()}
            dd["w"] = wl.to_torch(wl.host_weight(r, H, dt), dt, DEV)
            dd["pos"] = torch.from_numpy(
                r.integers(0, wl.MIXED_POS_MAX + 1, Tmax).astype(np.int32)).to(DEV)
            for o, s in (("y", "x"), ("res_out", "x"), ("out", "gate")):
                dd[o] = empty_like_layout(dd[s])
            bufs[key] = (h, dd)
        h, dd = bufs[key]
        d = {k: v[:T] for k, v in dd.items() if k != "w"}
        d["w"] = dd["w"]
        call = model_chain_call(d, 1e-6, wl.MIXED_BASE)
        missed = model.call(call) == S.MISS
        check_out = missed or n % check_every == 0
        if check_out:
            q0, k0 = host(d["q"]), host(d["k"])
        cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"], d["gate"],
                           d["up"], 1e-6, wl.MIXED_BASE, y=d["y"], residual_out=d["res_out"],
                           out=d["out"])
        if missed:
            model.install_last_miss()
            model.call(call)
        assert cache.last_selection().as_tuple() == model.last.as_tuple(), (n, T, dt, layout)
        if check_out:
            torch.cuda.synchronize()
            inp = dict(x=host(d["x"]), residual=host(d["residual"]), w=host(d["w"]), q=q0, k=k0,
                       pos=host(d["pos"]), gate=host(d["gate"]), up=host(d["up"]))
            want = O.decode_chain(inp, 1e-6, wl.MIXED_BASE, dt)
            for nme in ("y", "q", "k", "out"):
                check(f"{n}:{nme}", host(d[nme]), want[nme], dt)
            check(f"{n}:res_out", host(d["res_out"]), want["res_out"], dt, exact=True)
    torch.cuda.synchronize()
    s = cache.stats()
    assert s["misses"] == model.stats.misses and s["n_versions"] == len(model.versions)


def test_mixed_stream_selection_and_outputs(tri, cache):
    """All 10,000 calls of the mixed stream on real buffers: every selection
    record against the oracle's model, outputs against the oracle every 50th
    call (and on every miss)."""
    _mixed_stream_on_gpu(tri, cache, S.SpecCacheModel())


def test_mixed_stream_with_overlapping_generic_versions(tri):
    """The same stream on a cache that installs generic versions on a miss,
    with exact versions installed first for every third distinct key of the
    first 200 calls and, after 5,000 calls, for every other distinct key of
    the stream: versions overlap and the first in creation order runs.
    Records bit for bit against the model on every call; outputs against the
    oracle every 50th call and on every miss."""
    def mk(T, dt, layout):
        d = S.DT_BF16 if dt == wl.BF16 else S.DT_F32
        es = 2 if d == S.DT_BF16 else 4
        off = es if layout == wl.LAYOUT_UNALIGNED else 0
        pad = wl.MIXED_PAD if layout == wl.LAYOUT_STRIDED else 0
        from tests.selection_calls import chain_call
        return S.make_key(chain_call(d, T, wl.MIXED_H, wl.MIXED_I, wl.MIXED_NQ, wl.MIXED_NK,
                                     wl.MIXED_HD, res_off=off, rope_off=off, sw_off=off,
                                     res_pad=pad, rope_pad=pad, sw_pad=pad))
    stream = wl.mixed_stream()
    first, every = [], []
    for i, (T, dt, layout) in enumerate(stream):
        k = mk(T, dt, layout)
        if i < 200 and k not in first:
            first.append(k)
        if k not in every:
            every.append(k)
    flags = S.FLAG_GENERIC
    cache = tri.SpecCache(generic=True)
    try:
        _mixed_stream_on_gpu(tri, cache, S.SpecCacheModel(flags=flags), exact_before=first[::3],
                             exact_at=(5000, every[::2]))
        guards = [(cache.version_info(i).b_lo, cache.version_info(i).b_hi)
                  for i in range(cache.stats()["n_versions"])]
        assert any(b >= 0 for b, _ in guards) and any(b < 0 for b, _ in guards)
    finally:
        torch.cuda.synchronize()
        cache.close()


# ---- HIP graph capture of the hit path ------------------------------------------------------
def test_chain_call_replays_from_a_hip_graph(tri, cache):
    """A hit is one plain kernel launch, so it can be captured in a graph and
    replayed. Replays run with eager work and synchronisations in between and
    each must equal a direct call on a twin set of buffers, bit for bit."""
    cfg = wl.LLAMA7B_DECODE
    inp = wl.host_inputs(cfg)
    A = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    B = {k: v.clone() for k, v in A.items()}
    for d in (A, B):
        d["y"], d["res_out"], d["out"] = (torch.empty_like(d["x"]), torch.empty_like(d["x"]),
                                          torch.empty_like(d["gate"]))
    args_a, _ = cache.chain_args(A["x"], A["residual"], A["w"], A["q"], A["k"], A["pos"],
                                 A["gate"], A["up"], cfg.eps, cfg.base, y=A["y"],
                                 residual_out=A["res_out"], out=A["out"])
    args_b, _ = cache.chain_args(B["x"], B["residual"], B["w"], B["q"], B["k"], B["pos"],
                                 B["gate"], B["up"], cfg.eps, cfg.base, y=B["y"],
                                 residual_out=B["res_out"], out=B["out"])
    cache.decode_chain_args(args_b)            # installs the version (no allocation later)
    torch.cuda.synchronize()
    B["q"].copy_(A["q"])                       # undo B's rotation: both start equal
    B["k"].copy_(A["k"])
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        cache.decode_chain_args(args_a, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    # capture does not run the kernel: A is still untouched
    check("q before replay", host(A["q"]), host(B["q"]), cfg.dtype, exact=True)
    for step in range(4):
        for d in (A, B):                       # the program's own eager work in between
            d["x"].mul_(0.5).add_(0.25)
        torch.cuda.synchronize()
        g.replay()
        cache.decode_chain_args(args_b)
        torch.cuda.synchronize()
        for n in ("y", "res_out", "q", "k", "out"):
            check(f"replay {step}: {n}", host(A[n]), host(B[n]), cfg.dtype, exact=True)


@pytest.mark.parametrize("entry", ["ordinary", "noalloc"])
def test_split_norm_replays_from_a_hip_graph(tri, cache, entry):
    """A split residual norm (bf16 rows of 65536, 4 workgroups per row)
    captured in a graph after its version is installed: the captured launch
    exchanges partial sums through its scratch, which every launch leaves
    zeroed, so the graph needs no clearing node. Four replays, with the
    program's own eager work between them, each equal a direct call on twin
    buffers bit for bit and the oracle within tolerance."""
    print(f"graph replay of a split norm ({entry})", flush=True)
    T, H = 5, 65536
    r = rng(29)
    w = wl.host_weight(r, H, nm.BF16)
    x0, r0 = wl.host_array(r, (T, H), nm.BF16), wl.host_array(r, (T, H), nm.BF16)
    wd = wl.to_torch(w, nm.BF16, DEV)
    A = dict(x=wl.to_torch(x0, nm.BF16, DEV), r=wl.to_torch(r0, nm.BF16, DEV))
    B = {k: v.clone() for k, v in A.items()}
    for d in (A, B):
        d["y"], d["ro"] = torch.empty_like(d["x"]), torch.empty_like(d["x"])
    call = cache.residual_rmsnorm_noalloc if entry == "noalloc" else cache.residual_rmsnorm
    cache.residual_rmsnorm(B["x"], B["r"], wd, 1e-6, out=B["y"], residual_out=B["ro"])
    torch.cuda.synchronize()
    assert cache.last_selection().variant == S.RN_SPLIT
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call(A["x"], A["r"], wd, 1e-6, out=A["y"], residual_out=A["ro"],
             stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for step in range(4):
        for d in (A, B):                       # the program's own eager work in between
            d["x"].mul_(0.5).add_(0.25)
            d["r"].mul_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        cache.residual_rmsnorm(B["x"], B["r"], wd, 1e-6, out=B["y"], residual_out=B["ro"])
        torch.cuda.synchronize()
        for n in ("y", "ro"):
            check(f"replay {step}: {n}", host(A[n]), host(B[n]), nm.BF16, exact=True)
        wy, wh = O.residual_rmsnorm(host(A["x"]), host(A["r"]), w, 1e-6, nm.BF16)
        check(f"replay {step}: y vs oracle", host(A["y"]), wy, nm.BF16)
        check(f"replay {step}: res_out vs oracle", host(A["ro"]), wh, nm.BF16, exact=True)
    del g
    torch.cuda.synchronize()
