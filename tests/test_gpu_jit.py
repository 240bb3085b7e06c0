"""GPU: runtime-compiled specializations (TRI_CACHE_JIT) against the
precompiled kernels and the CPU oracle.

A specialization runs the same device body with the key's shape fields
fixed at compile time, so on identical inputs it must produce the
precompiled kernel's output bit for bit. Every output of every case is also
compared with the CPU oracle on its own (at the usual tolerance, bit for bit
where the op is exact), so a specialization is never checked only against
another HIP path. Every case prints its name (pytest -v) before touching
the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from oracle import selection as S
from tests.parity import binding_rope_ext, check, oracle_rope_kw
from tests.test_gpu_parity import CHAIN_CFGS, MEDIUM, place, empty_like_layout, host, rng
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


def _chain(tri, cache, cfg, d):
    rope = binding_rope_ext(tri, cfg.rope_ext) if cfg.rope_ext else None
    return cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                              d["gate"], d["up"], cfg.eps, cfg.base,
                              q_norm_w=d.get("q_norm_w"), k_norm_w=d.get("k_norm_w"),
                              rope=rope)


@pytest.mark.parametrize("cfg", CHAIN_CFGS + MEDIUM, ids=lambda c: c.name)
def test_jit_chain_equals_precompiled_bitwise(tri, cfg):
    inp = wl.host_inputs(cfg)
    a = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    b = {k: v.clone() for k, v in a.items()}
    pre, jit = tri.SpecCache(), tri.SpecCache(jit=True)
    try:
        outs_p = _chain(tri, pre, cfg, a)
        outs_j = _chain(tri, jit, cfg, b)
        torch.cuda.synchronize()
        assert jit.last_selection().as_tuple()[2:] == pre.last_selection().as_tuple()[2:]
        info = jit.version_info(0)
        assert info.jit == 1 and info.build_ms > 0 and pre.version_info(0).jit == 0
        for n, g, h in (("y", outs_j[0], outs_p[0]), ("res_out", outs_j[1], outs_p[1]),
                        ("out", outs_j[2], outs_p[2]), ("q", b["q"], a["q"]),
                        ("k", b["k"], a["k"])):
            check(n, host(g), host(h), cfg.dtype, exact=True)
        want = O.decode_chain(dict(inp, rope_ext=oracle_rope_kw(cfg.rope_ext))
                              if cfg.rope_ext else inp, cfg.eps, cfg.base, cfg.dtype)
        for n, g in (("y", outs_j[0]), ("res_out", outs_j[1]), ("out", outs_j[2]),
                     ("q", b["q"]), ("k", b["k"])):
            check(f"{n} vs oracle", host(g), want[n], cfg.dtype, exact=n == "res_out")
    finally:
        torch.cuda.synchronize()
        pre.close()
        jit.close()


# Standalone ops through a JIT cache: the scalar, loop, wide (1024-lane) and
# vector forms.
OP_CASES = [
    ("rmsnorm", nm.BF16, 5, 4096, "plain"), ("rmsnorm", nm.F32, 3, 65536, "plain"),
    ("rmsnorm", nm.BF16, 3, 65536, "plain"), ("residual", nm.F32, 4, 20480, "plain"),
    ("residual", nm.BF16, 2, 40960, "strided"),
    ("rmsnorm", nm.BF16, 7, 4097, "plain"), ("rmsnorm", nm.F32, 9, 520, "unaligned"),
    # plain rows of 5120 vectors on 256 workgroups that take 1-2 rows each
    ("rmsnorm", nm.BF16, 300, 40960, "plain"),
    ("residual", nm.BF16, 130, 4096, "plain"), ("residual", nm.F32, 6, 256, "strided"),
    ("swiglu", nm.BF16, 8, 14336, "plain"), ("swiglu", nm.F32, 130, 1000, "plain"),
    ("swiglu", nm.BF16, 5, 11008, "strided"), ("swiglu", nm.F32, 5, 1001, "unaligned"),
    ("silu", nm.BF16, 130, 4096, "plain"), ("add", nm.F32, 7, 1001, "unaligned"),
    ("masked_fill", nm.BF16, 9, 4096, "strided"), ("embedding", nm.BF16, 9, 4096, "plain"),
    ("embedding", nm.F32, 9, 1001, "plain"),
]


@pytest.mark.parametrize("op,dtype,T,W,layout", OP_CASES)
def test_jit_ops_equal_precompiled_bitwise(tri, op, dtype, T, W, layout):
    r = rng(T * 31 + W)
    x = wl.host_array(r, (T, W), dtype)
    x2 = wl.host_array(r, (T, W), dtype)
    w = wl.host_weight(r, W, dtype)
    mask = (np.arange(T * W) % 3 == 0).astype(np.uint8).reshape(T, W)
    ids = (np.arange(T) * 3 - 2).astype(np.int32)        # id -2 and ids past T: zero rows
    pre, jit = tri.SpecCache(), tri.SpecCache(jit=True)
    try:
        outs = []
        for cache in (pre, jit):
            xd, x2d, wd = place(x, dtype, layout), place(x2, dtype, layout), wl.to_torch(w, dtype, DEV)
            y = empty_like_layout(xd)
            if op == "rmsnorm":
                cache.rmsnorm(xd, wd, 1e-6, out=y)
                outs.append((y,))
            elif op == "residual":
                ro = empty_like_layout(xd)
                cache.residual_rmsnorm(xd, x2d, wd, 1e-6, out=y, residual_out=ro)
                outs.append((y, ro))
            elif op == "silu":
                outs.append((cache.silu(xd, out=y),))
            elif op == "add":
                outs.append((cache.add(xd, x2d, out=y),))
            elif op == "masked_fill":
                outs.append((cache.masked_fill(xd, torch.from_numpy(mask).to(DEV), -5.5,
                                               out=y),))
            elif op == "embedding":
                outs.append((cache.embedding(xd, torch.from_numpy(ids).to(DEV)),))
            else:
                cache.swiglu(xd, x2d, out=y)
                outs.append((y,))
        torch.cuda.synchronize()
        assert jit.version_info(0).jit == 1
        for g, h in zip(outs[1], outs[0]):
            check(op, host(g), host(h), dtype, exact=True)
        if op == "rmsnorm":
            want = (O.rmsnorm(x, w, 1e-6, dtype),)
        elif op == "residual":
            want = O.residual_rmsnorm(x, x2, w, 1e-6, dtype)
        elif op == "silu":
            want = (O.silu(x, dtype),)
        elif op == "add":
            want = (O.add(x, x2, dtype),)
        elif op == "masked_fill":
            want = (O.masked_fill(x, mask, -5.5, dtype),)
        elif op == "embedding":
            want = (O.embedding(x, ids, dtype),)
        else:
            want = (O.swiglu(x, x2, dtype),)
        exact = {"residual": (False, True), "add": (True,), "masked_fill": (True,),
                 "embedding": (True,)}.get(op, (False,))
        for i, (g, e) in enumerate(zip(want, exact)):
            check(f"{op}[{i}] vs oracle", host(outs[1][i]), g, dtype, exact=e)
    finally:
        torch.cuda.synchronize()
        pre.close()
        jit.close()


RANGE_CASES = [
    # dtype, T, nq, nk, hd, variant, QK norm, layout
    (nm.BF16, 5, 8, 2, 128, {}, False, "plain"),
    (nm.BF16, 5, 8, 2, 96, {}, False, "plain"),
    (nm.F32, 6, 8, 2, 128, dict(interleaved=1, rotary_dim=64, pos_int64=1), False, "plain"),
    (nm.BF16, 5, 32, 8, 128, {}, True, "plain"),
    (nm.BF16, 5, 8, 2, 128, dict(rotary_dim=64), True, "plain"),
    (nm.F32, 4, 300, 20, 64, dict(interleaved=1), True, "unaligned"),
    (nm.BF16, 6, 8, 2, 128, dict(cache=1, interleaved=1), False, "plain"),
]


@pytest.mark.parametrize("dtype,T,nq,nk,hd,ext,qkn,layout", RANGE_CASES)
def test_jit_rope_equals_precompiled_bitwise(tri, dtype, T, nq, nk, hd, ext, qkn, layout):
    r = rng(T * 13 + nq + hd)
    q = wl.host_array(r, (T, nq, hd), dtype)
    k = wl.host_array(r, (T, nk, hd), dtype)
    qw, kw = wl.host_weight(r, hd, dtype), wl.host_weight(r, hd, dtype)
    ext = dict(ext)
    rd = ext.get("rotary_dim") or hd
    table = None
    if ext.pop("cache", 0):
        table = wl.cos_sin_table(r, 64, rd)
        pos = r.integers(-3, 70, size=T)
    else:
        pos = r.integers(0, 1 << 20, size=T)
    pos = torch.from_numpy(pos.astype(np.int64 if ext.get("pos_int64") else np.int32)).to(DEV)
    td = torch.from_numpy(table).to(DEV) if table is not None else None
    pre, jit = tri.SpecCache(), tri.SpecCache(jit=True)
    try:
        res = []
        for cache in (pre, jit):
            qd, kd = place(q, dtype, layout), place(k, dtype, layout)
            cache.rope(qd, kd, pos, 5e5, binding_rope_ext(tri, ext, td),
                       q_w=wl.to_torch(qw, dtype, DEV) if qkn else None,
                       k_w=wl.to_torch(kw, dtype, DEV) if qkn else None)
            res.append((qd, kd))
        torch.cuda.synchronize()
        assert jit.version_info(0).jit == 1
        check("q", host(res[1][0]), host(res[0][0]), dtype, exact=True)
        check("k", host(res[1][1]), host(res[0][1]), dtype, exact=True)
        wq, wk = O.rope_ext(q, k, host(pos), 5e5, dtype, q_w=qw if qkn else None,
                            k_w=kw if qkn else None, eps=1e-6, **oracle_rope_kw(ext, table))
        check("q vs oracle", host(res[1][0]), wq, dtype)
        check("k vs oracle", host(res[1][1]), wk, dtype)
    finally:
        torch.cuda.synchronize()
        pre.close()
        jit.close()


def test_prewarmed_jit_cache_has_no_misses(tri):
    """Export the keys of a cache, import them into a JIT cache: the same calls
    then hit without a single miss."""
    cfgs = [wl.LLAMA7B_DECODE, wl.QWEN3_8B_DECODE, wl.GPTJ_DECODE]
    inputs = [{k: wl.to_torch(v, c.dtype, DEV) for k, v in wl.host_inputs(c).items()}
              for c in cfgs]
    src = tri.SpecCache()
    dst = tri.SpecCache(jit=True)
    try:
        for c, d in zip(cfgs, inputs):
            _chain(tri, src, c, {k: v.clone() for k, v in d.items()})
        keys = src.export_keys()
        assert len(keys) == len(cfgs)
        assert dst.import_keys(keys) == len(keys)
        for c, d in zip(cfgs, inputs):
            _chain(tri, dst, c, {k: v.clone() for k, v in d.items()})
        torch.cuda.synchronize()
        st = dst.stats()
        assert st["misses"] == 0 and st["hits"] == len(cfgs) and st["installs"] == len(cfgs)
        assert all(dst.version_info(i).jit == 1 for i in range(len(cfgs)))
    finally:
        torch.cuda.synchronize()
        src.close()
        dst.close()


def test_code_directory_loads_compiled_kernels(tri, tmp_path):
    """A second JIT cache on the same code directory loads the compiled
    kernels instead of compiling them, and they compute the same bits."""
    cfg = wl.GQA_DECODE
    inp = wl.host_inputs(cfg)
    outs, infos = [], []
    for _ in range(2):
        d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
        c = tri.SpecCache(jit=True, code_dir=str(tmp_path))
        try:
            y, ro, out = _chain(tri, c, cfg, d)
            torch.cuda.synchronize()
            outs.append([host(t) for t in (y, ro, out, d["q"], d["k"])])
            infos.append((c.version_info(0).jit, c.version_info(0).build_ms))
        finally:
            torch.cuda.synchronize()
            c.close()
    assert infos[0][0] == 1 and infos[1][0] == 2
    assert infos[1][1] < infos[0][1]
    assert len(list(tmp_path.iterdir())) == 1
    for a, b in zip(*outs):
        check("loaded == compiled", a, b, cfg.dtype, exact=True)


def test_jit_generic_versions(tri):
    """A compiling cache that installs generic versions: one compiled chain
    specialization serves the Llama-7B chain at 1-64 tokens (its run of
    buckets: the key's shape fields are compiled in, the tokens stay a
    run-time argument), and a norm version with a row-length range runs
    the precompiled kernel (a compiled one would fix H); every output
    against the oracle."""
    r = rng(23)
    dt, H, I, nq, nk, hd, base, eps = nm.BF16, 4096, 11008, 32, 32, 128, 1e4, 1e-6
    w = wl.host_weight(r, H, dt)
    wd = wl.to_torch(w, dt, DEV)
    c = tri.SpecCache(auto_install=True, jit=True, generic=True)
    try:
        for T in (3, 1, 50, 64):
            print(f"jit generic chain: T={T}", flush=True)
            h = dict(x=wl.host_array(r, (T, H), dt), residual=wl.host_array(r, (T, H), dt),
                     q=wl.host_array(r, (T, nq, hd), dt), k=wl.host_array(r, (T, nk, hd), dt),
                     gate=wl.host_array(r, (T, I), dt), up=wl.host_array(r, (T, I), dt))
            pos = r.integers(0, 4096, T).astype(np.int32)
            d = {k: wl.to_torch(v, dt, DEV) for k, v in h.items()}
            y, ro, out = c.decode_chain(d["x"], d["residual"], wd, d["q"], d["k"],
                                        torch.from_numpy(pos).to(DEV), d["gate"], d["up"],
                                        eps, base)
            torch.cuda.synchronize()
            want = O.decode_chain(dict(h, w=w, pos=pos), eps, base, dt)
            for n, g in (("y", y), ("out", out), ("q", d["q"]), ("k", d["k"])):
                check(f"T={T} {n}", host(g), want[n], dt)
            check(f"T={T} res_out", host(ro), want["res_out"], dt, exact=True)
        st = c.stats()
        assert st["n_versions"] == 1 and st["misses"] == 1
        v = c.version_info(0)
        assert v.jit == 1 and (v.b_lo, v.b_hi) == (0, 6)
        for T, Hn in ((5, 4000), (9, 3000)):             # 257..512 vectors: one kernel class
            print(f"jit generic rmsnorm: T={T} H={Hn}", flush=True)
            x = wl.host_array(r, (T, Hn), dt)
            wn = wl.host_weight(r, Hn, dt)
            y = c.rmsnorm(wl.to_torch(x, dt, DEV), wl.to_torch(wn, dt, DEV), eps)
            torch.cuda.synchronize()
            check(f"rmsnorm T={T} H={Hn}", host(y), O.rmsnorm(x, wn, eps, dt), dt)
        st = c.stats()
        assert st["n_versions"] == 2 and st["misses"] == 2
        v = c.version_info(1)
        assert v.jit == 0 and (v.h_lo, v.h_hi) == (2056, 4096)
    finally:
        torch.cuda.synchronize()
        c.close()
