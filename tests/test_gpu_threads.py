"""Caches on several host threads (one cache per thread; caches share no
state), and concurrent compilations into one code directory.

Each case prints its name before touching the GPU. Inputs from `workloads`,
expected values from `oracle`.
"""
import threading

import numpy as np
import pytest
import torch

from oracle import ops as O
from tests.parity import check
from tests.test_gpu_parity import host
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


def _run_threads(fn, n):
    errors = []

    def wrap(i):
        try:
            fn(i)
        except BaseException as e:  # noqa: BLE001 - reported below
            errors.append((i, e))
    ts = [threading.Thread(target=wrap, args=(i,)) for i in range(n)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=300)
    assert not any(t.is_alive() for t in ts), "a thread did not finish"
    assert not errors, errors


@pytest.mark.parametrize("resident", [False, True], ids=["kernel_args", "resident"])
def test_one_cache_per_thread(tri, resident):
    """Four threads, each with its own cache, stream and buffers, 200 decode
    chains each (q / k restored before every call); the last results match
    the oracle. With resident argument blocks the caches claim slots of the
    device's shared pools at the same time and each launch finds its own."""
    print(f"threads: one cache per thread (resident={resident})", flush=True)
    cfgs = [wl.LLAMA7B_DECODE, wl.GQA_DECODE, wl.QWEN3_8B_DECODE, wl.TINY_F32]
    results = {}

    def work(i):
        cfg = cfgs[i]
        inp = wl.host_inputs(cfg, seed=100 + i)
        stream = torch.cuda.Stream(device=DEV)
        cache = tri.SpecCache(auto_install=True, resident_args=resident)
        try:
            with torch.cuda.stream(stream):
                d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
                q0, k0 = d["q"].clone(), d["k"].clone()
                y = torch.empty_like(d["x"])
                ro = torch.empty_like(d["x"])
                out = torch.empty_like(d["gate"])
            for _ in range(200):
                with torch.cuda.stream(stream):
                    d["q"].copy_(q0)
                    d["k"].copy_(k0)
                cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                   d["gate"], d["up"], cfg.eps, cfg.base, y=y, residual_out=ro,
                                   out=out, q_norm_w=d.get("q_norm_w"),
                                   k_norm_w=d.get("k_norm_w"), stream=stream)
            stream.synchronize()
            st = cache.stats()
            assert (st["hits"], st["misses"], st["n_versions"]) == (199, 1, 1)
            if resident:
                assert cache.resident_info() == {"enabled": 1, "held": 1, "launches": 200}
            results[i] = (inp, dict(y=host(y), res_out=host(ro), out=host(out),
                                    q=host(d["q"]), k=host(d["k"])))
        finally:
            torch.cuda.synchronize()
            cache.close()
    _run_threads(work, len(cfgs))
    for i, cfg in enumerate(cfgs):
        inp, got = results[i]
        want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
        for n in ("y", "out", "q", "k"):
            check(f"{cfg.name} {n}", got[n], want[n], cfg.dtype)
        check(f"{cfg.name} res_out", got["res_out"], want["res_out"], cfg.dtype, exact=True)


def test_concurrent_compiles_into_one_code_directory(tri, tmp_path):
    """Three threads compile the same specialization into one code directory
    at once; a fourth cache then loads the stored object, which computes
    exactly what the precompiled kernel computes."""
    print("threads: concurrent compiles, one code directory", flush=True)
    cfg = wl.LLAMA7B_DECODE
    inp = wl.host_inputs(cfg)
    barrier = threading.Barrier(3)

    def work(i):
        d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
        cache = tri.SpecCache(auto_install=True, jit=True, code_dir=str(tmp_path))
        try:
            barrier.wait(timeout=120)
            cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                               d["gate"], d["up"], cfg.eps, cfg.base)
            torch.cuda.synchronize()
            assert cache.version_info(0).jit in (1, 2)
        finally:
            torch.cuda.synchronize()
            cache.close()
    _run_threads(work, 3)
    files = sorted(p.name for p in tmp_path.iterdir())
    assert len(files) == 1 and files[0].endswith(".co"), files     # no temporary left behind
    a = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    b = {k: v.clone() for k, v in a.items()}
    loaded = tri.SpecCache(auto_install=True, jit=True, code_dir=str(tmp_path))
    pre = tri.SpecCache(auto_install=True)
    try:
        oj = loaded.decode_chain(a["x"], a["residual"], a["w"], a["q"], a["k"], a["pos"],
                                 a["gate"], a["up"], cfg.eps, cfg.base)
        op = pre.decode_chain(b["x"], b["residual"], b["w"], b["q"], b["k"], b["pos"],
                              b["gate"], b["up"], cfg.eps, cfg.base)
        torch.cuda.synchronize()
        assert loaded.version_info(0).jit == 2
        for n, g, h in (("y", oj[0], op[0]), ("res_out", oj[1], op[1]), ("out", oj[2], op[2]),
                        ("q", a["q"], b["q"]), ("k", a["k"], b["k"])):
            check(n, host(g), host(h), cfg.dtype, exact=True)
    finally:
        torch.cuda.synchronize()
        loaded.close()
        pre.close()
