"""Parity report: for every chain configuration of the parity tests, and
every row of the 8192-token prefill chains, the largest absolute and
relative error, the largest ulp distance from the oracle's correctly rounded
value and the fraction of bit-exact elements, per output. Every output is
also held to the tolerance (`tests.parity.check`).

With TRI_PARITY_REPORT=<path> the table is written there as markdown.
Inputs from `workloads`; expected values only from `oracle`. Each
configuration prints its name before touching the GPU.
"""
import os

import numpy as np
import pytest
import torch

from oracle import ops as O
from tests.parity import check, error_stats
from tests.test_gpu_parity import CHAIN_CFGS, MEDIUM, chain_oracle, host, run_chain
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
OUTPUTS = ("y", "res_out", "q", "k", "out")


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


def _chain_rows(tri, cfg):
    print(f"report: {cfg.name}", flush=True)
    inp = wl.host_inputs(cfg)
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    d["y"], d["res_out"], d["out"] = (torch.empty_like(d["x"]), torch.empty_like(d["x"]),
                                      torch.empty_like(d["gate"]))
    cache = tri.SpecCache(auto_install=True)
    try:
        run_chain(cache, cfg, d)
        torch.cuda.synchronize()
    finally:
        cache.close()
    want = chain_oracle(inp, cfg)
    return cfg, {n: (host(d[n]), want[n]) for n in OUTPUTS}


def _prefill_rows(tri, cfg):
    """Every row of the 8192-token chain, compared 512 rows at a time; the
    statistics of the chunks are merged (largest errors, element-weighted
    bit-exact fraction)."""
    print(f"report: {cfg.name} (every row)", flush=True)
    d = wl.device_inputs(cfg, DEV)
    q0, k0 = d["q"].clone(), d["k"].clone()
    cache = tri.SpecCache(auto_install=True)
    try:
        y, ro, out = cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                        d["gate"], d["up"], cfg.eps, cfg.base)
        torch.cuda.synchronize()
    finally:
        cache.close()
    w = host(d["w"])
    stats = {n: [] for n in OUTPUTS}
    for r0 in range(0, cfg.T, 512):
        sl = slice(r0, min(cfg.T, r0 + 512))
        wy, wh = O.residual_rmsnorm(host(d["x"][sl]), host(d["residual"][sl]), w, cfg.eps,
                                    cfg.dtype)
        wq, wk = O.rope_qk(host(q0[sl]), host(k0[sl]), host(d["pos"][sl]), cfg.base, cfg.dtype)
        wo = O.swiglu(host(d["gate"][sl]), host(d["up"][sl]), cfg.dtype)
        got = {"y": y[sl], "res_out": ro[sl], "q": d["q"][sl], "k": d["k"][sl], "out": out[sl]}
        want = {"y": wy, "res_out": wh, "q": wq, "k": wk, "out": wo}
        for n in OUTPUTS:
            g = host(got[n])
            check(f"{cfg.name} {n} {sl}", g, want[n], cfg.dtype, exact=n == "res_out")
            stats[n].append(error_stats(g, want[n], cfg.dtype))
    del d, q0, k0, y, ro, out
    torch.cuda.synchronize()
    return cfg, {n: merge_stats(stats[n]) for n in OUTPUTS}


def merge_stats(parts):
    n = sum(p["n"] for p in parts)
    return {"n": n, "max_abs": max(p["max_abs"] for p in parts),
            "max_rel": max(p["max_rel"] for p in parts),
            "max_ulp": max(p["max_ulp"] for p in parts),
            "exact": sum(p["exact"] * p["n"] for p in parts) / max(n, 1)}


def test_parity_report(tri):
    runs = [_chain_rows(tri, c) for c in CHAIN_CFGS + MEDIUM]
    runs += [_prefill_rows(tri, c) for c in (wl.PREFILL_8K, wl.PREFILL_8K_TP8)]
    lines = ["| configuration | dtype | output | elements | max abs err | max rel err | "
             "max ulp | bit-exact |", "|---|---|---|---:|---:|---:|---:|---:|"]
    for cfg, res in runs:
        for n in OUTPUTS:
            if isinstance(res[n], dict):          # merged statistics, already checked
                s = res[n]
            else:
                g, w = res[n]
                check(f"{cfg.name} {n}", g, w, cfg.dtype, exact=n == "res_out")
                s = error_stats(g, w, cfg.dtype)
            lines.append(f"| {cfg.name} | {cfg.dtype} | {n} | {s['n']} | {s['max_abs']:.3g} | "
                         f"{s['max_rel']:.3g} | {s['max_ulp']} | {100 * s['exact']:.2f} % |")
    table = "\n".join(lines) + "\n"
    print(table, flush=True)
    path = os.environ.get("TRI_PARITY_REPORT")
    if path:
        with open(path, "w") as f:
            f.write(table)
