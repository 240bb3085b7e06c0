"""Every op the benchmark times at 8192 tokens, at that size and in that
launch configuration (one default cache, the benchmark's shapes), checked
against the oracle on sampled rows.

Inputs: the prefill workload drawn on the device (workloads.device_inputs),
plus the benchmark's extra operands (head-norm weights, a 10 % mask, a
128,256-row table of hidden/2 columns with int32 ids). Each case prints its
name before touching the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from oracle import selection as S
from tests.parity import check
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
CFG = wl.PREFILL_8K


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


@pytest.fixture(scope="module")
def data():
    d = wl.device_inputs(CFG, DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    td = d["x"].dtype
    d["qw"] = (torch.rand(CFG.hd, generator=g, device=DEV) + 0.5).to(td)
    d["kw"] = (torch.rand(CFG.hd, generator=g, device=DEV) + 0.5).to(td)
    d["mask"] = (torch.rand(d["x"].shape, generator=g, device=DEV) < 0.1).to(torch.uint8)
    d["table"] = torch.randn((128256, CFG.H // 2), generator=g, device=DEV).to(td)
    d["ids"] = torch.randint(0, 128256, (CFG.T,), generator=g, device=DEV, dtype=torch.int32)
    yield d
    del d
    torch.cuda.synchronize()


def host(t):
    return wl.from_torch(t)


ROWS = np.unique(np.concatenate([[0, 1, 2, 3, CFG.T // 2, CFG.T - 2, CFG.T - 1],
                                 np.random.Generator(np.random.PCG64(42)).choice(
                                     CFG.T, size=32, replace=False)]))


def rows(t):
    return host(t[torch.from_numpy(ROWS).to(DEV)])


def run(tri, fn):
    cache = tri.SpecCache(auto_install=True)
    try:
        out = fn(cache)
        torch.cuda.synchronize()
        return out, cache.last_selection()
    finally:
        torch.cuda.synchronize()
        cache.close()


def test_rmsnorm_8192(tri, data):
    print("full size: rmsnorm", flush=True)
    y, sel = run(tri, lambda c: c.rmsnorm(data["x"], data["w"], CFG.eps))
    assert sel.variant == S.RN_BLOCK[4] and sel.launch[0].grid_x == CFG.T
    check("y", rows(y), O.rmsnorm(rows(data["x"]), host(data["w"]), CFG.eps, nm.BF16), nm.BF16)


def test_residual_rmsnorm_8192(tri, data):
    print("full size: residual rmsnorm", flush=True)
    (y, ro), _ = run(tri, lambda c: c.residual_rmsnorm(data["x"], data["residual"], data["w"],
                                                          CFG.eps))
    wy, wh = O.residual_rmsnorm(rows(data["x"]), rows(data["residual"]), host(data["w"]),
                                CFG.eps, nm.BF16)
    check("y", rows(y), wy, nm.BF16)
    check("res_out", rows(ro), wh, nm.BF16, exact=True)


@pytest.mark.parametrize("qkn", [False, True], ids=["rope", "qk_norm_rope"])
def test_rope_8192(tri, data, qkn):
    print(f"full size: rope (qk norm {qkn})", flush=True)
    q, k = data["q"].clone(), data["k"].clone()
    if qkn:
        run(tri, lambda c: c.qk_norm_rope(q, k, data["pos"], data["qw"], data["kw"], CFG.base,
                                          CFG.eps))
        wq, wk = O.qk_norm_rope(rows(data["q"]), rows(data["k"]), rows(data["pos"]), CFG.base,
                                host(data["qw"]), host(data["kw"]), CFG.eps, nm.BF16)
    else:
        run(tri, lambda c: c.rope_qk(q, k, data["pos"], CFG.base))
        wq, wk = O.rope_qk(rows(data["q"]), rows(data["k"]), rows(data["pos"]), CFG.base,
                           nm.BF16)
    check("q", rows(q), wq, nm.BF16)
    check("k", rows(k), wk, nm.BF16)


def test_swiglu_8192(tri, data):
    print("full size: swiglu", flush=True)
    out, sel = run(tri, lambda c: c.swiglu(data["gate"], data["up"]))
    assert sel.variant == S.SW_FLAT_NT                       # 1.3 GiB: streams
    check("out", rows(out), O.swiglu(rows(data["gate"]), rows(data["up"]), nm.BF16), nm.BF16)


def test_chain_with_qk_norm_8192(tri, data):
    print("full size: chain with QK norm", flush=True)
    q, k = data["q"].clone(), data["k"].clone()
    (y, ro, out), sel = run(tri, lambda c: c.decode_chain(
        data["x"], data["residual"], data["w"], q, k, data["pos"], data["gate"], data["up"],
        CFG.eps, CFG.base, q_norm_w=data["qw"], k_norm_w=data["kw"]))
    assert sel.variant == S.CH_FUSED and sel.roles[1] == S.ROPE_QKN_VEC
    inp = dict(x=rows(data["x"]), residual=rows(data["residual"]), w=host(data["w"]),
               q=rows(data["q"]), k=rows(data["k"]), pos=rows(data["pos"]),
               gate=rows(data["gate"]), up=rows(data["up"]), q_norm_w=host(data["qw"]),
               k_norm_w=host(data["kw"]))
    want = O.decode_chain(inp, CFG.eps, CFG.base, nm.BF16)
    for n, got in (("y", y), ("out", out), ("q", q), ("k", k)):
        check(n, rows(got), want[n], nm.BF16)
    check("res_out", rows(ro), want["res_out"], nm.BF16, exact=True)


@pytest.mark.parametrize("op", ["silu", "add", "masked_fill"])
def test_short_ops_8192(tri, data, op):
    print(f"full size: {op}", flush=True)
    x, r = data["x"], data["residual"]
    if op == "silu":
        out, sel = run(tri, lambda c: c.silu(x))
        want = O.silu(rows(x), nm.BF16)
    elif op == "add":
        out, sel = run(tri, lambda c: c.add(x, r))
        want = O.add(rows(x), rows(r), nm.BF16)
    else:
        out, sel = run(tri, lambda c: c.masked_fill(x, data["mask"], -1e4))
        want = O.masked_fill(rows(x), rows(data["mask"]), -1e4, nm.BF16)
    assert sel.variant == S.ELT_FLAT_U2
    check(op, rows(out), want, nm.BF16, exact=op != "silu")


def test_embedding_8192(tri, data):
    print("full size: embedding", flush=True)
    out, sel = run(tri, lambda c: c.embedding(data["table"], data["ids"]))
    assert sel.variant == S.EMB_VEC and sel.launch[0].grid_x == CFG.T
    ids = rows(data["ids"]).astype(np.int64)
    table_rows = host(data["table"][torch.from_numpy(ids).to(DEV)])
    # the oracle gathers from the rows it is given: present them as a table
    # indexed 0..k-1 so the sampled rows map one to one
    want = O.embedding(table_rows, np.arange(len(ids), dtype=np.int32), nm.BF16)
    check("embedding", rows(out), want, nm.BF16, exact=True)
