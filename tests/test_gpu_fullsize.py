"""Every op the benchmark times at 8192 tokens, at that size and in that
launch configuration (one default cache, the benchmark's shapes), checked
against the oracle on every row, in chunks of 512 rows (the float64 oracle
of one chunk fits comfortably in host memory).

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


CHUNK = 512


def chunks(T=CFG.T):
    """Row ranges covering all T rows, CHUNK at a time."""
    return [slice(r0, min(T, r0 + CHUNK)) for r0 in range(0, T, CHUNK)]


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
    w = host(data["w"])
    for sl in chunks():
        check(f"y {sl}", host(y[sl]), O.rmsnorm(host(data["x"][sl]), w, CFG.eps, nm.BF16),
              nm.BF16)


def test_residual_rmsnorm_8192(tri, data):
    print("full size: residual rmsnorm", flush=True)
    (y, ro), _ = run(tri, lambda c: c.residual_rmsnorm(data["x"], data["residual"], data["w"],
                                                          CFG.eps))
    w = host(data["w"])
    for sl in chunks():
        wy, wh = O.residual_rmsnorm(host(data["x"][sl]), host(data["residual"][sl]), w,
                                    CFG.eps, nm.BF16)
        check(f"y {sl}", host(y[sl]), wy, nm.BF16)
        check(f"res_out {sl}", host(ro[sl]), wh, nm.BF16, exact=True)


@pytest.mark.parametrize("qkn", [False, True], ids=["rope", "qk_norm_rope"])
def test_rope_8192(tri, data, qkn):
    print(f"full size: rope (qk norm {qkn})", flush=True)
    q, k = data["q"].clone(), data["k"].clone()
    if qkn:
        run(tri, lambda c: c.qk_norm_rope(q, k, data["pos"], data["qw"], data["kw"], CFG.base,
                                          CFG.eps))
    else:
        run(tri, lambda c: c.rope_qk(q, k, data["pos"], CFG.base))
    qw, kw = host(data["qw"]), host(data["kw"])
    for sl in chunks():
        q0, k0, p = host(data["q"][sl]), host(data["k"][sl]), host(data["pos"][sl])
        if qkn:
            wq, wk = O.qk_norm_rope(q0, k0, p, CFG.base, qw, kw, CFG.eps, nm.BF16)
        else:
            wq, wk = O.rope_qk(q0, k0, p, CFG.base, nm.BF16)
        check(f"q {sl}", host(q[sl]), wq, nm.BF16)
        check(f"k {sl}", host(k[sl]), wk, nm.BF16)


def test_swiglu_8192(tri, data):
    print("full size: swiglu", flush=True)
    out, sel = run(tri, lambda c: c.swiglu(data["gate"], data["up"]))
    assert sel.variant == S.SW_FLAT_NT                       # 1.3 GiB: streams
    for sl in chunks():
        check(f"out {sl}", host(out[sl]),
              O.swiglu(host(data["gate"][sl]), host(data["up"][sl]), nm.BF16), nm.BF16)


def test_chain_with_qk_norm_8192(tri, data):
    print("full size: chain with QK norm", flush=True)
    q, k = data["q"].clone(), data["k"].clone()
    (y, ro, out), sel = run(tri, lambda c: c.decode_chain(
        data["x"], data["residual"], data["w"], q, k, data["pos"], data["gate"], data["up"],
        CFG.eps, CFG.base, q_norm_w=data["qw"], k_norm_w=data["kw"]))
    assert sel.variant == S.CH_FUSED and sel.roles[1] == S.ROPE_QKN_VEC
    w, qw, kw = host(data["w"]), host(data["qw"]), host(data["kw"])
    for sl in chunks():
        inp = dict(x=host(data["x"][sl]), residual=host(data["residual"][sl]), w=w,
                   q=host(data["q"][sl]), k=host(data["k"][sl]), pos=host(data["pos"][sl]),
                   gate=host(data["gate"][sl]), up=host(data["up"][sl]), q_norm_w=qw,
                   k_norm_w=kw)
        want = O.decode_chain(inp, CFG.eps, CFG.base, nm.BF16)
        for n, got in (("y", y), ("out", out), ("q", q), ("k", k)):
            check(f"{n} {sl}", host(got[sl]), want[n], nm.BF16)
        check(f"res_out {sl}", host(ro[sl]), want["res_out"], nm.BF16, exact=True)


@pytest.mark.parametrize("op", ["silu", "add", "masked_fill"])
def test_short_ops_8192(tri, data, op):
    print(f"full size: {op}", flush=True)
    x, r = data["x"], data["residual"]
    if op == "silu":
        out, sel = run(tri, lambda c: c.silu(x))
    elif op == "add":
        out, sel = run(tri, lambda c: c.add(x, r))
    else:
        out, sel = run(tri, lambda c: c.masked_fill(x, data["mask"], -1e4))
    assert sel.variant == S.ELT_FLAT_U2
    for sl in chunks():
        if op == "silu":
            want = O.silu(host(x[sl]), nm.BF16)
        elif op == "add":
            want = O.add(host(x[sl]), host(r[sl]), nm.BF16)
        else:
            want = O.masked_fill(host(x[sl]), host(data["mask"][sl]), -1e4, nm.BF16)
        check(f"{op} {sl}", host(out[sl]), want, nm.BF16, exact=op != "silu")


def test_embedding_8192(tri, data):
    print("full size: embedding", flush=True)
    out, sel = run(tri, lambda c: c.embedding(data["table"], data["ids"]))
    assert sel.variant == S.EMB_VEC and sel.launch[0].grid_x == CFG.T
    table = host(data["table"])                  # 128,256 x 4096 bf16: 1 GB on the host
    for sl in chunks():
        want = O.embedding(table, host(data["ids"][sl]), nm.BF16)
        check(f"embedding {sl}", host(out[sl]), want, nm.BF16, exact=True)


# ---- long rows: the benchmark's bf16 [2048, 65536] and the same memory as
# [1024, 131072]: rows split over 4 / 8 workgroups, except plain rows of 65536
# (256 workgroups of 1024, each taking every 256th row) -----------------------------------------
@pytest.fixture(scope="module")
def long_rows():
    g = torch.Generator(device=DEV)
    g.manual_seed(12)
    d = dict(x=torch.randn((2048, 65536), generator=g, device=DEV).to(torch.bfloat16),
             r=torch.randn((2048, 65536), generator=g, device=DEV).to(torch.bfloat16),
             w=(torch.rand(65536, generator=g, device=DEV) + 0.5).to(torch.bfloat16),
             w2=(torch.rand(131072, generator=g, device=DEV) + 0.5).to(torch.bfloat16))
    yield d
    del d
    torch.cuda.synchronize()


@pytest.mark.parametrize("H,res", [(65536, False), (65536, True), (131072, False),
                                   (131072, True)],
                         ids=["rmsnorm65536", "residual65536", "rmsnorm131072",
                              "residual131072"])
def test_long_rows_all_rows(tri, long_rows, H, res):
    T = 2048 * 65536 // H
    S_ = H // 8 // 2048                                  # slices of 2048 vectors
    print(f"full size: long rows T={T} H={H} residual={res}", flush=True)
    x, r = long_rows["x"].view(T, H), long_rows["r"].view(T, H)
    w = long_rows["w"] if H == 65536 else long_rows["w2"]
    if res:
        (y, ro), sel = run(tri, lambda c: c.residual_rmsnorm(x, r, w, CFG.eps))
    else:
        y, sel = run(tri, lambda c: c.rmsnorm(x, w, CFG.eps))
    if res or H > 65536:                                 # split rows
        assert sel.variant == S.RN_SPLIT and sel.launch[0].grid_x == T * S_
    else:                                                # 256 workgroups, 8 rows each
        assert sel.variant == S.RN_WIDE and sel.launch[0].grid_x == 256
    wh = host(w)
    for a in range(0, T, 256):                           # 256 rows: 16-32 M elements
        b = slice(a, min(T, a + 256))
        if res:
            wy, wr = O.residual_rmsnorm(host(x[b]), host(r[b]), wh, CFG.eps, nm.BF16)
            check(f"res_out {b}", host(ro[b]), wr, nm.BF16, exact=True)
        else:
            wy = O.rmsnorm(host(x[b]), wh, CFG.eps, nm.BF16)
        check(f"y {b}", host(y[b]), wy, nm.BF16)
