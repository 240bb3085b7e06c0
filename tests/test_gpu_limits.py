"""GPU: the library's size limits, on real buffers (sampled oracle checks).

T = 2^22 tokens (the most a call accepts), 4096 + 4096 heads, SwiGLU rows
of 2^31 - 3 elements (the widest accepted; two such rows put element
indices past 2^31) and a Llama-3 sized embedding table.
Inputs are drawn on the device with torch's seeded generator; the oracle
evaluates sampled rows / elements copied back. Every case prints its name
(pytest -v) before touching the GPU.
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


def gen(seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return g


def host(t):
    return wl.from_torch(t)


def sample_rows(n, k, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    rows = np.concatenate([[0, 1, n // 2, n - 2, n - 1], r.choice(n, size=k, replace=False)])
    return np.unique(rows)


@pytest.mark.parametrize("H", [64, 4096])
def test_max_tokens_residual_rmsnorm(tri, cache, H):
    T = S.T_MAX if H == 64 else 1 << 18
    g = gen(5)
    x = torch.randn((T, H), generator=g, device=DEV, dtype=torch.bfloat16)
    r = torch.randn((T, H), generator=g, device=DEV, dtype=torch.bfloat16)
    w = (torch.rand((H,), generator=g, device=DEV) + 0.5).to(torch.bfloat16)
    y, ro = cache.residual_rmsnorm(x, r, w, 1e-6)
    torch.cuda.synchronize()
    rec = cache.last_selection()
    assert rec.launch[0].grid_x == (T // 4 if H == 64 else T)
    rows = torch.from_numpy(sample_rows(T, 60, 1)).to(DEV)
    wy, wh = O.residual_rmsnorm(host(x[rows]), host(r[rows]), host(w), 1e-6, nm.BF16)
    check("y", host(y[rows]), wy, nm.BF16)
    check("res_out", host(ro[rows]), wh, nm.BF16, exact=True)


def test_max_tokens_fused_chain(tri, cache):
    """2^22 tokens through the fused chain: 2^20 norm workgroups (a wavefront
    per row), 2^20 RoPE workgroups (three heads of one vector fill 3 lanes:
    four tokens per workgroup) and the SwiGLU role at its grid cap."""
    T, H, I, hd = S.T_MAX, 256, 256, 16
    g = gen(6)
    bf = torch.bfloat16
    x = torch.randn((T, H), generator=g, device=DEV, dtype=bf)
    res = torch.randn((T, H), generator=g, device=DEV, dtype=bf)
    w = (torch.rand((H,), generator=g, device=DEV) + 0.5).to(bf)
    q = torch.randn((T, 2, hd), generator=g, device=DEV, dtype=bf)
    k = torch.randn((T, 1, hd), generator=g, device=DEV, dtype=bf)
    pos = torch.randint(0, 1 << 20, (T,), generator=g, device=DEV, dtype=torch.int32)
    gate = torch.randn((T, I), generator=g, device=DEV, dtype=bf)
    up = torch.randn((T, I), generator=g, device=DEV, dtype=bf)
    q0, k0 = q.clone(), k.clone()
    y, ro, out = cache.decode_chain(x, res, w, q, k, pos, gate, up, 1e-6, 5e5)
    torch.cuda.synchronize()
    rec = cache.last_selection()
    assert rec.variant == S.CH_FUSED
    assert rec.launch[0].grid_x == T // 4 + T // 4 + min((T * I // 8) // 256, S.GRID_CAP)
    rows = torch.from_numpy(sample_rows(T, 40, 2)).to(DEV)
    wy, wh = O.residual_rmsnorm(host(x[rows]), host(res[rows]), host(w), 1e-6, nm.BF16)
    check("y", host(y[rows]), wy, nm.BF16)
    check("res_out", host(ro[rows]), wh, nm.BF16, exact=True)
    wq, wk = O.rope_qk(host(q0[rows]), host(k0[rows]), host(pos[rows]), 5e5, nm.BF16)
    check("q", host(q[rows]), wq, nm.BF16)
    check("k", host(k[rows]), wk, nm.BF16)
    check("out", host(out[rows]), O.swiglu(host(gate[rows]), host(up[rows]), nm.BF16), nm.BF16)


@pytest.mark.parametrize("dtype,hd,qkn,unaligned", [(nm.BF16, 128, False, False),
                                                    (nm.F32, 512, False, False),
                                                    (nm.BF16, 128, True, False),
                                                    (nm.F32, 64, True, True)])
def test_max_heads_rope(tri, cache, dtype, hd, qkn, unaligned):
    """4096 Q + 4096 K heads (the most a call accepts), every output checked."""
    T = 3 if hd < 512 else 1
    nh = S.HEADS_MAX
    r = np.random.Generator(np.random.PCG64(hd + qkn))
    q = wl.host_array(r, (T, nh, hd), dtype)
    k = wl.host_array(r, (T, nh, hd), dtype)
    qw, kw = wl.host_weight(r, hd, dtype), wl.host_weight(r, hd, dtype)
    pos = r.integers(0, 8192, size=T).astype(np.int32)
    td = wl.torch_dtype(dtype)

    def put(a):
        t = wl.to_torch(a, dtype, DEV)
        if not unaligned:
            return t
        buf = torch.zeros(t.numel() + 1, dtype=td, device=DEV)
        view = buf[1:].view(t.shape)
        view.copy_(t)
        return view
    qd, kd = put(q), put(k)
    cache.rope(qd, kd, wl.to_torch(pos, dtype, DEV), 1e6, None,
               q_w=wl.to_torch(qw, dtype, DEV) if qkn else None,
               k_w=wl.to_torch(kw, dtype, DEV) if qkn else None)
    torch.cuda.synchronize()
    if qkn:
        wq, wk = O.qk_norm_rope(q, k, pos, 1e6, qw, kw, 1e-6, dtype)
    else:
        wq, wk = O.rope_qk(q, k, pos, 1e6, dtype)
    check("q", host(qd), wq, dtype)
    check("k", host(kd), wk, dtype)
    want = S.ROPE_QKN_SCALAR if unaligned else (S.ROPE_QKN_VEC if qkn else S.ROPE_VEC)
    assert cache.last_selection().variant == want


@pytest.mark.parametrize("I,variant", [(S.I_LIMIT - 8, S.SW_FLAT_NT),
                                       (S.I_LIMIT - 3, S.SW_SCALAR)])
def test_widest_swiglu_rows_sampled(tri, cache, I, variant):
    """Two rows of nearly 2^31 elements (2^31 - 3 is the widest accepted):
    element indices past 2^31 and grid-stride passes at the grid cap -- the
    flat vector form, streaming (rows a whole number of vectors; the call
    moves 24 GiB), or the element-wise form (odd rows are not 16-byte
    aligned)."""
    T = 2
    g = gen(7)
    gate = torch.randn((T, I), generator=g, device=DEV, dtype=torch.bfloat16)
    up = torch.randn((T, I), generator=g, device=DEV, dtype=torch.bfloat16)
    out = cache.swiglu(gate, up)
    torch.cuda.synchronize()
    rec = cache.last_selection()
    assert rec.variant == variant and rec.launch[0].grid_x == S.GRID_CAP
    n = T * I
    r = np.random.Generator(np.random.PCG64(3))
    idx = np.unique(np.concatenate([np.arange(8), n - 1 - np.arange(13),
                                    (1 << 31) + np.arange(-12, 12), (1 << 30) * 3 + np.arange(4),
                                    r.integers(0, n, size=200)]))
    it = torch.from_numpy(idx).to(DEV)
    gh, uh = host(gate.view(-1)[it]), host(up.view(-1)[it])
    check("out", host(out.view(-1)[it]), O.swiglu(gh, uh, nm.BF16), nm.BF16)
    del gate, up, out


def test_large_vocabulary_embedding(tri, cache):
    vocab, H, T = 128256, 4096, 4096
    g = gen(8)
    table = torch.randn((vocab, H), generator=g, device=DEV, dtype=torch.bfloat16)
    ids = torch.randint(0, vocab, (T,), generator=g, device=DEV, dtype=torch.int64)
    ids[0], ids[1], ids[2] = vocab - 1, -1, vocab
    out = cache.embedding(table, ids)
    torch.cuda.synchronize()
    rows = np.union1d(sample_rows(T, 50, 4), [1, 2])
    ih = host(ids)
    for t in rows:
        i = int(ih[t])
        got = host(out[int(t)])
        if 0 <= i < vocab:
            check(f"row {t}", got, host(table[i]), nm.BF16, exact=True)
        else:
            assert not got.any(), t
