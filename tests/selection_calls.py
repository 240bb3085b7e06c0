"""Builders of oracle selection-model calls from plain dimensions.

Shared by the CPU tests of the selection model and of the host library, so
both see the same synthetic addresses and strides. Addresses are integers
(no memory behind them): the selection depends only on their values.
"""
from oracle import selection as S

BASE_ADDR = 0x7F0000000000


def _addr(i):
    return BASE_ADDR + i * (1 << 32)


def rn_call(dtype, T, H, *, eps=1e-6, off=0, pad=0, null=()):
    ptr = {n: (_addr(i) + off if n != "w" else _addr(i)) for i, n in enumerate(S.RN_PTRS)}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_RMSNORM, dtype, T, H=H, eps=eps, ptr=ptr,
                  stride={"x": H + pad, "y": H + pad})


def res_call(dtype, T, H, *, eps=1e-6, off=0, pad=0, null=(), op=S.OP_RES_RMSNORM):
    ptr = {n: (_addr(i) + off if n != "w" else _addr(i)) for i, n in enumerate(S.RES_PTRS)}
    for n in null:
        ptr[n] = None
    return S.Call(op, dtype, T, H=H, eps=eps, ptr=ptr,
                  stride={n: H + pad for n in S.RES_STRIDES})


CACHE_ADDR = _addr(15)


def rope_call(dtype, T, nq, nk, hd, *, base=10000.0, off=0, pad=0, pos_off=0, null=(),
              ext=None):
    """RoPE call; `ext` (keys of the selection model's PLAIN_EXT, cos_sin as
    an address) selects a variant."""
    ptr = {"q": _addr(10) + off, "k": _addr(11) + off, "pos": _addr(12) + pos_off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_ROPE_QK, dtype, T, hd=hd, nq=nq, nk=nk, base=base, ptr=ptr,
                  stride={"q": nq * hd + pad, "k": nk * hd + pad}, ext=ext)


def qkn_call(dtype, T, nq, nk, hd, *, base=10000.0, eps=1e-6, off=0, pad=0, w_off=0,
             pos_off=0, null=(), ext=None):
    """QK-RMSNorm + RoPE; w_off displaces both head-norm weights."""
    ptr = {"q": _addr(10) + off, "k": _addr(11) + off, "pos": _addr(12) + pos_off,
           "q_w": _addr(13) + w_off, "k_w": _addr(14) + w_off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_QK_NORM_ROPE, dtype, T, hd=hd, nq=nq, nk=nk, base=base, eps=eps,
                  ptr=ptr, stride={"q": nq * hd + pad, "k": nk * hd + pad}, ext=ext)


def sw_call(dtype, T, I, *, off=0, pad=0, null=()):
    ptr = {"gate": _addr(20) + off, "up": _addr(21) + off, "out": _addr(22) + off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_SWIGLU, dtype, T, I=I, ptr=ptr,
                  stride={"gate": I + pad, "up": I + pad, "out": I + pad})


def chain_call(dtype, T, H, I, nq, nk, hd, *, base=10000.0, eps=1e-6,
               res_off=0, res_pad=0, rope_off=0, rope_pad=0, sw_off=0, sw_pad=0,
               qk_norm=False, qk_eps=1e-6, w_off=0, null=(), ext=None):
    r = res_call(dtype, T, H, eps=eps, off=res_off, pad=res_pad)
    if qk_norm:
        q = qkn_call(dtype, T, nq, nk, hd, base=base, off=rope_off, pad=rope_pad, w_off=w_off)
    else:
        q = rope_call(dtype, T, nq, nk, hd, base=base, off=rope_off, pad=rope_pad)
    s = sw_call(dtype, T, I, off=sw_off, pad=sw_pad)
    ptr = dict(r.ptr)
    ptr.update(q.ptr)
    ptr.update(s.ptr)
    stride = dict(r.stride)
    stride.update(q.stride)
    stride.update(s.stride)
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_CHAIN, dtype, T, H=H, I=I, hd=hd, nq=nq, nk=nk, eps=eps,
                  base=base, qk_eps=qk_eps, ptr=ptr, stride=stride, ext=ext)


def elem_offset(dtype, n=1):
    """Byte offset of n elements (used to build unaligned layouts)."""
    return n * S.elem_size(dtype)


def silu_call(dtype, T, W, *, off=0, pad=0, null=()):
    ptr = {"a": _addr(30) + off, "b": _addr(30) + off, "out": _addr(32) + off}
    for n in null:
        ptr[n] = None
    if "a" in null:
        ptr["b"] = None
    return S.Call(S.OP_SILU, dtype, T, H=W, ptr=ptr, stride={n: W + pad for n in ("a", "b", "out")})


def add_call(dtype, T, W, *, off=0, b_off=0, pad=0, null=()):
    ptr = {"a": _addr(30) + off, "b": _addr(31) + off + b_off, "out": _addr(32) + off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_ADD, dtype, T, H=W, ptr=ptr, stride={n: W + pad for n in ("a", "b", "out")})


def mf_call(dtype, T, W, *, off=0, m_off=0, pad=0, m_pad=0, value=-1e4, null=()):
    ptr = {"a": _addr(30) + off, "b": _addr(33) + m_off, "out": _addr(32) + off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_MASKED_FILL, dtype, T, H=W, value=value, ptr=ptr,
                  stride={"a": W + pad, "b": W + m_pad, "out": W + pad})


def emb_call(dtype, T, H, n_rows, *, ids64=0, off=0, pad=0, ids_off=0, null=()):
    ptr = {"table": _addr(34) + off, "ids": _addr(35) + ids_off, "out": _addr(36) + off}
    for n in null:
        ptr[n] = None
    return S.Call(S.OP_EMBEDDING, dtype, T, H=H, n_rows=n_rows, ids64=ids64, ptr=ptr,
                  stride={"table": H + pad, "out": H + pad})
