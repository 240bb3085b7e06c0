"""The decode ops, evaluated plainly in float64 (test infrastructure only).

The paper names these kernels without writing their formulas: `rms_norm`
is its motivating example (Sec. 2.3, Fig. 1) and `rms_norm`, `silu` and
`add` are in its kernel suite (Sec. 4.1). The definitions below are the
standard Llama-family forms; the readings taken where the paper is silent
are:

* RMSNorm: y = w * x / sqrt(mean(x^2) + eps), eps inside the square root,
  the mean accumulated in float64 here (float32 on the GPU), one rounding
  of the final product to the output dtype.
* Residual add: h = RN_dtype(x + r); the norm is applied to the ROUNDED h,
  which is also the residual output. (For two bf16 or two f32 operands the
  exact sum rounded once equals a float32 add followed by a rounding to the
  dtype, so this is also what the GPU computes.)
* RoPE: rotate-half pairing (i, i + hd/2); inverse frequencies are the
  correctly rounded float32 values of base^(-2i/hd); the angle is ONE
  float32 product float32(pos) * inv_i, as every float32 implementation
  forms it; cos and sin of that float32 angle are taken in float64 and not
  rounded before use. Every head of a token (Q and K) uses the same angles.
* SwiGLU: out = g / (1 + exp(-g)) * u with the gate as the first operand;
  for very negative g the exponential overflows and the result is a signed
  zero, never NaN.
* QK-RMSNorm before RoPE (Qwen3-style heads): every Q and K head vector is
  RMS-normalised over its hd elements with a per-dimension weight (one
  weight vector for Q, one for K) and then rotated; the normalised head is
  not rounded in between, so the fused op rounds once, like every op here.
* Decode chain: the three ops above on disjoint operands, in one call; with
  head-norm weights given, RoPE becomes QK-RMSNorm + RoPE.
"""
from __future__ import annotations

from decimal import Decimal, localcontext
from typing import Dict

import numpy as np

from .numerics import BF16, F32, round_to, values


def _rmsnorm64(xv: np.ndarray, wv: np.ndarray, eps: float) -> np.ndarray:
    """w * x / sqrt(mean(x^2) + eps) over the last axis, float64 in and out."""
    eps64 = float(np.float32(eps))          # the caller passes eps as float32
    ms = np.mean(xv * xv, axis=-1, keepdims=True)
    return wv * xv / np.sqrt(ms + eps64)


def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float, dtype: str) -> np.ndarray:
    """RMSNorm over the last axis. x: [..., H], w: [H]."""
    return round_to(_rmsnorm64(values(x, dtype), values(w, dtype), eps), dtype)


def residual_add(x: np.ndarray, r: np.ndarray, dtype: str) -> np.ndarray:
    """h = RN_dtype(x + r), the residual stream after the add."""
    return round_to(values(x, dtype) + values(r, dtype), dtype)


def residual_rmsnorm(x, r, w, eps, dtype):
    """Fused residual add + RMSNorm: returns (y, h) with y = RMSNorm(h)."""
    h = residual_add(x, r, dtype)
    return rmsnorm(h, w, eps, dtype), h


def _decimal_to_f32(d: Decimal) -> np.float32:
    """Nearest float32 to a positive Decimal, ties to even."""
    f = np.float32(float(d))
    cands = [np.nextafter(f, np.float32(0)), f, np.nextafter(f, np.float32(np.inf))]
    best = None
    for c in cands:
        err = abs(Decimal(float(c)) - d)
        even = (int(np.float32(c).view(np.uint32)) & 1) == 0
        rank = (err, not even)
        if best is None or rank < best[0]:
            best = (rank, c)
    return np.float32(best[1])


def rope_inv_freq(base: float, hd: int) -> np.ndarray:
    """inv_i = RN_f32(base^(-2i/hd)) for i in [0, hd/2), exactly rounded.

    The power is evaluated with 60 significant decimal digits
    (exp(ln(base) * -2i/hd)) and then rounded to the nearest float32.
    `base` is the float32 value the caller passes.
    """
    b = Decimal(float(np.float32(base)))
    out = np.empty(hd // 2, dtype=np.float32)
    with localcontext() as ctx:
        ctx.prec = 60
        lnb = b.ln()
        for i in range(hd // 2):
            ex = Decimal(-2 * i) / Decimal(hd)
            out[i] = _decimal_to_f32((lnb * ex).exp())
    return out


def rope_angles(pos: np.ndarray, inv: np.ndarray) -> np.ndarray:
    """theta[t, i] = RN_f32(float32(pos_t) * inv_i), returned as float64."""
    p32 = np.asarray(pos, dtype=np.int32).astype(np.float32)
    th = p32[:, None] * np.asarray(inv, dtype=np.float32)[None, :]   # float32 product
    assert th.dtype == np.float32
    return th.astype(np.float64)


def _rotate64(vv: np.ndarray, theta: np.ndarray) -> np.ndarray:
    """Rotate-half of float64 heads vv: [T, nh, hd] by theta: [T, hd/2]."""
    half = vv.shape[-1] // 2
    c = np.cos(theta)[:, None, :]
    s = np.sin(theta)[:, None, :]
    v1 = vv[..., :half]
    v2 = vv[..., half:]
    return np.concatenate([v1 * c - v2 * s, v2 * c + v1 * s], axis=-1)


def rope_apply(v: np.ndarray, theta: np.ndarray, dtype: str) -> np.ndarray:
    """Rotate-half RoPE of v: [T, nh, hd] by angles theta: [T, hd/2]."""
    return round_to(_rotate64(values(v, dtype), theta), dtype)


def rope_qk(q, k, pos, base, dtype):
    """RoPE on Q [T, nq, hd] and K [T, nk, hd] with one position per token."""
    hd = q.shape[-1]
    theta = rope_angles(pos, rope_inv_freq(base, hd))
    qo = rope_apply(q, theta, dtype)
    ko = rope_apply(k, theta, dtype) if k is not None and k.size else k
    return qo, ko


def qk_norm_rope(q, k, pos, base, q_w, k_w, eps, dtype):
    """Per-head RMSNorm of Q [T, nq, hd] and K [T, nk, hd] (weights [hd]),
    then rotate-half RoPE of the normalised heads; one rounding at the end."""
    hd = q.shape[-1]
    theta = rope_angles(pos, rope_inv_freq(base, hd))

    def one(v, w):
        n = _rmsnorm64(values(v, dtype), values(w, dtype), eps)
        return round_to(_rotate64(n, theta), dtype)
    qo = one(q, q_w)
    ko = one(k, k_w) if k is not None and k.size else k
    return qo, ko


def swiglu(gate, up, dtype):
    """out = silu(gate) * up with silu(g) = g / (1 + exp(-g))."""
    g = values(gate, dtype)
    u = values(up, dtype)
    with np.errstate(over="ignore"):
        out = g / (1.0 + np.exp(-g)) * u
    return round_to(out, dtype)


def decode_chain(inp: Dict[str, np.ndarray], eps: float, base: float,
                 dtype: str) -> Dict[str, np.ndarray]:
    """Residual add + RMSNorm, RoPE on Q/K and SwiGLU on disjoint operands."""
    y, h = residual_rmsnorm(inp["x"], inp["residual"], inp["w"], eps, dtype)
    if inp.get("q_norm_w") is not None:
        qo, ko = qk_norm_rope(inp["q"], inp["k"], inp["pos"], base, inp["q_norm_w"],
                              inp["k_norm_w"], inp.get("qk_eps", eps), dtype)
    else:
        qo, ko = rope_qk(inp["q"], inp["k"], inp["pos"], base, dtype)
    out = swiglu(inp["gate"], inp["up"], dtype)
    return dict(y=y, res_out=h, q=qo, k=ko, out=out)


__all__ = ["rmsnorm", "residual_add", "residual_rmsnorm", "rope_inv_freq",
           "rope_angles", "rope_apply", "rope_qk", "qk_norm_rope", "swiglu", "decode_chain",
           "F32", "BF16"]
