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
  where the exponential overflows (in float64, below g = -709) the result is
  a signed zero, never NaN; g = -inf gives NaN (-inf / inf).
* QK-RMSNorm before RoPE (Qwen3-style heads): every Q and K head vector is
  RMS-normalised over its hd elements with a per-dimension weight (one
  weight vector for Q, one for K) and then rotated; the normalised head is
  not rounded in between, so the fused op rounds once, like every op here.
* Short ops of the paper's suite (`silu`, `add`, `masked_fill`,
  `embedding`): silu as in SwiGLU without the up operand; add rounds the
  exact sum once; masked_fill writes the fill value rounded to the dtype
  where the uint8 mask is nonzero and copies x bit for bit elsewhere;
  embedding copies table rows by id and writes zeros for ids out of range.
* Decode chain: the three ops above on disjoint operands, in one call; with
  head-norm weights given, RoPE becomes QK-RMSNorm + RoPE.
* RoPE variants (`rope_ext`): GPT-J pairs (2i, 2i + 1) instead of
  rotate-half; partial rotary over the first rd <= hd elements of each head
  with inv_i = RN_f32(base^(-2i/rd)) and the rest passed through (or only
  normalised, with the QK norm); int64 positions, converted to float32 with
  one round-to-nearest-even step; Llama-3 frequency scaling of the inverse
  frequencies (the published piecewise rule: wavelengths below
  L / high_freq_factor keep their frequency, those above L / low_freq_factor
  are divided by `factor`, and those in between interpolate linearly in
  L / wavelength, L the original context length), evaluated exactly and
  rounded to float32 once; or cos / sin read from a caller's float32 cache
  with rows [cos_0 .. cos_{rd/2-1}, sin_0 .. sin_{rd/2-1}] per position,
  positions clamped to the cache's rows.
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


_PREC = 60


def _inv_freq_exact(base: float, hd: int):
    """base^(-2i/hd) for i in [0, hd/2) as 60-digit Decimals (exp of a log);
    `base` is the float32 value the caller passes."""
    b = Decimal(float(np.float32(base)))
    with localcontext() as ctx:
        ctx.prec = _PREC
        lnb = b.ln()
        return [(lnb * (Decimal(-2 * i) / Decimal(hd))).exp() for i in range(hd // 2)]


def rope_inv_freq(base: float, hd: int) -> np.ndarray:
    """inv_i = RN_f32(base^(-2i/hd)) for i in [0, hd/2), exactly rounded.

    The power is evaluated with 60 significant decimal digits
    (exp(ln(base) * -2i/hd)) and then rounded to the nearest float32.
    """
    return np.array([_decimal_to_f32(v) for v in _inv_freq_exact(base, hd)], dtype=np.float32)


def _decimal_pi() -> Decimal:
    """pi to the working precision (Machin: 16 atan(1/5) - 4 atan(1/239))."""
    def atan_inv(n: int) -> Decimal:
        x = Decimal(1) / n
        x2 = x * x
        term, total, k = x, x, 1
        while True:
            term = -term * x2
            k += 2
            t = term / k
            if t == 0 or abs(t) < Decimal(10) ** (-(_PREC + 5)):
                break
            total += t
        return total
    with localcontext() as ctx:
        ctx.prec = _PREC + 10
        return 16 * atan_inv(5) - 4 * atan_inv(239)


def llama3_scale(inv: Decimal, factor: float, low: float, high: float, orig: int) -> Decimal:
    """The Llama-3 rule applied to one exact inverse frequency (Decimal)."""
    f, lo, hi = (Decimal(float(np.float32(v))) for v in (factor, low, high))
    L = Decimal(int(orig))
    with localcontext() as ctx:
        ctx.prec = _PREC
        wavelen = 2 * _decimal_pi() / inv
        if wavelen < L / hi:
            return inv
        if wavelen > L / lo:
            return inv / f
        smooth = (L / wavelen - lo) / (hi - lo)
        return (1 - smooth) * inv / f + smooth * inv


def rope_inv_freq_llama3(base: float, hd: int, factor: float, low: float, high: float,
                         orig: int) -> np.ndarray:
    """Llama-3-scaled inverse frequencies, evaluated exactly, rounded once."""
    return np.array([_decimal_to_f32(llama3_scale(v, factor, low, high, orig))
                     for v in _inv_freq_exact(base, hd)], dtype=np.float32)


def rope_angles(pos: np.ndarray, inv: np.ndarray) -> np.ndarray:
    """theta[t, i] = RN_f32(float32(pos_t) * inv_i), returned as float64.
    Positions are int32 or int64; the conversion to float32 rounds to
    nearest, ties to even."""
    p = np.asarray(pos)
    assert p.dtype in (np.int32, np.int64)
    p32 = p.astype(np.float32)
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


def _rotate_pairs64(vv: np.ndarray, c: np.ndarray, s: np.ndarray, rd: int,
                    interleaved: bool) -> np.ndarray:
    """Rotate the first rd elements of float64 heads vv [T, nh, hd] by cos c /
    sin s [T, rd/2]: pairs (i, i + rd/2), or (2i, 2i + 1) when interleaved.
    Elements past rd are returned unchanged."""
    out = vv.copy()
    c = c[:, None, :]
    s = s[:, None, :]
    if interleaved:
        x, y = vv[..., 0:rd:2], vv[..., 1:rd:2]
        out[..., 0:rd:2] = x * c - y * s
        out[..., 1:rd:2] = y * c + x * s
    else:
        h = rd // 2
        x, y = vv[..., :h], vv[..., h:rd]
        out[..., :h] = x * c - y * s
        out[..., h:rd] = y * c + x * s
    return out


def rope_ext(q, k, pos, base, dtype, *, rotary_dim=None, interleaved=False, scaling=None,
             cos_sin=None, q_w=None, k_w=None, eps=1e-6):
    """RoPE on Q [T, nq, hd] and K [T, nk, hd] with the variants above.

    rotary_dim: rd (default hd). scaling: None or a dict with factor,
    low_freq_factor, high_freq_factor, original_max_pos (Llama-3 rule).
    cos_sin: float32 [n, rd] cache (base and scaling unused). q_w / k_w:
    QK-RMSNorm over the whole head first. One rounding at the end.
    """
    hd = q.shape[-1]
    rd = hd if rotary_dim is None else rotary_dim
    if cos_sin is not None:
        cache = np.asarray(cos_sin, dtype=np.float32)
        p = np.clip(np.asarray(pos).astype(np.int64), 0, cache.shape[0] - 1)
        c = cache[p, : rd // 2].astype(np.float64)
        s = cache[p, rd // 2: rd].astype(np.float64)
    else:
        if scaling is None:
            inv = rope_inv_freq(base, rd)
        else:
            inv = rope_inv_freq_llama3(base, rd, scaling["factor"], scaling["low_freq_factor"],
                                       scaling["high_freq_factor"],
                                       scaling["original_max_pos"])
        theta = rope_angles(pos, inv)
        c, s = np.cos(theta), np.sin(theta)

    def one(v, w):
        vv = values(v, dtype)
        if w is not None:
            vv = _rmsnorm64(vv, values(w, dtype), eps)
        return round_to(_rotate_pairs64(vv, c, s, rd, interleaved), dtype)
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


# ---- short element-wise and gather ops (the paper's operator suite, Sec. 4.1) ----
def silu(x, dtype):
    """silu(x) = x / (1 + exp(-x)), one rounding; below x = -709 the float64
    exponential overflows and the result is a signed zero, never NaN."""
    v = values(x, dtype)
    with np.errstate(over="ignore"):
        return round_to(v / (1.0 + np.exp(-v)), dtype)


def add(a, b, dtype):
    """a + b, one rounding of the exact sum."""
    return round_to(values(a, dtype) + values(b, dtype), dtype)


def masked_fill(x, mask, value, dtype):
    """Where mask (uint8, nonzero = set) the element becomes `value` rounded
    to the dtype (from the float32 the caller passes); elsewhere x is copied."""
    v = round_to(np.full(1, float(np.float32(value)), dtype=np.float64), dtype)[0]
    out = np.array(x, copy=True)
    out[np.asarray(mask) != 0] = v
    return out


def embedding(table, ids, dtype):
    """Rows of table [n_rows, H] picked by ids [T] (int32 or int64); an id
    outside [0, n_rows) gives a row of zeros."""
    ids = np.asarray(ids).astype(np.int64)
    n_rows = table.shape[0]
    ok = (ids >= 0) & (ids < n_rows)
    out = np.zeros((ids.shape[0],) + table.shape[1:], dtype=table.dtype)
    out[ok] = table[ids[ok]]
    return out


def decode_chain(inp: Dict[str, np.ndarray], eps: float, base: float,
                 dtype: str) -> Dict[str, np.ndarray]:
    """Residual add + RMSNorm, RoPE on Q/K and SwiGLU on disjoint operands.
    inp["rope_ext"] (keyword arguments of rope_ext) selects a RoPE variant."""
    y, h = residual_rmsnorm(inp["x"], inp["residual"], inp["w"], eps, dtype)
    if inp.get("rope_ext") is not None:
        qo, ko = rope_ext(inp["q"], inp["k"], inp["pos"], base, dtype, q_w=inp.get("q_norm_w"),
                          k_w=inp.get("k_norm_w"), eps=inp.get("qk_eps", eps),
                          **inp["rope_ext"])
    elif inp.get("q_norm_w") is not None:
        qo, ko = qk_norm_rope(inp["q"], inp["k"], inp["pos"], base, inp["q_norm_w"],
                              inp["k_norm_w"], inp.get("qk_eps", eps), dtype)
    else:
        qo, ko = rope_qk(inp["q"], inp["k"], inp["pos"], base, dtype)
    out = swiglu(inp["gate"], inp["up"], dtype)
    return dict(y=y, res_out=h, q=qo, k=ko, out=out)


__all__ = ["silu", "add", "masked_fill", "embedding", "rmsnorm", "residual_add", "residual_rmsnorm", "rope_inv_freq",
           "rope_inv_freq_llama3", "llama3_scale", "rope_angles", "rope_apply", "rope_qk",
           "qk_norm_rope", "rope_ext", "swiglu", "decode_chain", "F32", "BF16"]
