"""Tolerance checks and oracle-model calls built from real device tensors.

Tolerances: float32 outputs pass when |g - o| <= 1e-5 |o| + 1e-6 (the
absolute floor covers cancellation near zero in RoPE); bfloat16 outputs pass
when |g - o| <= 2e-2 or g is within one bf16 ulp of the oracle's correctly
rounded value (2e-2 alone is less than one ulp once |o| >= 4, and the
prefill inputs carry x50 outliers).
"""
import numpy as np

from oracle import numerics as nm
from oracle import selection as S
import workloads as wl


def check(name, got, want, dtype, exact=False):
    """Compare a GPU result (host repr) with the oracle's (host repr)."""
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    if exact:
        bad = got.view(np.uint16 if dtype == nm.BF16 else np.uint32) != \
            want.view(np.uint16 if dtype == nm.BF16 else np.uint32)
        assert not bad.any(), f"{name}: {int(bad.sum())} of {bad.size} differ (bit-exact)"
        return
    g = nm.values(got, dtype)
    o = nm.values(want, dtype)
    if dtype == nm.F32:
        bad = ~(np.abs(g - o) <= 1e-5 * np.abs(o) + 1e-6)
    else:
        ulps = nm.bf16_ulp_distance(got, want)
        bad = ~((np.abs(g - o) <= 2e-2) | (ulps <= 1))
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{name}: {int(bad.sum())} of {bad.size} outside tolerance; "
                             f"first at {tuple(i)}: got {g[tuple(i)]!r} want {o[tuple(i)]!r}")


def f32_ulp_distance(a, b) -> np.ndarray:
    """Number of representable float32 values between two float32 arrays
    (sign-magnitude patterns mapped onto a monotone integer line)."""
    def line(x):
        i = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.int64)
        mag = i & 0x7FFFFFFF
        return np.where(i & 0x80000000, -mag, mag)
    return np.abs(line(a) - line(b))


def error_stats(got, want, dtype):
    """Largest |g - o|, largest |g - o| / |o| (over o != 0), largest ulp
    distance from the oracle's correctly rounded value, and the fraction of
    elements equal to it bit for bit. Finite oracle values only."""
    got, want = np.asarray(got), np.asarray(want)
    g, o = nm.values(got, dtype), nm.values(want, dtype)
    fin = np.isfinite(o)
    g, o, got, want = g[fin], o[fin], got[fin], want[fin]
    err = np.abs(g - o)
    nz = o != 0
    ulps = nm.bf16_ulp_distance(got, want) if dtype == nm.BF16 else f32_ulp_distance(got, want)
    bits = np.uint16 if dtype == nm.BF16 else np.uint32
    return {"n": int(o.size), "max_abs": float(err.max(initial=0.0)),
            "max_rel": float((err[nz] / np.abs(o[nz])).max(initial=0.0)),
            "max_ulp": int(ulps.max(initial=0)),
            "exact": float(np.mean(got.view(bits) == want.view(bits))) if o.size else 1.0}


def dt_code(dtype):
    return S.DT_F32 if dtype == nm.F32 else S.DT_BF16


def rows_stride(t):
    return t.stride(0) if t.shape[0] > 1 else max(t.stride(0), t.shape[1])


def tok_stride(t):
    return t.stride(0) if t.shape[0] > 1 else max(t.stride(0), t.shape[1] * t.shape[2])


def oracle_rope_kw(ext, cos_sin=None):
    """Keyword arguments of oracle.ops.rope_ext for an ABI-style variant dict
    (keys of the selection model's PLAIN_EXT); cos_sin: the host table."""
    ext = ext or {}
    kw = dict(rotary_dim=ext.get("rotary_dim") or None,
              interleaved=bool(ext.get("interleaved", 0)))
    if ext.get("scaling", 0) == S.SCALING_LLAMA3:
        kw["scaling"] = {n: ext[n] for n in ("factor", "low_freq_factor", "high_freq_factor",
                                             "original_max_pos")}
    if cos_sin is not None:
        kw["cos_sin"] = cos_sin
    return kw


def binding_rope_ext(tri, ext, cos_sin=None):
    """The binding's RopeExt for an ABI-style variant dict (cos_sin: device table)."""
    ext = ext or {}
    scaling = None
    if ext.get("scaling", 0) == S.SCALING_LLAMA3:
        scaling = {n: ext[n] for n in ("factor", "low_freq_factor", "high_freq_factor",
                                       "original_max_pos")}
    return tri.rope_ext(rotary_dim=ext.get("rotary_dim", 0),
                        interleaved=bool(ext.get("interleaved", 0)),
                        pos_int64=bool(ext.get("pos_int64", 0)), scaling=scaling,
                        cos_sin=cos_sin)


def model_chain_call(d, eps, base, qk_eps=None, ext=None):
    """An oracle-model Call for a decode chain over device tensors `d` (with
    head-norm weights when `d` holds q_norm_w / k_norm_w)."""
    dt = nm.BF16 if str(d["x"].dtype).endswith("bfloat16") else nm.F32
    T, H = d["x"].shape
    _, nq, hd = d["q"].shape
    nk = d["k"].shape[1]
    ptr = dict(x=d["x"].data_ptr(), res=d["residual"].data_ptr(), w=d["w"].data_ptr(),
               y=d["y"].data_ptr(), res_out=d["res_out"].data_ptr(), q=d["q"].data_ptr(),
               k=d["k"].data_ptr(), pos=d["pos"].data_ptr(), gate=d["gate"].data_ptr(),
               up=d["up"].data_ptr(), out=d["out"].data_ptr())
    stride = dict(x=rows_stride(d["x"]), res=rows_stride(d["residual"]),
                  y=rows_stride(d["y"]), res_out=rows_stride(d["res_out"]),
                  q=tok_stride(d["q"]), k=tok_stride(d["k"]), gate=rows_stride(d["gate"]),
                  up=rows_stride(d["up"]), out=rows_stride(d["out"]))
    if d.get("q_norm_w") is not None:
        ptr["q_w"] = d["q_norm_w"].data_ptr()
        ptr["k_w"] = d["k_norm_w"].data_ptr()
    return S.Call(S.OP_CHAIN, dt_code(dt), T, H=H, I=d["gate"].shape[1], hd=hd, nq=nq, nk=nk,
                  eps=eps, base=base, qk_eps=eps if qk_eps is None else qk_eps, ptr=ptr,
                  stride=stride, ext=ext)


def expected_record(call: S.Call, version: int):
    """The oracle model's selection record for a hit on `version`."""
    key = S.make_key(call)
    variant, roles, launches = S.plan(key, call.T)
    rec = S.Record(op=call.op, status=S.OK, version=version, variant=variant,
                   n_launches=len(launches), roles=roles,
                   launch=tuple(launches) + ((0, 0, 0),) * (3 - len(launches)), key=key)
    return rec.as_tuple()


__all__ = ["check", "model_chain_call", "expected_record", "oracle_rope_kw", "binding_rope_ext",
           "wl"]
