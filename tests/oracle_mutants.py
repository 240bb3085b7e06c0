"""Pytest plugin (loaded with -p tests.oracle_mutants) that plants one
plausible mistake in the oracle (its op definitions or its selection model),
named by TRI_ORACLE_MUTANT, before the oracle's pin tests run. tests/test_oracle_mutants.py runs the pins once per
mistake and requires each run to fail: the pins catch a dropped term, a
wrong sign or index, a swapped operand or a wrong rounding step. CPU only;
nothing here touches a GPU or the library."""
import os

import numpy as np

from oracle import ops as O
from oracle.numerics import round_to, values


def _eps_outside(xv, wv, eps):
    ms = np.mean(xv * xv, axis=-1, keepdims=True)
    return wv * xv / (np.sqrt(ms) + float(np.float32(eps)))


def _no_weight(xv, wv, eps):
    ms = np.mean(xv * xv, axis=-1, keepdims=True)
    return xv / np.sqrt(ms + float(np.float32(eps)))


def _mean_n_minus_1(xv, wv, eps):
    ms = np.sum(xv * xv, axis=-1, keepdims=True) / (xv.shape[-1] - 1)
    return wv * xv / np.sqrt(ms + float(np.float32(eps)))


def _rope_sign(vv, theta):
    half = vv.shape[-1] // 2
    c, s = np.cos(theta)[:, None, :], np.sin(theta)[:, None, :]
    v1, v2 = vv[..., :half], vv[..., half:]
    return np.concatenate([v1 * c + v2 * s, v2 * c - v1 * s], axis=-1)


def _rope_adjacent(vv, theta):
    c, s = np.cos(theta)[:, None, :], np.sin(theta)[:, None, :]
    a, b = vv[..., 0::2], vv[..., 1::2]
    out = np.empty_like(vv)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = b * c + a * s
    return out


def _rope_reversed_freqs(vv, theta):
    half = vv.shape[-1] // 2
    th = theta[:, ::-1]
    c, s = np.cos(th)[:, None, :], np.sin(th)[:, None, :]
    v1, v2 = vv[..., :half], vv[..., half:]
    return np.concatenate([v1 * c - v2 * s, v2 * c + v1 * s], axis=-1)


_orig_inv_exact = O._inv_freq_exact


def _inv_freq_no_two(base, hd):
    return _orig_inv_exact(base, 2 * hd)[: hd // 2]       # base^(-i/hd)


def _angles_f64(pos, inv):
    p = np.asarray(pos).astype(np.float64)
    return p[:, None] * np.asarray(inv, dtype=np.float64)[None, :]


def _swiglu_swapped(gate, up, dtype):
    g, u = values(up, dtype), values(gate, dtype)
    with np.errstate(over="ignore"):
        return round_to(g / (1.0 + np.exp(-g)) * u, dtype)


def _swiglu_no_up(gate, up, dtype):
    g = values(gate, dtype)
    with np.errstate(over="ignore"):
        return round_to(g / (1.0 + np.exp(-g)), dtype)


def _swiglu_sigmoid_sign(gate, up, dtype):
    g, u = values(gate, dtype), values(up, dtype)
    with np.errstate(over="ignore"):
        return round_to(g / (1.0 + np.exp(g)) * u, dtype)


def _residual_unrounded(x, r, w, eps, dtype):
    h64 = values(x, dtype) + values(r, dtype)
    return round_to(O._rmsnorm64(h64, values(w, dtype), eps), dtype), round_to(h64, dtype)


_orig_chain = O.decode_chain


def _chain_swaps_q_k(inp, eps, base, dtype):
    d = _orig_chain(inp, eps, base, dtype)
    if d["q"].shape == d["k"].shape:
        d["q"], d["k"] = d["k"], d["q"]
    else:
        d["out"] = d["out"] * 0
    return d


def _qk_norm_after_rope(q, k, pos, base, q_w, k_w, eps, dtype):
    hd = q.shape[-1]
    theta = O.rope_angles(pos, O.rope_inv_freq(base, hd))

    def one(v, w):
        r = O._rotate64(values(v, dtype), theta)
        return round_to(O._rmsnorm64(r, values(w, dtype), eps), dtype)
    return one(q, q_w), (one(k, k_w) if k is not None and k.size else k)


def _silu_no_x(x, dtype):
    v = values(x, dtype)
    with np.errstate(over="ignore"):
        return round_to(1.0 / (1.0 + np.exp(-v)), dtype)


def _embedding_clamps(table, ids, dtype):
    ids = np.clip(np.asarray(ids).astype(np.int64), 0, table.shape[0] - 1)
    return table[ids].copy()


MUTANTS = {
    "rmsnorm_eps_outside_sqrt": ("_rmsnorm64", _eps_outside),
    "rmsnorm_no_weight": ("_rmsnorm64", _no_weight),
    "rmsnorm_mean_over_h_minus_1": ("_rmsnorm64", _mean_n_minus_1),
    "rope_sin_sign": ("_rotate64", _rope_sign),
    "rope_adjacent_pairs": ("_rotate64", _rope_adjacent),
    "rope_frequencies_reversed": ("_rotate64", _rope_reversed_freqs),
    "inv_freq_exponent_without_2": ("_inv_freq_exact", _inv_freq_no_two),
    "angle_product_in_float64": ("rope_angles", _angles_f64),
    "swiglu_gate_and_up_swapped": ("swiglu", _swiglu_swapped),
    "swiglu_without_up": ("swiglu", _swiglu_no_up),
    "swiglu_sigmoid_sign": ("swiglu", _swiglu_sigmoid_sign),
    "residual_norm_of_unrounded_sum": ("residual_rmsnorm", _residual_unrounded),
    "chain_swaps_outputs": ("decode_chain", _chain_swaps_q_k),
    "qk_norm_after_rotation": ("qk_norm_rope", _qk_norm_after_rope),
    "silu_without_x": ("silu", _silu_no_x),
    "embedding_clamps_ids": ("embedding", _embedding_clamps),
}

# ---- the selection model: the install policy, the keys, Algorithm 1 ----------------
from oracle import selection as S   # noqa: E402

_orig_split_words = S.split_words
_orig_rope_slices = S.rope_slices
_orig_generic = S.generic_guard
_orig_h_range = S._norm_h_range
_orig_rn_role = S.rn_role


def _bucket_floor(T):
    b = 0
    while (1 << (b + 1)) <= T:
        b += 1
    return b


def _lookup_last(self, key):
    hit = -1
    for i, g in enumerate(self.guards):
        if g.holds(key):
            hit = i
    return hit


def _split_fits_next_bucket(dtype, H, b):
    n = S.split_slices(dtype, H)
    return n <= S.SPLIT_MAX_SLICES and _orig_split_words(1 << (b + 1), n) <= S.SPLIT_SCRATCH_WORDS


def _rope_slices_floor(dtype, rd, interleaved, n_heads, b, variant):
    s_ = _orig_rope_slices(dtype, rd, interleaved, n_heads, b, variant)
    return max(1, s_ - 1) if s_ > 1 else s_


def _tune_always_fastest(times):
    return min(range(len(times)), key=lambda i: (times[i], i))


def _generic_one_short(key, plan=None):
    g = _orig_generic(key, plan)
    if g.b_lo >= 0 and g.b_hi > g.b_lo:
        return S.Guard(g.key, g.b_lo, g.b_hi - 1, g.h_lo, g.h_hi, g.h_mod)
    return g


def _h_range_shifted(dt, H, fl, res=True):
    r = _orig_h_range(dt, H, fl, res)
    if r is None or r[2] != S.H_MULTIPLE:
        return r
    return r[0], r[1] - 16 // S.elem_size(dt), r[2]


def _rn_role_wide_wave(dtype, H, flags, T, b, res=True):
    v = 16 // S.elem_size(dtype)
    if (flags & S.ALIGN) and H % v == 0 and 128 < H // v <= 256:
        return S.RN_WAVE[4], S.cdiv(T, 4)
    return _orig_rn_role(dtype, H, flags, T, b, res)


def _rn_role_residual_wide(dtype, H, flags, T, b, res=True):
    v = 16 // S.elem_size(dtype)
    if res and (flags & S.ALIGN) and H % v == 0 and 4096 < H // v <= S.WIDE_ROW_VECS:
        return S.RN_WIDE, T
    return _orig_rn_role(dtype, H, flags, T, b, res)


SELECTION_MUTANTS = {
    "bucket_floor_log2": (S, "bucket", _bucket_floor),
    "lookup_last_match": (S.SpecCacheModel, "lookup", _lookup_last),
    "split_scratch_for_the_next_bucket": (S, "split_fits", _split_fits_next_bucket),
    "rope_slices_one_too_few": (S, "rope_slices", _rope_slices_floor),
    "tuning_ignores_the_margin": (S, "tune_choice", _tune_always_fastest),
    "stream_threshold_256_mib": (S, "STREAM_BYTES", 256 << 20),
    "generic_run_one_bucket_short": (S, "generic_guard", _generic_one_short),
    "generic_row_class_one_vector_short": (S, "_norm_h_range", _h_range_shifted),
    "wavefront_rows_up_to_256_vectors": (S, "rn_role", _rn_role_wide_wave),
    "plain_wide_rows_up_to_8192_vectors": (S, "WIDE_PLAIN_VECS", 8 * S.WIDE_LANES),
    "residual_rows_wide_instead_of_split": (S, "rn_role", _rn_role_residual_wide),
    "plain_wide_rows_one_workgroup_each": (S, "WIDE_GRID", 1 << 40),
    "plain_8192_vector_rows_wide_one_bucket_early": (S, "WIDE_PLAIN_BUCKET", 8),
}

_name = os.environ.get("TRI_ORACLE_MUTANT")
if _name in MUTANTS:
    attr, fn = MUTANTS[_name]
    setattr(O, attr, fn)
elif _name:
    obj, attr, val = SELECTION_MUTANTS[_name]
    setattr(obj, attr, val)
