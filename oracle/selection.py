"""Model of the guarded specialization cache (test infrastructure only).

What it models
--------------
* Ordered dispatch, Algorithm 1 of the paper (Sec. 3.2): versions are kept
  in creation order; a call runs the first version whose guards hold; if
  none holds the result is a distinguished MISS; an execution error of the
  selected version is returned as an error and no other version is tried.
* The three runtime paths of Sec. 3.5: a hit runs compiled code; a miss
  returns to the caller, who installs a new version and calls again (the
  paper recompiles here; this library selects among precompiled kernels);
  an error never installs anything.
* Guards are the ones a specialization of these ops depends on: dtype,
  hidden / intermediate sizes, head_dim and head counts, a token-count
  bucket, 16-byte alignment, contiguity, whether the RoPE step carries the
  per-head QK RMSNorm, the RoPE variant (rotary dim, pairing, position
  width, angle source, frequency scaling and its parameters) and the RoPE
  base (captured constants of the version, as source-visible constants are
  in Sec. 3.3).

Guards are equality tests on a packed key, so two versions can never both
match and "first match in creation order" is the unique match.

The install policy (which kernel variant a key selects and how many
workgroups a call launches) is restated here from its specification,
independently of the C++ library; the two must agree bit for bit on every
selection record. Norm rows of up to 128 16-byte vectors take one wavefront
each, longer rows one workgroup each; calls that move at most 320 MiB at the
top of their token bucket use cached SwiGLU loads, larger calls stream SwiGLU
nontemporally.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

# ---- enumerations (the ABI's numeric values) --------------------------------
OP_RMSNORM, OP_RES_RMSNORM, OP_ROPE_QK, OP_SWIGLU, OP_CHAIN, OP_QK_NORM_ROPE = 1, 2, 3, 4, 5, 6
ROPE_OPS = (OP_ROPE_QK, OP_QK_NORM_ROPE, OP_CHAIN)
OP_CHAIN_LAYERS = 7        # records of the several-chains entry point
OP_SILU, OP_ADD, OP_MASKED_FILL, OP_EMBEDDING = 8, 9, 10, 11
ELT_OPS = (OP_SILU, OP_ADD, OP_MASKED_FILL)
SHORT_OPS = ELT_OPS + (OP_EMBEDDING,)
MAX_LAYERS = 1024
DT_F32, DT_BF16 = 0, 1
OK, MISS = 0, 1
E_INVALID, E_UNSUPPORTED, E_FULL, E_NOMEM, E_LAUNCH, E_RUNTIME = -1, -2, -3, -4, -5, -6

RN_SCALAR = 10
RN_WAVE = {1: 11, 2: 12}
RN_BLOCK = {1: 13, 2: 14, 4: 15, 8: 16, 16: 17}
RN_LOOP = 18
RN_WIDE = 19               # 1024-work-item workgroups, a row each, 8 vectors per lane
WIDE_LANES = 1024
WIDE_ROW_VECS = 8 * WIDE_LANES   # the longest row it holds (16-byte vectors)
WIDE_PLAIN_VECS = 7 * WIDE_LANES  # plain rows up to here take it by policy
WIDE_PLAIN_BUCKET = 9             # plain rows up to WIDE_ROW_VECS take it from here
WIDE_GRID = 256                   # plain rows: at most this many workgroups, each
                                  # taking rows b, b + 256, ... (residual: one per row)
RN_SPLIT = 20              # a row over S workgroups of 256, 8 vectors per work-item
SPLIT_SPAN = 8 * 256       # vectors one split workgroup holds
SPLIT_MAX_SLICES = 64      # workgroups per row, at most
SPLIT_HEADER_WORDS = 8     # scratch: header, then T*S slots and T counters (64-bit words)
SPLIT_SCRATCH_WORDS = 1 << 22   # a version's scratch for the top of its bucket, at most
NOALLOC_SCRATCH_BYTES = 1 << 20  # the allocation-free entry point's fixed scratch per GPU
NORM_VARIANTS = (RN_SCALAR, *RN_WAVE.values(), *RN_BLOCK.values(), RN_LOOP, RN_WIDE, RN_SPLIT)
ROPE_SCALAR, ROPE_VEC, ROPE_VEC_I, ROPE_QKN_SCALAR, ROPE_QKN_VEC, ROPE_QKN_VEC_I = \
    30, 31, 32, 33, 34, 35
ROPE_VEC_ROLES = (ROPE_VEC, ROPE_VEC_I, ROPE_QKN_VEC, ROPE_QKN_VEC_I)
SW_SCALAR, SW_FLAT, SW_FLAT_NT, SW_ROWS = 40, 41, 42, 43
CH_FUSED, CH_SEQ = 50, 51
ELT_SCALAR, ELT_FLAT, ELT_FLAT_U2, ELT_ROWS = 60, 61, 62, 63
EMB_SCALAR, EMB_VEC = 70, 71
DECODE_BUCKET_MAX = 6       # buckets up to here are decode sized
BUCKET_MAX = 22             # ceil(log2 T) of the largest T

BLOCK = 256
GRID_CAP = 1 << 20
T_MAX = 1 << 22
H_LIMIT = 1 << 24          # H must be below this
I_LIMIT = 1 << 31          # I must be below this
SPAN_MAX = 2 ** 47         # bytes the rows of one operand may span (a bound on strides)
HD_MAX = 512
HEADS_MAX = 4096
DEFAULT_CAPACITY = 256
MAX_CAPACITY = 4096
FLAG_AUTO_INSTALL = 1
FLAG_JIT = 2               # compiled specializations: same selections, same records
FLAG_GENERIC = 8           # a miss installs a generic (range-guarded) version

ALIGN, CONTIG = 1, 2       # per-op guard flag bits
CHAIN_QK_NORM = 0x40       # chain key flag: the RoPE step has the QK RMSNorm
# RoPE variant bits (key word 3, above the 16-bit rotary dim)
ROPE_INTERLEAVED, ROPE_POS64, ROPE_CACHE = 1, 2, 4
SCALING_NONE, SCALING_LLAMA3 = 0, 1
PLAIN_EXT = dict(rotary_dim=0, interleaved=0, pos_int64=0, scaling=SCALING_NONE, factor=0.0,
                 low_freq_factor=0.0, high_freq_factor=0.0, original_max_pos=0, cos_sin=None,
                 cos_sin_len=0)


def elem_size(dtype: int) -> int:
    return 4 if dtype == DT_F32 else 2


def bucket(T: int) -> int:
    """Smallest b >= 0 with 2^b >= T (T >= 1)."""
    b = 0
    while (1 << b) < T:
        b += 1
    return b


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


def block_of(variant: int) -> int:
    """Work-items per workgroup: 1024 for the wide norm rows, 256 otherwise."""
    return WIDE_LANES if variant == RN_WIDE else BLOCK


def next_pow2(n: int) -> int:
    p = 1
    while p < n:
        p *= 2
    return p


def is_pow2(n: int) -> bool:
    return n > 0 and (n & (n - 1)) == 0


def f32_bits(x: float) -> int:
    return int(np.array([x], dtype=np.float64).astype(np.float32).view(np.uint32)[0])


def _finite(x: float) -> bool:
    return math.isfinite(x)


def _f32(x: float) -> float:
    """The float32 value a C caller passes for x (overflow -> inf)."""
    with np.errstate(over="ignore"):
        return float(np.array([x], dtype=np.float64).astype(np.float32)[0])


def _aligned(es: int, ptrs, strides) -> bool:
    return all(p % 16 == 0 for p in ptrs) and all((s * es) % 16 == 0 for s in strides)


# ---- role policies -----------------------------------------------------------
def split_slices(dtype: int, H: int) -> int:
    """Workgroups per row of the split form: the row's 16-byte vectors in
    spans of SPLIT_SPAN."""
    return cdiv(H // (16 // elem_size(dtype)), SPLIT_SPAN)


def split_words(T: int, S: int) -> int:
    """Scratch words a split call of T rows uses: the header, one slot per
    workgroup, one counter per row."""
    return SPLIT_HEADER_WORDS + T * (S + 1)


def split_fits(dtype: int, H: int, b: int) -> bool:
    """The split form serves rows of at most SPLIT_MAX_SLICES workgroups whose
    version scratch, sized for the top of bucket b, stays within
    SPLIT_SCRATCH_WORDS."""
    S = split_slices(dtype, H)
    return S <= SPLIT_MAX_SLICES and split_words(1 << b, S) <= SPLIT_SCRATCH_WORDS


def rn_role(dtype: int, H: int, flags: int, T: int, b: int,
            res: bool = True) -> Tuple[int, int]:
    """(variant, grid) for residual RMSNorm rows (res) or plain RMSNorm rows
    (b: the token bucket of the key)."""
    v = 16 // elem_size(dtype)
    if not (flags & ALIGN) or H % v:
        return RN_SCALAR, T
    nvec = H // v
    if nvec <= 128:                       # short rows: a wavefront each, 4 per block
        return RN_WAVE[next_pow2(cdiv(nvec, 64))], cdiv(T, 4)
    nb = next_pow2(cdiv(nvec, 256))       # a workgroup per row
    if nb <= 16:
        return RN_BLOCK[nb], T
    if not res and nvec <= WIDE_PLAIN_VECS:  # plain rows: 1024-lane workgroups
        return RN_WIDE, wide_grid(T, res)
    if not res and nvec <= WIDE_ROW_VECS and b >= WIDE_PLAIN_BUCKET:  # the same, past 256 rows
        return RN_WIDE, wide_grid(T, res)
    if split_fits(dtype, H, b):           # several workgroups per row
        return RN_SPLIT, T * split_slices(dtype, H)
    if nvec <= WIDE_ROW_VECS:             # 1024-lane workgroups
        return RN_WIDE, wide_grid(T, res)
    return RN_LOOP, T                     # two passes over memory


def wide_grid(T: int, res: bool) -> int:
    """Workgroups of a wide-row norm launch: one per row for residual rows;
    for plain rows at most WIDE_GRID, each taking every WIDE_GRID-th row."""
    return T if res else min(T, WIDE_GRID)


def rope_role(dtype: int, hd: int, flags: int, T: int, qk_norm: bool = False,
              rd: Optional[int] = None, interleaved: bool = False) -> Tuple[int, int]:
    """Vector path when 16-byte aligned and the rotated span of a head (rd/2
    elements per half for rotate-half pairs, rd for GPT-J pairs) is a
    power-of-two number of 16-byte vectors; with the QK norm the vector path
    also needs rd == hd and at most 64 vectors in that span."""
    rd = hd if rd is None else rd
    v = 16 // elem_size(dtype)
    span = rd if interleaved else rd // 2
    vec = bool(flags & ALIGN) and span % v == 0 and is_pow2(span // v)
    if qk_norm:
        vec = vec and rd == hd and span // v <= 64
    if not vec:
        return (ROPE_QKN_SCALAR if qk_norm else ROPE_SCALAR), T
    if interleaved:
        return (ROPE_QKN_VEC_I if qk_norm else ROPE_VEC_I), T
    return (ROPE_QKN_VEC if qk_norm else ROPE_VEC), T


def rope_slices(dtype: int, rd: int, interleaved: bool, n_heads: int, b: int,
                variant: int) -> int:
    """Workgroups per token of a vector RoPE role at decode sizes: the heads'
    work-item groups (n_heads * cpb lanes) over 256-wide workgroups, at most
    4; one otherwise."""
    if variant not in ROPE_VEC_ROLES or b > DECODE_BUCKET_MAX:
        return 1
    v = 16 // elem_size(dtype)
    cpb = (rd if interleaved else rd // 2) // v
    return max(1, min(4, cdiv(n_heads * cpb, BLOCK)))


def rope_tokens(dtype: int, rd: int, interleaved: bool, n_heads: int, b: int,
                variant: int) -> int:
    """Tokens per workgroup of a vector RoPE role beyond decode sizes: when
    a token's heads fill fewer than 256 lanes (n_heads * cpb), enough
    tokens to fill them, rounded up to a power of two, at most 4; one at
    decode sizes and for the scalar roles."""
    if variant not in ROPE_VEC_ROLES or b <= DECODE_BUCKET_MAX:
        return 1
    v = 16 // elem_size(dtype)
    lanes = n_heads * ((rd if interleaved else rd // 2) // v)
    if lanes >= BLOCK:
        return 1
    return min(4, next_pow2(cdiv(BLOCK, lanes)))


def rope_grid(T: int, slices: int, tokens: int) -> int:
    """Workgroups of a vector RoPE role: T * slices with head slices, else
    ceil(T / tokens)."""
    return T * slices if slices > 1 else cdiv(T, tokens)


STREAM_BYTES = 320 << 20     # calls moving more stream SwiGLU nontemporally


def call_bytes(key) -> int:
    """Bytes a call at the top of the key's token bucket moves, each
    activation read once and each output written once (weights, positions
    and tables left out): SwiGLU 3 T I elements; the chain 4 T H (norm) +
    2 T (nq + nk) hd (RoPE, whole heads) + 3 T I (SwiGLU); 0 for other ops."""
    f = unpack_key(key)
    T, es = 1 << f["bucket"], elem_size(f["dtype"])
    if f["op"] == OP_SWIGLU:
        return 3 * T * f["I"] * es
    if f["op"] == OP_CHAIN:
        return T * es * (4 * f["H"] + 2 * (f["nq"] + f["nk"]) * f["hd"] + 3 * f["I"])
    return 0


def sw_role(dtype: int, I: int, flags: int, stream: bool, T: int) -> Tuple[int, int]:
    """Flat when aligned and contiguous (nontemporal when the call streams,
    call_bytes > STREAM_BYTES, the same as the fused chain's role), vector
    rows when only the rows are aligned, element-wise otherwise."""
    v = 16 // elem_size(dtype)
    if (flags & ALIGN) and (flags & CONTIG):
        nvec = (T * I) // v
        return (SW_FLAT_NT if stream else SW_FLAT), max(1, min(cdiv(nvec, BLOCK), GRID_CAP))
    if (flags & ALIGN) and I % v == 0:
        cb = cdiv(I // v, BLOCK)
        return SW_ROWS, min(T * cb, GRID_CAP)
    return SW_SCALAR, min(cdiv(T * I, BLOCK), GRID_CAP)


def elt_role(dtype: int, W: int, flags: int, b: int, T: int) -> Tuple[int, int]:
    """silu / add / masked_fill: flat vectors when aligned and contiguous
    (beyond decode sizes two per work-item), vector rows when only the rows
    are aligned, element-wise otherwise."""
    v = 16 // elem_size(dtype)
    if (flags & ALIGN) and (flags & CONTIG):
        if b <= DECODE_BUCKET_MAX:
            return ELT_FLAT, max(1, min(cdiv((T * W) // v, BLOCK), GRID_CAP))
        return ELT_FLAT_U2, max(1, min(cdiv((T * W) // v, 2 * BLOCK), GRID_CAP))
    if (flags & ALIGN) and W % v == 0:
        return ELT_ROWS, min(T * cdiv(W // v, BLOCK), GRID_CAP)
    return ELT_SCALAR, min(cdiv(T * W, BLOCK), GRID_CAP)


def emb_role(dtype: int, H: int, flags: int, T: int) -> Tuple[int, int]:
    """One workgroup per output row; vectors when aligned and H % v == 0."""
    v = 16 // elem_size(dtype)
    return (EMB_VEC if (flags & ALIGN) and H % v == 0 else EMB_SCALAR), max(1, min(T, GRID_CAP))


# ---- calls -------------------------------------------------------------------
@dataclasses.dataclass
class Call:
    """One entry call: the op and every argument the guards can see."""
    op: int
    dtype: int
    T: int
    H: int = 0                # RMSNorm hidden size; row width W of the short ops
    I: int = 0
    n_rows: int = 0           # embedding table rows
    ids64: int = 0            # embedding: int64 ids
    value: float = 0.0        # masked_fill value
    hd: int = 0
    nq: int = 0
    nk: int = 0
    eps: float = 1e-6
    base: float = 10000.0
    qk_eps: float = 1e-6     # chain only: epsilon of the QK RMSNorm
    ext: Optional[dict] = None   # RoPE variant (keys of PLAIN_EXT); None = plain
    # addresses (integers) and strides in elements; None = null pointer
    ptr: Dict[str, Optional[int]] = dataclasses.field(default_factory=dict)
    stride: Dict[str, int] = dataclasses.field(default_factory=dict)


@dataclasses.dataclass
class Record:
    op: int = 0
    status: int = 0
    version: int = -1
    variant: int = 0
    n_launches: int = 0
    roles: Tuple[int, int, int] = (0, 0, 0)
    launch: Tuple[Tuple[int, int, int], ...] = ((0, 0, 0), (0, 0, 0), (0, 0, 0))
    key: Tuple[int, ...] = (0, 0, 0, 0, 0, 0)

    def as_tuple(self):
        return (self.op, self.status, self.version, self.variant, self.n_launches,
                tuple(self.roles), tuple(tuple(l) for l in self.launch), tuple(self.key))


def _validate_common(c: Call) -> Optional[int]:
    if c.dtype not in (DT_F32, DT_BF16):
        return E_INVALID
    if c.T < 0:
        return E_INVALID
    if c.T == 0:
        return OK
    if c.T > T_MAX:
        return E_UNSUPPORTED
    return None


def _extent_ok(rows: int, stride: int, width: int, es: int) -> bool:
    """`rows` rows of `width` elements, `stride` elements apart, span
    ((rows - 1) * stride + width) * es bytes; a call is valid only when every
    operand's span is at most SPAN_MAX (a safety rule of this library, not of
    the paper: no buffer is that large, and it keeps the kernels' offsets
    far from int64 overflow)."""
    return ((rows - 1) * stride + width) * es <= SPAN_MAX


def _validate_rn(c: Call, names, strides) -> Optional[int]:
    if c.H < 1:
        return E_INVALID
    if c.H >= H_LIMIT:
        return E_UNSUPPORTED
    if any(c.ptr.get(n) is None for n in names):
        return E_INVALID
    es = elem_size(c.dtype)
    if any(c.ptr[n] % es for n in names):
        return E_INVALID
    if any(c.stride[s] < c.H or not _extent_ok(c.T, c.stride[s], c.H, es) for s in strides):
        return E_INVALID
    eps = _f32(c.eps)
    if not _finite(eps) or eps < 0:
        return E_INVALID
    return None


def rope_ext_of(c: Call) -> dict:
    x = dict(PLAIN_EXT)
    if c.ext:
        x.update(c.ext)
    return x


def _validate_rope(c: Call) -> Optional[int]:
    """Head dim and head counts; the variant fields; pointers and their
    alignment; strides; the angle source."""
    x = rope_ext_of(c)
    if c.hd < 2 or c.hd % 2:
        return E_INVALID
    if c.hd > HD_MAX:
        return E_UNSUPPORTED
    if c.nq < 1 or c.nk < 0:
        return E_INVALID
    if c.nq > HEADS_MAX or c.nk > HEADS_MAX:
        return E_UNSUPPORTED
    rd = x["rotary_dim"]
    if rd != 0 and (rd < 2 or rd % 2 or rd > c.hd):
        return E_INVALID
    if x["interleaved"] not in (0, 1) or x["pos_int64"] not in (0, 1):
        return E_INVALID
    if x["scaling"] not in (SCALING_NONE, SCALING_LLAMA3):
        return E_INVALID
    if c.ptr.get("q") is None or c.ptr.get("pos") is None:
        return E_INVALID
    if c.nk > 0 and c.ptr.get("k") is None:
        return E_INVALID
    if c.ptr["pos"] % (8 if x["pos_int64"] else 4):
        return E_INVALID
    es = elem_size(c.dtype)
    if c.ptr["q"] % es or (c.nk > 0 and c.ptr["k"] % es):
        return E_INVALID
    if c.stride["q"] < c.nq * c.hd or not _extent_ok(c.T, c.stride["q"], c.nq * c.hd, es):
        return E_INVALID
    if c.nk > 0 and (c.stride["k"] < c.nk * c.hd
                     or not _extent_ok(c.T, c.stride["k"], c.nk * c.hd, es)):
        return E_INVALID
    if x["cos_sin"] is not None:
        rdc = rd if rd else c.hd
        if (x["cos_sin"] % 4 or x["cos_sin_len"] < 1
                or not _extent_ok(x["cos_sin_len"], rdc, rdc, 4)
                or x["scaling"] != SCALING_NONE):
            return E_INVALID
        return None
    base = _f32(c.base)
    if not _finite(base) or base <= 1.0:
        return E_INVALID
    if x["scaling"] == SCALING_LLAMA3:
        f, lo, hi = _f32(x["factor"]), _f32(x["low_freq_factor"]), _f32(x["high_freq_factor"])
        if not _finite(f) or f <= 0 or not _finite(lo) or lo <= 0:
            return E_INVALID
        if not _finite(hi) or hi <= lo:
            return E_INVALID
        if x["original_max_pos"] < 1:
            return E_INVALID
    return None


def _validate_qkn(c: Call, eps: float) -> Optional[int]:
    """Head-norm weights: q_w always, k_w when nk > 0; element-aligned."""
    if c.ptr.get("q_w") is None or (c.nk > 0 and c.ptr.get("k_w") is None):
        return E_INVALID
    es = elem_size(c.dtype)
    if c.ptr["q_w"] % es or (c.nk > 0 and c.ptr["k_w"] % es):
        return E_INVALID
    eps = _f32(eps)
    if not _finite(eps) or eps < 0:
        return E_INVALID
    return None


def chain_has_qk_norm(c: Call) -> bool:
    return c.ptr.get("q_w") is not None


def _validate_sw(c: Call) -> Optional[int]:
    if c.I < 1:
        return E_INVALID
    if c.I >= I_LIMIT:
        return E_UNSUPPORTED
    if any(c.ptr.get(n) is None for n in ("gate", "up", "out")):
        return E_INVALID
    es = elem_size(c.dtype)
    if any(c.ptr[n] % es for n in ("gate", "up", "out")):
        return E_INVALID
    if any(c.stride[s] < c.I for s in ("gate", "up", "out")):
        return E_INVALID
    if not all(_extent_ok(c.T, c.stride[s], c.I, es) for s in ("gate", "up", "out")):
        return E_INVALID
    return None


RN_PTRS = ("x", "w", "y")
RN_STRIDES = ("x", "y")
RES_PTRS = ("x", "res", "w", "y", "res_out")
RES_STRIDES = ("x", "res", "y", "res_out")


def _validate_short(c: Call) -> Optional[int]:
    es = elem_size(c.dtype)
    p, s = c.ptr, c.stride
    if c.op == OP_EMBEDDING:
        if c.H < 1 or c.n_rows < 1 or c.ids64 not in (0, 1):
            return E_INVALID
        if c.H >= I_LIMIT:
            return E_UNSUPPORTED
        if any(p.get(n) is None for n in ("table", "ids", "out")):
            return E_INVALID
        if p["table"] % es or p["out"] % es or p["ids"] % (8 if c.ids64 else 4):
            return E_INVALID
        if s["table"] < c.H or s["out"] < c.H:
            return E_INVALID
        if not _extent_ok(c.n_rows, s["table"], c.H, es) or not _extent_ok(c.T, s["out"], c.H, es):
            return E_INVALID
        return None
    names = ("a", "b", "out")
    if c.H < 1:
        return E_INVALID
    if c.H >= I_LIMIT:
        return E_UNSUPPORTED
    if any(p.get(n) is None for n in names):
        return E_INVALID
    if p["a"] % es or p["out"] % es or (c.op != OP_MASKED_FILL and p["b"] % es):
        return E_INVALID
    if any(s[n] < c.H for n in names):
        return E_INVALID
    b_es = 1 if c.op == OP_MASKED_FILL else es
    if (not _extent_ok(c.T, s["a"], c.H, es) or not _extent_ok(c.T, s["b"], c.H, b_es)
            or not _extent_ok(c.T, s["out"], c.H, es)):
        return E_INVALID
    return None


def validate(c: Call) -> Optional[int]:
    """None if the call is valid and non-empty, else its status."""
    st = _validate_common(c)
    if st is not None:
        return st
    if c.op == OP_RMSNORM:
        return _validate_rn(c, RN_PTRS, RN_STRIDES)
    if c.op == OP_RES_RMSNORM:
        return _validate_rn(c, RES_PTRS, RES_STRIDES)
    if c.op == OP_ROPE_QK:
        return _validate_rope(c)
    if c.op == OP_QK_NORM_ROPE:
        st = _validate_rope(c)
        return st if st is not None else _validate_qkn(c, c.eps)
    if c.op == OP_SWIGLU:
        return _validate_sw(c)
    if c.op in SHORT_OPS:
        return _validate_short(c)
    if c.op == OP_CHAIN:
        checks = [lambda: _validate_rn(c, RES_PTRS, RES_STRIDES), lambda: _validate_rope(c)]
        if chain_has_qk_norm(c):
            checks.append(lambda: _validate_qkn(c, c.qk_eps))
        checks.append(lambda: _validate_sw(c))
        for f in checks:
            st = f()
            if st is not None:
                return st
        return None
    return E_INVALID


# ---- guard flags and key ------------------------------------------------------
def rn_flags(c: Call, names, strides) -> int:
    es = elem_size(c.dtype)
    f = 0
    if _aligned(es, [c.ptr[n] for n in names], [c.stride[s] for s in strides]):
        f |= ALIGN
    if all(c.stride[s] == c.H for s in strides):
        f |= CONTIG
    return f


def rope_flags(c: Call, qk_norm: bool = False) -> int:
    """With the QK norm the head-norm weights join the alignment test."""
    es = elem_size(c.dtype)
    ptrs, strides = [c.ptr["q"]], [c.stride["q"]]
    if qk_norm:
        ptrs.append(c.ptr["q_w"])
    contig = c.stride["q"] == c.nq * c.hd
    if c.nk > 0:
        ptrs.append(c.ptr["k"])
        strides.append(c.stride["k"])
        if qk_norm:
            ptrs.append(c.ptr["k_w"])
        contig = contig and c.stride["k"] == c.nk * c.hd
    f = ALIGN if _aligned(es, ptrs, strides) else 0
    return f | (CONTIG if contig else 0)


def sw_flags(c: Call) -> int:
    es = elem_size(c.dtype)
    names = ("gate", "up", "out")
    f = ALIGN if _aligned(es, [c.ptr[n] for n in names], [c.stride[n] for n in names]) else 0
    if all(c.stride[n] == c.I for n in names):
        f |= CONTIG
    return f


def short_flags(c: Call) -> int:
    es = elem_size(c.dtype)
    p, s = c.ptr, c.stride
    if c.op == OP_EMBEDDING:
        return ALIGN if _aligned(es, [p["table"], p["out"]], [s["table"], s["out"]]) else 0
    v = 16 // es
    if c.op == OP_MASKED_FILL:
        al = (_aligned(es, [p["a"], p["out"]], [s["a"], s["out"]])
              and p["b"] % v == 0 and s["b"] % v == 0)
    else:
        al = _aligned(es, [p["a"], p["b"], p["out"]], [s["a"], s["b"], s["out"]])
    contig = all(s[n] == c.H for n in ("a", "b", "out"))
    return (ALIGN if al else 0) | (CONTIG if contig else 0)


def op_flags(c: Call) -> int:
    if c.op == OP_RMSNORM:
        return rn_flags(c, RN_PTRS, RN_STRIDES)
    if c.op == OP_RES_RMSNORM:
        return rn_flags(c, RES_PTRS, RES_STRIDES)
    if c.op == OP_ROPE_QK:
        return rope_flags(c)
    if c.op == OP_QK_NORM_ROPE:
        return rope_flags(c, True)
    if c.op == OP_SWIGLU:
        return sw_flags(c)
    if c.op in SHORT_OPS:
        return short_flags(c)
    qkn = chain_has_qk_norm(c)
    return (rn_flags(c, RES_PTRS, RES_STRIDES) | (rope_flags(c, qkn) << 2)
            | (sw_flags(c) << 4) | (CHAIN_QK_NORM if qkn else 0))


def make_key(c: Call) -> Tuple[int, ...]:
    """Six 64-bit words:
    k0 op | dtype << 8 | bucket << 16 | flags << 24 | base bits << 32;
    k1 H | I << 32;  k2 hd | nq << 16 | nk << 32;
    k3 rotary dim | variant bits << 16 | scaling << 24 | original_max_pos << 32;
    k4 factor bits | low_freq_factor bits << 32;  k5 high_freq_factor bits.
    Unused fields are zero; with a cos/sin cache the base and scaling fields
    are unused."""
    b = bucket(c.T)
    flags = op_flags(c)
    H = c.H if c.op in (OP_RMSNORM, OP_RES_RMSNORM, OP_CHAIN) + SHORT_OPS else 0
    I = c.I if c.op in (OP_SWIGLU, OP_CHAIN) else 0
    hd, nq, nk = (c.hd, c.nq, c.nk) if c.op in ROPE_OPS else (0, 0, 0)
    base_bits, k3, k4, k5 = 0, 0, 0, 0
    if c.op in ROPE_OPS:
        x = rope_ext_of(c)
        rd = x["rotary_dim"] or c.hd
        bits = ((ROPE_INTERLEAVED if x["interleaved"] else 0)
                | (ROPE_POS64 if x["pos_int64"] else 0)
                | (ROPE_CACHE if x["cos_sin"] is not None else 0))
        k3 = rd | (bits << 16)
        if x["cos_sin"] is None:
            base_bits = f32_bits(c.base)
            if x["scaling"] == SCALING_LLAMA3:
                k3 |= (SCALING_LLAMA3 << 24) | ((x["original_max_pos"] & 0xFFFFFFFF) << 32)
                k4 = f32_bits(x["factor"]) | (f32_bits(x["low_freq_factor"]) << 32)
                k5 = f32_bits(x["high_freq_factor"])
    if c.op == OP_EMBEDDING:
        k3 = c.ids64 << 16
    k0 = c.op | (c.dtype << 8) | (b << 16) | (flags << 24) | (base_bits << 32)
    k1 = H | (I << 32)
    k2 = hd | (nq << 16) | (nk << 32)
    return (k0, k1, k2, k3, k4, k5)


def unpack_key(key):
    k0, k1, k2, k3, k4, k5 = key
    return dict(op=k0 & 0xFF, dtype=(k0 >> 8) & 0xFF, bucket=(k0 >> 16) & 0xFF,
                flags=(k0 >> 24) & 0xFF, base_bits=k0 >> 32,
                H=k1 & 0xFFFFFFFF, I=k1 >> 32,
                hd=k2 & 0xFFFF, nq=(k2 >> 16) & 0xFFFF, nk=(k2 >> 32) & 0xFFFF,
                rd=k3 & 0xFFFF, rope_bits=(k3 >> 16) & 0xFF, scaling=(k3 >> 24) & 0xFF,
                orig_max=k3 >> 32, factor_bits=k4 & 0xFFFFFFFF, low_bits=k4 >> 32,
                high_bits=k5 & 0xFFFFFFFF)


def _f32_of_bits(b: int) -> float:
    return float(np.array([b], dtype=np.uint32).view(np.float32)[0])


def key_valid(key) -> bool:
    """A key the entry points could have produced: known op and dtype, bucket
    <= 22, the op's flags, sizes within the argument limits, consistent RoPE
    fields, unused fields zero (the check applied to imported keys)."""
    f = unpack_key(key)
    k0, k1, k2, k3, k4, k5 = key
    op = f["op"]
    if op not in (OP_RMSNORM, OP_RES_RMSNORM, OP_ROPE_QK, OP_SWIGLU, OP_CHAIN,
                  OP_QK_NORM_ROPE) + SHORT_OPS:
        return False
    if f["dtype"] not in (DT_F32, DT_BF16) or f["bucket"] > 22:
        return False
    if f["flags"] > (0x7F if op == OP_CHAIN else 0x3):
        return False
    if op in SHORT_OPS:
        if not (1 <= f["H"] < I_LIMIT) or f["I"] != 0:
            return False
        if op == OP_EMBEDDING and f["flags"] & CONTIG:
            return False
        k3_ok = (1 << 16) if op == OP_EMBEDDING else 0
        return f["base_bits"] == 0 and k2 == 0 and (k3 & ~k3_ok) == 0 and k4 == 0 and k5 == 0
    norm = op in (OP_RMSNORM, OP_RES_RMSNORM, OP_CHAIN)
    sw = op in (OP_SWIGLU, OP_CHAIN)
    if (not (1 <= f["H"] < H_LIMIT)) if norm else f["H"] != 0:
        return False
    if (not (1 <= f["I"] < I_LIMIT)) if sw else f["I"] != 0:
        return False
    if op not in ROPE_OPS:
        return f["base_bits"] == 0 and k2 == 0 and k3 == 0 and k4 == 0 and k5 == 0
    if k2 >> 48:
        return False
    hd, rd = f["hd"], f["rd"]
    if hd < 2 or hd % 2 or hd > HD_MAX or not (1 <= f["nq"] <= HEADS_MAX) or f["nk"] > HEADS_MAX:
        return False
    if rd < 2 or rd % 2 or rd > hd or f["rope_bits"] > 7:
        return False
    if f["rope_bits"] & ROPE_CACHE:
        return (k3 >> 24) == 0 and f["base_bits"] == 0 and k4 == 0 and k5 == 0
    base = _f32_of_bits(f["base_bits"])
    if not (_finite(base) and base > 1.0):
        return False
    if f["scaling"] == SCALING_NONE:
        return (k3 >> 24) == 0 and k4 == 0 and k5 == 0
    if f["scaling"] != SCALING_LLAMA3 or k5 >> 32:
        return False
    fa, lo, hi = (_f32_of_bits(f[n]) for n in ("factor_bits", "low_bits", "high_bits"))
    if not (_finite(fa) and fa > 0 and _finite(lo) and lo > 0 and _finite(hi) and hi > lo):
        return False
    return 1 <= f["orig_max"] < 2 ** 31


# ---- install policy: key -> variants, and per-call launch geometry ---------------
def plan(key, T: int):
    """(variant, roles, launches) for a version with `key`, called with T tokens."""
    f = unpack_key(key)
    op, dt, b, fl = f["op"], f["dtype"], f["bucket"], f["flags"]
    if op in (OP_RMSNORM, OP_RES_RMSNORM):
        v, g = rn_role(dt, f["H"], fl, T, b, op == OP_RES_RMSNORM)
        return v, (0, 0, 0), [(v, g, block_of(v))]
    inter = bool(f["rope_bits"] & ROPE_INTERLEAVED)
    nh = f["nq"] + f["nk"]
    if op in (OP_ROPE_QK, OP_QK_NORM_ROPE):
        v, g = rope_role(dt, f["hd"], fl, T, op == OP_QK_NORM_ROPE, f["rd"], inter)
        if v in ROPE_VEC_ROLES:
            g = rope_grid(T, rope_slices(dt, f["rd"], inter, nh, b, v),
                          rope_tokens(dt, f["rd"], inter, nh, b, v))
        return v, (0, 0, 0), [(v, g, BLOCK)]
    if op == OP_SWIGLU:
        v, g = sw_role(dt, f["I"], fl, call_bytes(key) > STREAM_BYTES, T)
        return v, (0, 0, 0), [(v, g, BLOCK)]
    if op in ELT_OPS:
        v, g = elt_role(dt, f["H"], fl, b, T)
        return v, (0, 0, 0), [(v, g, BLOCK)]
    if op == OP_EMBEDDING:
        v, g = emb_role(dt, f["H"], fl, T)
        return v, (0, 0, 0), [(v, g, BLOCK)]
    rn = rn_role(dt, f["H"], fl & 3, T, b)
    ro = rope_role(dt, f["hd"], (fl >> 2) & 3, T, bool(fl & CHAIN_QK_NORM), f["rd"], inter)
    if ro[0] in ROPE_VEC_ROLES:
        ro = (ro[0], rope_grid(T, rope_slices(dt, f["rd"], inter, nh, b, ro[0]),
                               rope_tokens(dt, f["rd"], inter, nh, b, ro[0])))
    sw = sw_role(dt, f["I"], (fl >> 4) & 3, call_bytes(key) > STREAM_BYTES, T)
    roles = (rn[0], ro[0], sw[0])
    fused = ((fl & 0x3F) == 0x3F
             and (rn[0] in RN_WAVE.values() or rn[0] in RN_BLOCK.values())
             and ro[0] in ROPE_VEC_ROLES
             and sw[0] in (SW_FLAT, SW_FLAT_NT))
    if fused:
        return CH_FUSED, roles, [(CH_FUSED, rn[1] + ro[1] + sw[1], BLOCK)]
    return CH_SEQ, roles, [(rn[0], rn[1], block_of(rn[0])), (ro[0], ro[1], BLOCK),
                           (sw[0], sw[1], BLOCK)]



# ---- install-time tuning (the benchmark-and-keep scheme of Sec. 2) ------------------
# A key has an ordered list of candidate plans: index 0 is the policy's plan
# above, the others are the other kernel variants whose preconditions the
# key guarantees. A tuning cache times every candidate on a call of the
# key's shapes and keeps the fastest; the policy's plan stays unless another
# candidate is faster than TUNE_MARGIN times its time.
FLAG_AUTOTUNE = 4
TUNE_MARGIN = 0.97
SLICE_CHOICES = (1, 2, 4)
SLICE_BUCKET_MAX = 13        # head-slice alternatives up to 8192 tokens
TUNE_SCRATCH_MAX = 4 << 30   # tuning calls with more operand bytes are not timed
TUNE_NONE, TUNE_MEASURED, TUNE_STORED, TUNE_SKIPPED = 0, 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Cand:
    """One candidate plan: the version's variant, the chain's roles, the
    kernel of each launch, the RoPE role's workgroups per token (slices) and
    tokens per workgroup."""
    variant: int
    roles: Tuple[int, int, int]
    kernels: Tuple[int, ...]
    slices: int
    tokens: int = 1


def _geometry_options(S: int, P: int, b: int) -> List[Tuple[int, int]]:
    """(slices, tokens per workgroup) of a vector RoPE role, the policy's
    first. Decode sizes: slice counts 1, 2, 4. Beyond: tokens per workgroup
    1, 2, 4, then (up to bucket 13) 2 and 4 slices of one token."""
    if b <= DECODE_BUCKET_MAX:
        return [(S, 1)] + [(s, 1) for s in SLICE_CHOICES if s != S]
    out = [(1, P)] + [(1, p) for p in SLICE_CHOICES if p != P]
    if b <= SLICE_BUCKET_MAX:
        out += [(2, 1), (4, 1)]
    return out


def _rn_options(dt: int, H: int, fl: int, b: int, standalone: bool,
                res: bool = True) -> List[int]:
    """Norm rows: a row held by one wavefront can also be held by one
    256-lane workgroup (one vector per lane); standalone (the fused chain
    takes only the 256-lane register forms), a row of more than 1024
    vectors held by a 256-lane workgroup can also be held by a 1024-lane
    one, a row of more than 2048 vectors (RN_BLOCK[16]) can also be split
    over two workgroups when its scratch fits, a split row of at most
    WIDE_ROW_VECS vectors can be held by a 1024-lane workgroup and a row
    held by a 1024-lane workgroup can be split when its scratch fits, and
    any row held in registers can take the two-pass loop kernel."""
    P = rn_role(dt, H, fl, 1, b, res)[0]
    if P in (RN_SCALAR, RN_LOOP):
        return [P]
    out = [P]
    if P in RN_WAVE.values():
        out.append(RN_BLOCK[1])
    if standalone:
        if P in (RN_BLOCK[8], RN_BLOCK[16]):
            out.append(RN_WIDE)
            if P == RN_BLOCK[16] and split_words(1 << b, split_slices(dt, H)) <= \
                    SPLIT_SCRATCH_WORDS:
                out.append(RN_SPLIT)
        if P == RN_SPLIT and H // (16 // elem_size(dt)) <= WIDE_ROW_VECS:
            out.append(RN_WIDE)
        if P == RN_WIDE and split_fits(dt, H, b):
            out.append(RN_SPLIT)
        out.append(RN_LOOP)
    return out


def _other(P: int, a: int, b: int) -> List[int]:
    return [P, b if P == a else a]


def candidates(key) -> List[Cand]:
    """The candidate plans of `key`, in the library's order (index 0 is the
    policy's plan).

    * RMSNorm rows: the policy's register layout, the workgroup layout when
      the policy takes a wavefront, the two-pass loop.
    * RoPE with a vector role: the vector kernel at each geometry option
      (_geometry_options), then the scalar kernel.
    * SwiGLU / silu / add / masked_fill, flat: the policy's flat form, the
      other flat form (cached / nontemporal, one / two vectors per
      work-item), vector rows when a row is a whole number of vectors.
    * The fused chain: every combination of norm role options x geometry
      options x SwiGLU flat forms (nested in that order, each list starting
      with the policy's choice), then the three-launch sequence of the
      policy's roles.
    * Every other plan is the only candidate of its key.
    """
    f = unpack_key(key)
    op, dt, b, fl = f["op"], f["dtype"], f["bucket"], f["flags"]
    v = 16 // elem_size(dt)
    z = (0, 0, 0)
    if op in (OP_RMSNORM, OP_RES_RMSNORM):
        return [Cand(r, z, (r,), 1)
                for r in _rn_options(dt, f["H"], fl, b, True, op == OP_RES_RMSNORM)]
    inter = bool(f["rope_bits"] & ROPE_INTERLEAVED)
    nh = f["nq"] + f["nk"]
    if op in (OP_ROPE_QK, OP_QK_NORM_ROPE):
        qkn = op == OP_QK_NORM_ROPE
        P = rope_role(dt, f["hd"], fl, 1, qkn, f["rd"], inter)[0]
        if P not in ROPE_VEC_ROLES:
            return [Cand(P, z, (P,), 1)]
        S = rope_slices(dt, f["rd"], inter, nh, b, P)
        Pt = rope_tokens(dt, f["rd"], inter, nh, b, P)
        sc = ROPE_QKN_SCALAR if qkn else ROPE_SCALAR
        return [Cand(P, z, (P,), s, t) for s, t in _geometry_options(S, Pt, b)] + \
            [Cand(sc, z, (sc,), 1)]
    if op == OP_SWIGLU:
        P = sw_role(dt, f["I"], fl, call_bytes(key) > STREAM_BYTES, 1)[0]
        opts = [P]
        if P in (SW_FLAT, SW_FLAT_NT):
            opts = _other(P, SW_FLAT, SW_FLAT_NT) + ([SW_ROWS] if f["I"] % v == 0 else [])
        return [Cand(w, z, (w,), 1) for w in opts]
    if op in ELT_OPS:
        P = elt_role(dt, f["H"], fl, b, 1)[0]
        opts = [P]
        if P in (ELT_FLAT, ELT_FLAT_U2):
            opts = _other(P, ELT_FLAT, ELT_FLAT_U2) + ([ELT_ROWS] if f["H"] % v == 0 else [])
        return [Cand(e, z, (e,), 1) for e in opts]
    if op == OP_EMBEDDING:
        P = emb_role(dt, f["H"], fl, 1)[0]
        return [Cand(P, z, (P,), 1)]
    variant, roles, _ = plan(key, 1)
    rn, ro, sw = roles
    S = rope_slices(dt, f["rd"], inter, nh, b, ro)
    Pt = rope_tokens(dt, f["rd"], inter, nh, b, ro)
    seq = Cand(CH_SEQ, roles, roles, S, Pt)
    if variant != CH_FUSED:
        return [seq]
    out = []
    for r in _rn_options(dt, f["H"], fl & 3, b, False):
        for s, t in _geometry_options(S, Pt, b):
            for w in _other(sw, SW_FLAT, SW_FLAT_NT):
                out.append(Cand(CH_FUSED, (r, ro, w), (CH_FUSED,), s, t))
    return out + [seq]


def grid_of(variant: int, dt: int, T: int, width: int, slices: int = 1, tokens: int = 1,
            res: bool = True) -> int:
    """Workgroups a kernel variant launches for T tokens (width: SwiGLU's I,
    a short op's row width). Wavefront norm rows: 4 rows per workgroup;
    plain wide norm rows (res False): wide_grid; other norm and RoPE
    kernels: one workgroup per row or token (vector RoPE:
    times its slices, or per `tokens` tokens); flat kernels: one 16-byte vector per work-item (two
    for ELT_FLAT_U2); row kernels: the row's vectors over 256 work-items,
    per row; element-wise kernels: one element per work-item. Flat, row and
    element-wise grids are capped at GRID_CAP (grid-stride beyond)."""
    v = 16 // elem_size(dt)
    if variant in RN_WAVE.values():
        return cdiv(T, 4)
    if variant == RN_SPLIT:               # width: the row width H
        return T * split_slices(dt, width)
    if variant == RN_WIDE:
        return wide_grid(T, res)
    if variant in (RN_SCALAR, RN_LOOP, ROPE_SCALAR, ROPE_QKN_SCALAR) or \
            variant in RN_BLOCK.values():
        return T
    if variant in ROPE_VEC_ROLES:
        return rope_grid(T, slices, tokens)
    if variant in (SW_FLAT, SW_FLAT_NT, ELT_FLAT):
        return max(1, min(cdiv((T * width) // v, BLOCK), GRID_CAP))
    if variant == ELT_FLAT_U2:
        return max(1, min(cdiv((T * width) // v, 2 * BLOCK), GRID_CAP))
    if variant in (EMB_VEC, EMB_SCALAR):
        return max(1, min(T, GRID_CAP))
    if variant in (SW_ROWS, ELT_ROWS):
        return min(T * cdiv(width // v, BLOCK), GRID_CAP)
    if variant in (SW_SCALAR, ELT_SCALAR):
        return min(cdiv(T * width, BLOCK), GRID_CAP)
    raise ValueError(variant)


def cand_plan(key, c: Cand, T: int):
    """(variant, roles, launches) of candidate c for a call with T tokens, in
    the form plan() returns."""
    f = unpack_key(key)
    dt = f["dtype"]

    def width(kv):        # the norm rows' H, a short op's W, else SwiGLU's I
        return f["H"] if f["op"] in SHORT_OPS or kv in NORM_VARIANTS else f["I"]
    if c.variant == CH_FUSED:
        g = (grid_of(c.roles[0], dt, T, f["H"])
             + grid_of(c.roles[1], dt, T, f["I"], c.slices, c.tokens)
             + grid_of(c.roles[2], dt, T, f["I"]))
        return CH_FUSED, c.roles, [(CH_FUSED, g, BLOCK)]
    res = f["op"] != OP_RMSNORM           # the chain's norm role is residual
    launches = [(kv, grid_of(kv, dt, T, width(kv), c.slices, c.tokens) if kv in ROPE_VEC_ROLES
                 else grid_of(kv, dt, T, width(kv), res=res), block_of(kv)) for kv in c.kernels]
    return c.variant, c.roles, launches


def tune_tokens(key) -> int:
    """Tokens of the tuning call: the top of the key's bucket."""
    return 1 << unpack_key(key)["bucket"]


def _tune_stride(width: int, fl: int, v: int) -> int:
    """Row stride of a tuning operand: the width when contiguous, else the
    next multiple of the vector width above it (aligned) or width + 1."""
    if fl & CONTIG:
        return width
    return cdiv(width + 1, v) * v if fl & ALIGN else width + 1


def tune_operand_bytes(key) -> int:
    """Bytes of the operands of the tuning call (T = tune_tokens(key), row
    strides by _tune_stride, weights and tables once)."""
    f = unpack_key(key)
    op, dt, fl = f["op"], f["dtype"], f["flags"]
    es = elem_size(dt)
    v = 16 // es
    T = tune_tokens(key)
    H, I = f["H"], f["I"]

    def norm(fl2, res):
        return (4 if res else 2) * T * _tune_stride(H, fl2, v) * es + H * es

    def rope(fl2, qkn):
        hd, nq, nk = f["hd"], f["nq"], f["nk"]
        n = T * _tune_stride(nq * hd, fl2, v) * es
        if nk:
            n += T * _tune_stride(nk * hd, fl2, v) * es
        n += T * (8 if f["rope_bits"] & ROPE_POS64 else 4)
        if qkn:
            n += hd * es * (2 if nk else 1)
        if f["rope_bits"] & ROPE_CACHE:
            n += f["rd"] * 4
        return n

    def swiglu(fl2):
        return 3 * T * _tune_stride(I, fl2, v) * es

    if op in (OP_RMSNORM, OP_RES_RMSNORM):
        return norm(fl, op == OP_RES_RMSNORM)
    if op in (OP_ROPE_QK, OP_QK_NORM_ROPE):
        return rope(fl, op == OP_QK_NORM_ROPE)
    if op == OP_SWIGLU:
        return swiglu(fl)
    if op in ELT_OPS:
        s = _tune_stride(H, fl, v)
        n = 2 * T * s * es
        if op == OP_ADD:
            n += T * s * es
        elif op == OP_MASKED_FILL:
            n += T * s
        return n
    if op == OP_EMBEDDING:
        return 0
    return norm(fl & 3, True) + rope((fl >> 2) & 3, bool(fl & CHAIN_QK_NORM)) + \
        swiglu((fl >> 4) & 3)


def tune_choice(times: List[float]) -> int:
    """Index of the kept candidate given each candidate's time: the fastest
    (the first of equals), unless it is not faster than TUNE_MARGIN times
    candidate 0's time, in which case the policy's plan (0) stays."""
    best = min(range(len(times)), key=lambda i: (times[i], i))
    keep = np.float32(times[best]) < np.float32(TUNE_MARGIN) * np.float32(times[0])
    return best if keep else 0

# ---- guards: exact and generic versions ------------------------------------------
# The paper's guards can hold across many concrete inputs (a rank check and a
# shape bound, Sec. 3.2, Fig. 4), so versions may overlap and Algorithm 1's
# first match in creation order decides. An exact version matches its key
# only. A generic version matches every key equal to its own except that
#  * the token bucket may lie anywhere in [b_lo, b_hi], the widest run of
#    buckets around its own over which the install policy's plan (kernels,
#    roles, RoPE geometry) does not change;
#  * for norm rows held by one wavefront or one workgroup (or the scalar
#    kernel) H may lie anywhere in [h_lo, h_hi] within its divisibility
#    class: the row lengths the same kernel serves, for every bucket.
# Plans that split norm rows (their scratch is sized by H and the bucket) get
# exact versions only. Plan equality is candidate-0 equality.
H_ANY, H_MULTIPLE, H_RAGGED = 0, 1, 2        # divisibility classes of a generic H range


@dataclasses.dataclass(frozen=True)
class Guard:
    """What a version matches: `key` exactly (b_lo < 0), or generic ranges."""
    key: Tuple[int, ...]
    b_lo: int = -1
    b_hi: int = -1
    h_lo: int = 0          # 0: H must equal the key's
    h_hi: int = 0
    h_mod: int = H_ANY

    def holds(self, key) -> bool:
        key = tuple(key)
        if self.b_lo < 0:
            return key == self.key
        bucket_bits = 0xFF << 16
        if key[0] & ~bucket_bits != self.key[0] & ~bucket_bits:
            return False
        if not self.b_lo <= (key[0] >> 16) & 0xFF <= self.b_hi:
            return False
        if self.h_lo:                      # word 1: H in the low half, I in the high half
            if key[1] >> 32 != self.key[1] >> 32:
                return False
            H = key[1] & 0xFFFFFFFF
            v = 16 // elem_size((self.key[0] >> 8) & 0xFF)
            if not self.h_lo <= H <= self.h_hi:
                return False
            if (self.h_mod == H_MULTIPLE and H % v) or (self.h_mod == H_RAGGED and H % v == 0):
                return False
        elif key[1] != self.key[1]:
            return False
        return key[2:] == self.key[2:]


def _with_bucket(key, b: int):
    k = list(key)
    k[0] = (k[0] & ~(0xFF << 16)) | (b << 16)
    return tuple(k)


def _norm_h_range(dt: int, H: int, fl: int, res: bool = True):
    """(h_lo, h_hi, h_mod) of the rows the norm kernel chosen for H serves at
    every bucket, or None when the choice depends on the bucket (residual
    rows beyond 4096 vectors, plain rows beyond 8192)."""
    v = 16 // elem_size(dt)
    if not fl & ALIGN:
        return 1, H_LIMIT - 1, H_ANY
    if H % v:
        return 1, H_LIMIT - 1, H_RAGGED
    n = H // v
    for lo, hi in ((1, 64), (65, 128), (129, 256), (257, 512), (513, 1024), (1025, 2048),
                   (2049, 4096)) + (() if res else ((4097, WIDE_PLAIN_VECS),)):
        if lo <= n <= hi:
            return lo * v, hi * v, H_MULTIPLE
    return None


def generic_guard(key, plan=None) -> Guard:
    """The guard of the generic version a miss on `key` installs, running
    `plan` (default: the policy's plan): the widest run of token buckets
    around the key's over which the policy keeps its plan and, for norm rows
    held by one wavefront or workgroup, the row lengths that kernel serves.
    A version whose plan splits norm rows keeps only the buckets whose
    scratch fits: its scratch is sized for the top of the run, at most
    SPLIT_SCRATCH_WORDS (when the policy itself splits, the run already ends
    there; a tuned split choice clamps it); and it matches only its own
    row length (the scratch is sized by the row's slice count)."""
    P = candidates(key)[0]
    f = unpack_key(key)
    b = f["bucket"]
    lo = b
    while lo > 0 and candidates(_with_bucket(key, lo - 1))[0] == P:
        lo -= 1
    hi = b
    while hi < BUCKET_MAX and candidates(_with_bucket(key, hi + 1))[0] == P:
        hi += 1
    run = plan if plan is not None else P
    splits = RN_SPLIT in run.kernels or RN_SPLIT in run.roles
    if splits:
        while hi > b and not split_fits(f["dtype"], f["H"], hi):
            hi -= 1
    h = None
    if f["op"] in (OP_RMSNORM, OP_RES_RMSNORM) and not splits:
        h = _norm_h_range(f["dtype"], f["H"], f["flags"], f["op"] == OP_RES_RMSNORM)
    if h is None:
        return Guard(tuple(key), lo, hi)
    return Guard(tuple(key), lo, hi, *h)


# ---- the cache -----------------------------------------------------------------
@dataclasses.dataclass
class Stats:
    calls: int = 0
    hits: int = 0
    misses: int = 0
    errors: int = 0
    empty: int = 0
    installs: int = 0


class SpecCacheModel:
    """Ordered versions, Algorithm 1 lookup, miss / install / error paths."""

    def __init__(self, capacity: int = 0, flags: int = 0, timer=None):
        """timer(key, index, cand) -> time of candidate `index` on the tuning
        call; used by a tuning cache (FLAG_AUTOTUNE) for keys with several
        candidates."""
        if capacity < 0 or capacity > MAX_CAPACITY or \
                flags & ~(FLAG_AUTO_INSTALL | FLAG_JIT | FLAG_AUTOTUNE | FLAG_GENERIC):
            raise ValueError("invalid cache parameters")
        self.capacity = capacity or DEFAULT_CAPACITY
        self.flags = flags
        self.timer = timer
        self.versions: List[Tuple[int, ...]] = []   # the key each version was made for
        self.guards: List[Guard] = []
        self.choice: List[int] = []        # candidate index per version
        self.tuned: List[int] = []         # TUNE_* per version
        self.version_hits: List[int] = []
        self.last_miss: Optional[Tuple[Tuple[int, ...], int]] = None
        self.stats = Stats()
        self.last = Record()
        # launch_fails: set of global launch ordinals (0-based) that fail,
        # mirroring fault injection in the host test double.
        self.launch_fails = set()
        self.launch_count = 0

    def lookup(self, key) -> int:
        """Algorithm 1's scan: index of the first version whose guards hold."""
        for i, g in enumerate(self.guards):
            if g.holds(key):
                return i
        return -1

    def _launch(self, launches) -> int:
        for _ in launches:
            n = self.launch_count
            self.launch_count += 1
            if n in self.launch_fails:
                return E_LAUNCH
        return OK

    def call(self, c: Call) -> int:
        self.stats.calls += 1
        rec = Record(op=c.op)
        st = validate(c)
        if st is not None:
            rec.status = st
            self.last = rec
            if st == OK:
                self.stats.empty += 1
            else:
                self.stats.errors += 1
            return st
        key = make_key(c)
        rec.key = key
        i = self.lookup(key)
        auto = False
        if i < 0:
            self.stats.misses += 1
            self.last_miss = (key, c.T)
            if not (self.flags & FLAG_AUTO_INSTALL):
                rec.status = MISS
                self.last = rec
                return MISS
            st = self._install(key, generic=bool(self.flags & FLAG_GENERIC))
            if st < 0:
                rec.status = st
                self.last = rec
                return st
            i = self.lookup(key)
            auto = True
        variant, roles, launches = self.version_plan(i, c.T)
        rec.version, rec.variant, rec.roles = i, variant, roles
        rec.n_launches = len(launches)
        rec.launch = tuple(launches) + ((0, 0, 0),) * (3 - len(launches))
        st = self._launch(launches)
        rec.status = st
        self.last = rec
        if st < 0:
            if not auto:
                self.stats.errors += 1
            return st
        if not auto:
            self.stats.hits += 1
            self.version_hits[i] += 1
        return OK

    def call_layers(self, calls: List[Call]) -> int:
        """Several decode chains in one entry call: validate and look up every
        layer first (nothing installed or launched if one fails or, without
        auto-install, misses), then launch them in order. One call in the
        statistics; a hit counts a hit on every layer's version."""
        self.stats.calls += 1
        rec = Record(op=OP_CHAIN_LAYERS)

        def done(st):
            rec.status = st
            self.last = rec
            return st
        if len(calls) > MAX_LAYERS:
            self.stats.errors += 1
            return done(E_INVALID)
        keys, vis = [], []
        first_miss, last = None, None
        for i, c in enumerate(calls):
            st = validate(c)
            if st == OK:
                keys.append(None)
                vis.append(None)
                continue
            if st is not None:
                self.stats.errors += 1
                return done(st)
            k = make_key(c)
            keys.append(k)
            vis.append(self.lookup(k))
            if vis[-1] < 0 and first_miss is None:
                first_miss = i
            last = i
        if last is None:
            self.stats.empty += 1
            return done(OK)
        missed = first_miss is not None
        if missed:
            self.stats.misses += 1
            self.last_miss = (keys[first_miss], calls[first_miss].T)
            rec.key = keys[first_miss]
            if not (self.flags & FLAG_AUTO_INSTALL):
                return done(MISS)
            for i in range(first_miss, last + 1):
                if vis[i] is not None and vis[i] < 0:
                    # an earlier layer's generic install may already cover it
                    st = self._install(keys[i], generic=bool(self.flags & FLAG_GENERIC))
                    if st < 0:
                        return done(st)
                    vis[i] = self.lookup(keys[i])
        total = 0
        for i, c in enumerate(calls):
            if vis[i] is None:
                continue
            variant, roles, launches = self.version_plan(vis[i], c.T)
            st = self._launch(launches)
            total += len(launches)
            if st < 0 or i == last:
                rec = Record(op=OP_CHAIN_LAYERS, status=st, version=vis[i], variant=variant,
                             n_launches=total, roles=roles,
                             launch=tuple(launches) + ((0, 0, 0),) * (3 - len(launches)),
                             key=keys[i])
                self.last = rec
            if st < 0:
                if not missed:
                    self.stats.errors += 1
                return st
        if not missed:
            self.stats.hits += 1
            for v in vis:
                if v is not None:
                    self.version_hits[v] += 1
        return OK

    def version_plan(self, i: int, T: int):
        """(variant, roles, launches) of version i for a call with T tokens."""
        key = self.versions[i]
        return cand_plan(key, candidates(key)[self.choice[i]], T)

    def _install(self, key, candidate: int = -1, generic: bool = False) -> int:
        """Install `key` with candidate plan `candidate` (-1: tuned on a
        tuning cache, else the policy's plan), as a generic version when
        `generic`. A key some version already matches adds nothing: a version
        appended behind it could never be selected."""
        if self.lookup(key) >= 0:
            return OK
        cands = candidates(key)
        if candidate < -1 or candidate >= len(cands):
            return E_INVALID
        if len(self.versions) >= self.capacity:
            return E_FULL
        choice, tuned = max(candidate, 0), TUNE_NONE
        if candidate < 0 and self.flags & FLAG_AUTOTUNE and len(cands) > 1:
            if tune_operand_bytes(key) > TUNE_SCRATCH_MAX:
                tuned = TUNE_SKIPPED
            else:
                choice = tune_choice([self.timer(key, j, c) for j, c in enumerate(cands)])
                tuned = TUNE_MEASURED
        self.versions.append(key)
        self.guards.append(generic_guard(key, cands[choice]) if generic else Guard(tuple(key)))
        self.choice.append(choice)
        self.tuned.append(tuned)
        self.version_hits.append(0)
        self.stats.installs += 1
        return OK

    def install_key(self, key, candidate: int = -1) -> int:
        """A key installed directly (tri_spec_install_key)."""
        if not key_valid(tuple(key)):
            return E_INVALID
        return self._install(tuple(key), candidate)

    def import_keys(self, keys) -> Tuple[int, int]:
        """Install `keys` in order (status, keys processed); a malformed key
        stops with E_INVALID."""
        for i, k in enumerate(keys):
            if not key_valid(tuple(k)):
                return E_INVALID, i
            st = self._install(tuple(k))
            if st < 0:
                return st, i
        return OK, len(keys)

    def install_last_miss(self) -> Tuple[int, Optional[Record]]:
        if self.last_miss is None:
            return E_INVALID, None
        key, T = self.last_miss
        st = self._install(key, generic=bool(self.flags & FLAG_GENERIC))
        if st < 0:
            return st, None
        variant, roles, launches = self.version_plan(self.lookup(key), T)
        rec = Record(op=key[0] & 0xFF, status=OK, version=self.lookup(key),
                     variant=variant, n_launches=len(launches), roles=roles,
                     launch=tuple(launches) + ((0, 0, 0),) * (3 - len(launches)),
                     key=key)
        return OK, rec
