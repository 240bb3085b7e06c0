"""tri: guarded dispatch of short LLM decode kernels on AMD MI355X (gfx950).

A thin binding over libtri's C ABI (include/tri.h). Every call marshals
torch tensors into pointers, element strides and the current HIP stream,
and makes ONE native entry call; guard evaluation, version lookup, argument
preparation, the launch and all arithmetic happen in libtri and its gfx950
kernels. On TRI_MISS the binding asks the library to install a version for
the missed key and calls again -- the paper's miss path (Sec. 3.5), with
"compile" replaced by selecting a precompiled kernel variant.

PyTorch is used for device memory and streams only. There is no fallback:
if libtri.so is missing, importing this package raises.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional, Tuple

import torch

from . import _lib as L
from ._lib import (AUTO_INSTALL, BF16, E_FULL, E_INVALID, E_LAUNCH, E_NOMEM, E_RUNTIME,
                   E_UNSUPPORTED, F32, MISS, OK, ROPE_SCALING_LLAMA3, ROPE_SCALING_NONE,
                   ChainArgs, RopeExt, Selection, Stats, VersionInfo)

__all__ = ["SpecCache", "Graph", "TriError", "dtype_code", "rope_ext", "Selection", "Stats",
           "ChainArgs", "RopeExt", "OK", "MISS", "E_INVALID", "E_UNSUPPORTED", "E_FULL",
           "E_NOMEM", "E_LAUNCH", "E_RUNTIME", "F32", "BF16", "AUTO_INSTALL"]

_dll = L.load()


class TriError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        name = _dll.tri_status_str(status).decode()
        super().__init__(f"{what}: {name} ({status})" if what else f"{name} ({status})")


_DT = {torch.float32: F32, torch.bfloat16: BF16}


def dtype_code(dt: torch.dtype) -> int:
    try:
        return _DT[dt]
    except KeyError:
        raise TypeError(f"unsupported dtype {dt} (float32 or bfloat16)") from None


def rope_ext(rotary_dim: int = 0, interleaved: bool = False, pos_int64: bool = False,
             scaling: Optional[dict] = None, cos_sin: Optional[torch.Tensor] = None) -> RopeExt:
    """A tri_rope_ext: rotary_dim (0 = head_dim), GPT-J pairs, int64 positions,
    Llama-3 scaling (dict with factor, low_freq_factor, high_freq_factor,
    original_max_pos) or a float32 cos/sin cache [n, rotary_dim]."""
    x = RopeExt()
    x.rotary_dim = rotary_dim
    x.interleaved = int(interleaved)
    x.pos_int64 = int(pos_int64)
    if scaling is not None:
        x.scaling = ROPE_SCALING_LLAMA3
        x.factor = scaling["factor"]
        x.low_freq_factor = scaling["low_freq_factor"]
        x.high_freq_factor = scaling["high_freq_factor"]
        x.original_max_pos = scaling["original_max_pos"]
    if cos_sin is not None:
        if cos_sin.dtype != torch.float32 or cos_sin.dim() != 2 or not cos_sin.is_contiguous():
            raise ValueError("cos_sin: contiguous float32 [n, rotary_dim] expected")
        x.cos_sin = cos_sin.data_ptr()
        x.cos_sin_len = cos_sin.shape[0]
        # The struct holds only the table's address: keep the tensor alive as
        # long as the struct, and remember its width and device for the
        # checks of each call that uses it (_check_cos_sin).
        x._cos_sin = cos_sin
    return x


def _check_cos_sin(ext: Optional[RopeExt], hd: int, dev: int) -> None:
    """A cos/sin table must be on the cache's device and exactly rd floats
    wide (rd = rotary_dim, or hd when 0): the kernels read rd floats of a
    row through the bare address, so a narrower table would be read past
    its end."""
    if ext is None or not ext.cos_sin:
        return
    t = getattr(ext, "_cos_sin", None)
    if t is None:
        raise ValueError("cos_sin: build the variant with rope_ext(cos_sin=...) so the "
                         "table's width and device can be checked")
    rd = ext.rotary_dim or hd
    _on(t, "cos_sin", dev)
    if t.shape[1] != rd:
        raise ValueError(f"cos_sin: expected rows of {rd} floats (rotary_dim), "
                         f"got {tuple(t.shape)}")


# The raw handle of a device's current stream, without building a Stream
# object (torch.cuda.current_stream() costs microseconds per call).
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream_ptr(stream, device: int = -1) -> Optional[int]:
    """hipStream_t of `stream`, or of the current stream of `device` (the
    current device when -1); None for the null stream."""
    if stream is not None:
        return stream.cuda_stream or None
    if device < 0:
        device = torch.cuda.current_device()
    if _raw_stream is not None:
        return _raw_stream(device) or None
    return torch.cuda.current_stream(device).cuda_stream or None


def _rows(t: torch.Tensor, name: str, W: int) -> int:
    """Row stride (elements) of a [T, W] tensor with unit inner stride (the
    caller has checked the shape); a single row reports at least W."""
    st = t.stride()
    if st[0] == W and st[1] == 1:
        return W
    sh = t.shape
    if sh[1] > 1 and st[1] != 1:
        raise ValueError(f"{name}: inner stride must be 1")
    return st[0] if sh[0] > 1 else max(st[0], sh[1])


def _tokens(t: torch.Tensor, name: str, nh: int, hd: int) -> int:
    """Token stride (elements) of a [T, nh, hd] tensor with heads packed (the
    caller has checked the shape); a single token reports at least nh * hd."""
    st = t.stride()
    if st[0] == nh * hd and st[1] == hd and st[2] == 1:
        return nh * hd
    sh = t.shape
    if (hd > 1 and st[2] != 1) or (nh > 1 and st[1] != hd):
        raise ValueError(f"{name}: heads must be packed (stride {hd}) with unit inner stride")
    return st[0] if sh[0] > 1 else max(st[0], nh * hd)


def _on(t: torch.Tensor, name: str, dev: int) -> None:
    """`t` must live on GPU `dev`, the device the cache is bound to: the C
    entry points take bare device addresses, and a kernel handed a host
    address or another GPU's memory would fault instead of failing a check."""
    if t.get_device() != dev:
        where = "the CPU" if t.device.type == "cpu" else str(t.device)
        raise ValueError(f"{name}: tensor on {where}, expected cuda:{dev} (the cache's device)")


def _dims(t: torch.Tensor, name: str, n: int, dev: int) -> tuple:
    """The shape of `t`, which must have n dimensions and live on GPU `dev`."""
    sh = t.shape
    if len(sh) != n:
        raise ValueError(f"{name}: expected {n} dims, got {tuple(sh)}")
    _on(t, name, dev)
    return sh


def _like(t: torch.Tensor, name: str, shape, dtype, dev: int) -> None:
    """`t` must have exactly `shape` and `dtype` and live on GPU `dev`: the
    kernels touch T rows of the given width through it, and only the tensor
    knows its extent."""
    if t.shape != shape or t.dtype != dtype:
        raise ValueError(f"{name}: expected {tuple(shape)} {dtype}, got {tuple(t.shape)} {t.dtype}")
    _on(t, name, dev)


def _vector(t: torch.Tensor, name: str, n: int, dtype, dev: int) -> None:
    """A weight: n contiguous elements of `dtype` on GPU `dev`."""
    if t.shape != (n,) or t.dtype != dtype or (n > 1 and t.stride(0) != 1):
        raise ValueError(f"{name}: expected a contiguous ({n},) {dtype} tensor, "
                         f"got {tuple(t.shape)} {t.dtype}")
    _on(t, name, dev)


class Graph:
    """A captured decode step (tri_graph); destroy before its cache."""

    def __init__(self, handle: C.c_void_p, cache: "SpecCache"):
        self._g = handle
        self._cache = cache          # keeps the cache alive while the graph lives

    @property
    def launch_count(self) -> int:
        return _dll.tri_graph_launch_count(self._g)

    def launch(self, stream=None) -> None:
        st = _dll.tri_graph_launch(self._g, _stream_ptr(stream, self._cache._dev))
        if st != OK:
            raise TriError(st, "tri_graph_launch")

    def close(self) -> None:
        if self._g:
            _dll.tri_graph_destroy(self._g)
            self._g = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Prepared:
    """One op call of a cache marshalled once (SpecCache.prepare): calling it
    issues the same entry call again -- same tensors, sizes and scalars -- on
    the given stream or the device's current one, without the binding's
    shape checks and argument conversion. The tensors it was made from stay
    alive with it: their contents may change between calls, their storage
    must not. A MISS installs and calls again, as the ordinary method does;
    an error raises TriError."""

    __slots__ = ("_cache", "_what", "_fn", "_raw", "_args", "_cargs", "_max_misses", "result")

    def __init__(self, cache: "SpecCache", what: str, fn, args, max_misses: int, result):
        self._cache = cache
        self._what = what
        self._fn = fn
        self._args = args                      # without the trailing stream
        self._max_misses = max_misses
        # every argument as its own ctypes object, for a call through a
        # prototype-free pointer to the same function (no per-call conversion)
        types = fn.argtypes[1:-1]
        self._cargs = (C.c_void_p(cache._h.value),) + tuple(
            t(a) if isinstance(a, (int, float)) else a     # None (NULL), byref(...) as they are
            for t, a in zip(types, args))
        self._raw = C.cast(fn, C.CFUNCTYPE(C.c_int))
        self.result = result

    def __call__(self, stream=None):
        cache = self._cache
        if not cache._h:
            raise TriError(E_INVALID, f"{self._what}: the cache is closed")
        s = _stream_ptr(stream, cache._dev)
        st = self._raw(*self._cargs, C.c_void_p(s))
        if st == MISS:
            cache._call(self._what, self._fn, *self._args, s, max_misses=self._max_misses)
        elif st != OK:
            raise TriError(st, self._what)
        return self.result


class SpecCache:
    """One native specialization cache (bound to the current device)."""

    def __init__(self, capacity: int = 0, auto_install: bool = False, jit: bool = False,
                 code_dir: Optional[str] = None, autotune: bool = False,
                 generic: bool = False, resident_args: bool = False):
        """jit: installs compile key-specialized kernels with hipRTC; autotune:
        installs time the key's candidate plans and keep the fastest; code_dir:
        a directory of compiled code objects and tuning results shared across
        processes; generic: a miss installs a generic version that also
        serves the token buckets (and norm row lengths) with the same plan;
        resident_args: fused-chain launches at decode sizes take their
        argument block from a table in device memory (written on the first
        call with that block) instead of kernel arguments."""
        h = C.c_void_p()
        st = _dll.tri_spec_cache_create(C.byref(h), capacity,
                                        (AUTO_INSTALL if auto_install else 0)
                                        | (L.JIT if jit else 0)
                                        | (L.AUTOTUNE if autotune else 0)
                                        | (L.GENERIC if generic else 0)
                                        | (L.RESIDENT_ARGS if resident_args else 0))
        if st != OK:
            raise TriError(st, "tri_spec_cache_create")
        self._h = h
        self._dev = torch.cuda.current_device()   # the device the cache is bound to
        self.misses_handled = 0
        self._rec = None                           # prepare(): the recorded entry call
        if code_dir is not None:
            st = _dll.tri_spec_set_code_dir(h, code_dir.encode())
            if st != OK:
                raise TriError(st, "tri_spec_set_code_dir")

    def close(self):
        if self._h:
            _dll.tri_spec_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self) -> C.c_void_p:
        return self._h

    # ---- miss path ---------------------------------------------------------
    def _call(self, what: str, fn, *args, max_misses: int = 1) -> None:
        """One entry call; on MISS install the recorded key and call again
        (a call over several layers can miss once per distinct version).
        While prepare() records, the call is noted instead of issued."""
        if self._rec is not None:
            self._rec.append((what, fn, args, max_misses))
            return
        st = fn(self._h, *args)
        for _ in range(max_misses):
            if st != MISS:
                break
            self.install_last_miss()
            self.misses_handled += 1
            st = fn(self._h, *args)
        if st != OK:
            raise TriError(st, what)

    def prepare(self, op: str, *args, **kwargs) -> Prepared:
        """Marshal one call of method `op` (e.g. "rmsnorm", "swiglu",
        "decode_chain") once and return it as a Prepared call: its `result`
        is what the method returns (output tensors allocated now when not
        given), and calling it issues the entry call with those arguments.
        Nothing is launched by prepare() itself."""
        if op in ("prepare", "close") or op.startswith("_") or not callable(getattr(self, op, None)):
            raise ValueError(f"prepare: {op!r} is not an op of the cache")
        if not self._h:
            raise TriError(E_INVALID, "prepare: the cache is closed")
        rec = []
        self._rec = rec
        try:
            result = getattr(self, op)(*args, **kwargs)
        finally:
            self._rec = None
        if len(rec) != 1:
            raise ValueError(f"prepare: {op!r} does not make exactly one entry call")
        what, fn, cargs, max_misses = rec[0]
        return Prepared(self, what, fn, cargs[:-1], max_misses, result)

    def install_last_miss(self) -> Selection:
        sel = Selection()
        st = _dll.tri_spec_install_last_miss(self._h, C.byref(sel))
        if st != OK:
            raise TriError(st, "tri_spec_install_last_miss")
        return sel

    # ---- ops ---------------------------------------------------------------
    def rmsnorm(self, x: torch.Tensor, w: torch.Tensor, eps: float = 1e-6,
                out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        T, H = _dims(x, "x", 2, self._dev)
        y = torch.empty_like(x) if out is None else out
        _like(y, "out", x.shape, x.dtype, self._dev)
        _vector(w, "w", H, x.dtype, self._dev)
        self._call("tri_rmsnorm", _dll.tri_rmsnorm, dtype_code(x.dtype), x.data_ptr(),
                   _rows(x, "x", H), w.data_ptr(), y.data_ptr(), _rows(y, "out", H), T, H, eps,
                   _stream_ptr(stream, self._dev))
        return y

    def residual_rmsnorm(self, x, residual, w, eps: float = 1e-6, out=None, residual_out=None,
                         stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
        T, H = _dims(x, "x", 2, self._dev)
        _like(residual, "residual", x.shape, x.dtype, self._dev)
        y = torch.empty_like(x) if out is None else out
        ro = torch.empty_like(residual) if residual_out is None else residual_out
        _like(y, "out", x.shape, x.dtype, self._dev)
        _like(ro, "residual_out", x.shape, x.dtype, self._dev)
        _vector(w, "w", H, x.dtype, self._dev)
        self._call("tri_residual_rmsnorm", _dll.tri_residual_rmsnorm, dtype_code(x.dtype),
                   x.data_ptr(), _rows(x, "x", H), residual.data_ptr(),
                   _rows(residual, "residual", H), w.data_ptr(), y.data_ptr(),
                   _rows(y, "out", H), ro.data_ptr(), _rows(ro, "residual_out", H), T, H, eps,
                   _stream_ptr(stream, self._dev))
        return y, ro

    def residual_rmsnorm_noalloc(self, x, residual, w, eps: float = 1e-6, out=None,
                                 residual_out=None, stream=None):
        """residual_rmsnorm through the allocation-free entry point
        (tri_residual_rmsnorm_noalloc): the outputs must be given, nothing is
        installed (a miss raises TriError with status MISS: install the
        version first, e.g. with an ordinary call), and a split version uses
        the GPU's fixed scratch."""
        if out is None or residual_out is None:
            raise ValueError("out and residual_out are required (nothing is allocated)")
        T, H = _dims(x, "x", 2, self._dev)
        _like(residual, "residual", x.shape, x.dtype, self._dev)
        _like(out, "out", x.shape, x.dtype, self._dev)
        _like(residual_out, "residual_out", x.shape, x.dtype, self._dev)
        _vector(w, "w", H, x.dtype, self._dev)
        st = _dll.tri_residual_rmsnorm_noalloc(
            self._h, dtype_code(x.dtype), x.data_ptr(), _rows(x, "x", H), residual.data_ptr(),
            _rows(residual, "residual", H), w.data_ptr(), out.data_ptr(), _rows(out, "out", H),
            residual_out.data_ptr(), _rows(residual_out, "residual_out", H), T, H, eps,
            _stream_ptr(stream, self._dev))
        if st != OK:
            raise TriError(st, "tri_residual_rmsnorm_noalloc")
        return out, residual_out

    def _qk(self, q, k, pos, pos_dtype):
        """Shapes of q [T, nq, hd], k [T, nk, hd] (or None) and pos [T]: returns
        (T, nq, nk, hd, k pointer, k token stride)."""
        T, nq, hd = _dims(q, "q", 3, self._dev)
        nk, kp, kts = 0, 0, 0
        if k is not None:
            _, nk, khd = _dims(k, "k", 3, self._dev)
            if k.shape[0] != T or khd != hd or k.dtype != q.dtype:
                raise ValueError(f"k: expected ({T}, nk, {hd}) {q.dtype}, "
                                 f"got {tuple(k.shape)} {k.dtype}")
            if nk:
                kp, kts = k.data_ptr(), _tokens(k, "k", nk, hd)
        if pos.shape != (T,) or pos.dtype != pos_dtype or (T > 1 and pos.stride(0) != 1):
            raise TypeError(f"pos must be a contiguous ({T},) {pos_dtype} tensor")
        _on(pos, "pos", self._dev)
        return T, nq, nk, hd, kp, kts

    def rope_qk(self, q, k, pos, base: float = 10000.0, stream=None):
        """In-place RoPE of q [T, nq, hd] and k [T, nk, hd] (k may be None)."""
        T, nq, nk, hd, kp, kts = self._qk(q, k, pos, torch.int32)
        self._call("tri_rope_qk", _dll.tri_rope_qk, dtype_code(q.dtype), q.data_ptr(),
                   _tokens(q, "q", nq, hd), kp, kts, pos.data_ptr(), T, nq, nk, hd, base,
                   _stream_ptr(stream, self._dev))
        return q, k

    def qk_norm_rope(self, q, k, pos, q_w, k_w=None, base: float = 10000.0, eps: float = 1e-6,
                     stream=None):
        """In-place per-head RMSNorm (weights q_w / k_w [hd]) then RoPE of
        q [T, nq, hd] and k [T, nk, hd] (k may be None)."""
        T, nq, nk, hd, kp, kts = self._qk(q, k, pos, torch.int32)
        _vector(q_w, "q_w", hd, q.dtype, self._dev)
        if k_w is not None:
            _vector(k_w, "k_w", hd, q.dtype, self._dev)
        kw = 0 if k_w is None else k_w.data_ptr()
        self._call("tri_qk_norm_rope", _dll.tri_qk_norm_rope, dtype_code(q.dtype), q.data_ptr(),
                   _tokens(q, "q", nq, hd), kp, kts, pos.data_ptr(), T, nq, nk, hd, base,
                   q_w.data_ptr(), kw, eps, _stream_ptr(stream, self._dev))
        return q, k

    def rope(self, q, k, pos, base: float = 10000.0, ext: Optional[RopeExt] = None, q_w=None,
             k_w=None, eps: float = 1e-6, stream=None):
        """In-place RoPE of q [T, nq, hd] and k [T, nk, hd] (k may be None)
        with an optional variant (`rope_ext(...)`) and, with q_w, the per-head
        QK RMSNorm first (tri_rope_qk_ext)."""
        pos_dt = torch.int64 if ext is not None and ext.pos_int64 else torch.int32
        T, nq, nk, hd, kp, kts = self._qk(q, k, pos, pos_dt)
        _check_cos_sin(ext, hd, self._dev)
        if q_w is not None:
            _vector(q_w, "q_w", hd, q.dtype, self._dev)
        if k_w is not None:
            _vector(k_w, "k_w", hd, q.dtype, self._dev)
        self._call("tri_rope_qk_ext", _dll.tri_rope_qk_ext, dtype_code(q.dtype), q.data_ptr(),
                   _tokens(q, "q", nq, hd), kp, kts, pos.data_ptr(), T, nq, nk, hd, base,
                   C.byref(ext) if ext is not None else None,
                   0 if q_w is None else q_w.data_ptr(), 0 if k_w is None else k_w.data_ptr(),
                   eps, _stream_ptr(stream, self._dev))
        return q, k

    def swiglu(self, gate, up, out=None, stream=None) -> torch.Tensor:
        T, I = _dims(gate, "gate", 2, self._dev)
        _like(up, "up", gate.shape, gate.dtype, self._dev)
        o = torch.empty_like(gate) if out is None else out
        _like(o, "out", gate.shape, gate.dtype, self._dev)
        self._call("tri_swiglu", _dll.tri_swiglu, dtype_code(gate.dtype), gate.data_ptr(),
                   _rows(gate, "gate", I), up.data_ptr(), _rows(up, "up", I), o.data_ptr(),
                   _rows(o, "out", I), T, I, _stream_ptr(stream, self._dev))
        return o

    # ---- short ops ---------------------------------------------------------------
    def silu(self, x, out=None, stream=None) -> torch.Tensor:
        """out = x / (1 + exp(-x)) over [T, W]."""
        T, W = _dims(x, "x", 2, self._dev)
        o = torch.empty_like(x) if out is None else out
        _like(o, "out", x.shape, x.dtype, self._dev)
        self._call("tri_silu", _dll.tri_silu, dtype_code(x.dtype), x.data_ptr(),
                   _rows(x, "x", W), o.data_ptr(), _rows(o, "out", W), T, W,
                   _stream_ptr(stream, self._dev))
        return o

    def add(self, a, b, out=None, stream=None) -> torch.Tensor:
        """out = a + b over [T, W] (one rounding)."""
        T, W = _dims(a, "a", 2, self._dev)
        _like(b, "b", a.shape, a.dtype, self._dev)
        o = torch.empty_like(a) if out is None else out
        _like(o, "out", a.shape, a.dtype, self._dev)
        self._call("tri_add", _dll.tri_add, dtype_code(a.dtype), a.data_ptr(),
                   _rows(a, "a", W), b.data_ptr(), _rows(b, "b", W), o.data_ptr(),
                   _rows(o, "out", W), T, W, _stream_ptr(stream, self._dev))
        return o

    def masked_fill(self, x, mask, value: float, out=None, stream=None) -> torch.Tensor:
        """out = where(mask, value, x); mask is uint8 (or bool) [T, W]."""
        if mask.dtype not in (torch.uint8, torch.bool):
            raise TypeError("mask must be uint8 or bool")
        T, W = _dims(x, "x", 2, self._dev)
        if mask.shape != x.shape:
            raise ValueError(f"mask: expected {tuple(x.shape)}, got {tuple(mask.shape)}")
        _on(mask, "mask", self._dev)
        o = torch.empty_like(x) if out is None else out
        _like(o, "out", x.shape, x.dtype, self._dev)
        self._call("tri_masked_fill", _dll.tri_masked_fill, dtype_code(x.dtype), x.data_ptr(),
                   _rows(x, "x", W), mask.data_ptr(), _rows(mask, "mask", W), value,
                   o.data_ptr(), _rows(o, "out", W), T, W, _stream_ptr(stream, self._dev))
        return o

    def embedding(self, table, ids, out=None, stream=None) -> torch.Tensor:
        """out[t] = table[ids[t]] (zeros for ids out of range); ids int32 / int64."""
        if ids.dtype not in (torch.int32, torch.int64) or ids.dim() != 1:
            raise TypeError("ids must be a 1-D int32 or int64 tensor")
        n_rows, H = _dims(table, "table", 2, self._dev)
        T = ids.shape[0]
        if T > 1 and ids.stride(0) != 1:
            raise ValueError("ids must be contiguous")
        _on(ids, "ids", self._dev)
        o = torch.empty((T, H), dtype=table.dtype, device=table.device) if out is None else out
        _like(o, "out", (T, H), table.dtype, self._dev)
        self._call("tri_embedding", _dll.tri_embedding, dtype_code(table.dtype),
                   table.data_ptr(), _rows(table, "table", H), n_rows, ids.data_ptr(),
                   int(ids.dtype == torch.int64), o.data_ptr(), _rows(o, "out", H), T, H,
                   _stream_ptr(stream, self._dev))
        return o

    def chain_args(self, x, residual, w, q, k, pos, gate, up, eps=1e-6, base=10000.0,
                   y=None, residual_out=None, out=None, q_norm_w=None, k_norm_w=None,
                   qk_eps=None, rope: Optional[RopeExt] = None) -> Tuple[ChainArgs, tuple]:
        """Build the tri_chain_args struct once (outputs allocated if absent).
        With q_norm_w (and k_norm_w) the RoPE step is QK-RMSNorm + RoPE with
        epsilon qk_eps (default: eps); `rope` selects a RoPE variant.

        The struct holds bare device addresses. It keeps a reference to every
        tensor whose address it holds (inputs, weights, positions and the
        outputs, including ones allocated here) and to the variant, so reusing
        it (decode_chain_args, decode_chain_layers, build_graph) never reaches
        freed memory; the tensors live at least as long as the struct."""
        T, H = _dims(x, "x", 2, self._dev)
        dt = x.dtype
        _like(residual, "residual", x.shape, dt, self._dev)
        _vector(w, "w", H, dt, self._dev)
        y = torch.empty_like(x) if y is None else y
        ro = torch.empty_like(residual) if residual_out is None else residual_out
        _like(y, "y", x.shape, dt, self._dev)
        _like(ro, "residual_out", x.shape, dt, self._dev)
        pos_dt = torch.int64 if rope is not None and rope.pos_int64 else torch.int32
        Tq, nq, nk, hd, kp, kts = self._qk(q, k, pos, pos_dt)
        if Tq != T or q.dtype != dt:
            raise ValueError(f"q: expected ({T}, nq, hd) {dt}, got {tuple(q.shape)} {q.dtype}")
        _check_cos_sin(rope, hd, self._dev)
        _, I = _dims(gate, "gate", 2, self._dev)
        _like(gate, "gate", (T, I), dt, self._dev)
        _like(up, "up", (T, I), dt, self._dev)
        o = torch.empty_like(gate) if out is None else out
        _like(o, "out", (T, I), dt, self._dev)
        a = ChainArgs()
        a.dtype = dtype_code(dt)
        a.T, a.H, a.I, a.nq, a.nk, a.hd = T, H, I, nq, nk, hd
        a.eps, a.base = eps, base
        a.x, a.x_rs = x.data_ptr(), _rows(x, "x", H)
        a.res, a.res_rs = residual.data_ptr(), _rows(residual, "residual", H)
        a.w = w.data_ptr()
        a.y, a.y_rs = y.data_ptr(), _rows(y, "y", H)
        a.res_out, a.ro_rs = ro.data_ptr(), _rows(ro, "residual_out", H)
        a.q, a.q_ts = q.data_ptr(), _tokens(q, "q", nq, hd)
        a.k, a.k_ts = kp, kts
        a.pos = pos.data_ptr()
        a.gate, a.g_rs = gate.data_ptr(), _rows(gate, "gate", I)
        a.up, a.u_rs = up.data_ptr(), _rows(up, "up", I)
        a.out, a.o_rs = o.data_ptr(), _rows(o, "out", I)
        if q_norm_w is not None:
            _vector(q_norm_w, "q_norm_w", hd, dt, self._dev)
            if k_norm_w is not None:
                _vector(k_norm_w, "k_norm_w", hd, dt, self._dev)
            a.q_norm_w = q_norm_w.data_ptr()
            a.k_norm_w = 0 if k_norm_w is None else k_norm_w.data_ptr()
            a.qk_eps = eps if qk_eps is None else qk_eps
        if rope is not None:
            a.rope_ext = C.pointer(rope)
        a._keep = (x, residual, w, y, ro, q, k, pos, gate, up, o, q_norm_w, k_norm_w, rope)
        return a, (y, ro, o)

    def decode_chain_args(self, args: ChainArgs, stream=None) -> None:
        self._call("tri_decode_chain", _dll.tri_decode_chain, C.byref(args),
                   _stream_ptr(stream, self._dev))

    def decode_chain_layers(self, layers, stream=None) -> None:
        """Several chains (a list of ChainArgs from chain_args) in one entry
        call, launched in list order (tri_decode_chain_layers)."""
        arr = (ChainArgs * max(1, len(layers)))(*layers)
        self._call("tri_decode_chain_layers", _dll.tri_decode_chain_layers, arr, len(layers),
                   _stream_ptr(stream, self._dev), max_misses=len(layers))

    def build_graph(self, layers) -> "Graph":
        """Capture the launches of decode_chain_layers(layers) into a HIP
        graph (guards evaluated once, now). Replays fix every pointer and size."""
        arr = (ChainArgs * max(1, len(layers)))(*layers)
        g = C.c_void_p()
        st = _dll.tri_graph_build_layers(self._h, arr, len(layers), C.byref(g))
        for _ in range(len(layers)):
            if st != MISS:
                break
            self.install_last_miss()
            self.misses_handled += 1
            st = _dll.tri_graph_build_layers(self._h, arr, len(layers), C.byref(g))
        if st != OK:
            raise TriError(st, "tri_graph_build_layers")
        return Graph(g, self)

    def decode_chain(self, x, residual, w, q, k, pos, gate, up, eps=1e-6, base=10000.0,
                     y=None, residual_out=None, out=None, stream=None, q_norm_w=None,
                     k_norm_w=None, qk_eps=None, rope: Optional[RopeExt] = None):
        """Residual+RMSNorm, in-place (QK-RMSNorm +) RoPE of q/k and SwiGLU in
        one entry call. Returns (y, residual_out, out)."""
        a, outs = self.chain_args(x, residual, w, q, k, pos, gate, up, eps, base, y,
                                  residual_out, out, q_norm_w, k_norm_w, qk_eps, rope)
        self.decode_chain_args(a, stream)
        return outs

    def export_keys(self):
        """Keys of the installed versions, creation order (tuples of 6 ints)."""
        n = C.c_uint32()
        _dll.tri_spec_export_keys(self._h, None, 0, C.byref(n))
        buf = (C.c_uint64 * (L.KEY_WORDS * max(1, n.value)))()
        st = _dll.tri_spec_export_keys(self._h, buf, n.value, C.byref(n))
        if st != OK:
            raise TriError(st, "tri_spec_export_keys")
        w = list(buf)
        return [tuple(w[i * L.KEY_WORDS:(i + 1) * L.KEY_WORDS]) for i in range(n.value)]

    def import_keys(self, keys) -> int:
        """Install versions for exported keys (pre-warm); returns the count."""
        flat = [int(x) for k in keys for x in k]
        buf = (C.c_uint64 * max(1, len(flat)))(*flat)
        done = C.c_uint32()
        st = _dll.tri_spec_import_keys(self._h, buf, len(keys), C.byref(done))
        if st != OK:
            raise TriError(st, f"tri_spec_import_keys (after {done.value} keys)")
        return done.value

    def export_plans(self):
        """(key, candidate index) of every installed version, creation order:
        a tuned set of versions that import_plans reinstalls without timing."""
        return [(k, self.version_info(i).candidate) for i, k in enumerate(self.export_keys())]

    def import_plans(self, plans) -> None:
        """Install (key, candidate) pairs as exported by export_plans."""
        for key, cand in plans:
            self.install_key(key, cand)

    def install_key(self, key, candidate: int = -1) -> None:
        """Install one key (6 words) with candidate plan `candidate` (-1: the
        cache's own rule: tuned under autotune, else the policy's plan)."""
        buf = (C.c_uint64 * L.KEY_WORDS)(*[int(x) for x in key])
        st = _dll.tri_spec_install_key(self._h, buf, candidate)
        if st != OK:
            raise TriError(st, "tri_spec_install_key")

    def launch_empty(self, stream=None) -> None:
        st = _dll.tri_launch_empty(self._h, _stream_ptr(stream, self._dev))
        if st != OK:
            raise TriError(st, "tri_launch_empty")

    # ---- introspection -------------------------------------------------------
    def last_selection(self) -> Selection:
        s = Selection()
        _dll.tri_spec_last_selection(self._h, C.byref(s))
        return s

    def stats(self) -> dict:
        s = Stats()
        _dll.tri_spec_stats(self._h, C.byref(s))
        return s.as_dict()

    def resident_info(self) -> dict:
        r = L.ResidentInfo()
        st = _dll.tri_spec_resident_info(self._h, C.byref(r))
        if st != OK:
            raise TriError(st, "tri_spec_resident_info")
        return {"enabled": r.enabled, "held": r.held, "launches": r.launches}

    def version_info(self, i: int) -> VersionInfo:
        v = VersionInfo()
        st = _dll.tri_spec_version_info(self._h, i, C.byref(v))
        if st != OK:
            raise TriError(st, "tri_spec_version_info")
        return v

    def version_constants(self, i: int):
        n = C.c_uint32()
        buf = (C.c_float * 256)()
        st = _dll.tri_spec_version_constants(self._h, i, buf, 256, C.byref(n))
        if st != OK:
            raise TriError(st, "tri_spec_version_constants")
        return list(buf[: n.value])
