"""ctypes declarations of the libtri C ABI (include/tri.h).

Loading order matters: torch is imported first so that libtri binds to the
HIP runtime torch already loaded (both carry the same SONAME), giving one
runtime, one set of streams and one device context per process.
"""
from __future__ import annotations

import ctypes as C
import os

import torch  # noqa: F401  -- must precede loading libtri (shared HIP runtime)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtri.so")

OK, MISS = 0, 1
E_INVALID, E_UNSUPPORTED, E_FULL, E_NOMEM, E_LAUNCH, E_RUNTIME = -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1
OP_RMSNORM, OP_RES_RMSNORM, OP_ROPE_QK, OP_SWIGLU, OP_CHAIN, OP_QK_NORM_ROPE = 1, 2, 3, 4, 5, 6
OP_CHAIN_LAYERS = 7
OP_SILU, OP_ADD, OP_MASKED_FILL, OP_EMBEDDING = 8, 9, 10, 11
MAX_LAYERS = 1024
AUTO_INSTALL = 1
JIT = 2
AUTOTUNE = 4
GENERIC = 8
RESIDENT_ARGS = 16
RESIDENT_SLOTS, RESIDENT_MAX_GRID, RESIDENT_ANY_GRID_SLOTS = 40, 512, 10
TUNE_NONE, TUNE_MEASURED, TUNE_STORED, TUNE_SKIPPED = 0, 1, 2, 3
KEY_WORDS = 6
NOALLOC_SCRATCH_BYTES = 1 << 20
ROPE_SCALING_NONE, ROPE_SCALING_LLAMA3 = 0, 1


class LaunchRec(C.Structure):
    _fields_ = [("variant", C.c_int32), ("grid_x", C.c_uint32), ("block_x", C.c_uint32)]


class Selection(C.Structure):
    _fields_ = [("op", C.c_int32), ("status", C.c_int32), ("version", C.c_int32),
                ("variant", C.c_int32), ("n_launches", C.c_int32),
                ("roles", C.c_int32 * 3), ("launch", LaunchRec * 3),
                ("key", C.c_uint64 * KEY_WORDS)]

    def as_tuple(self):
        return (self.op, self.status, self.version, self.variant, self.n_launches,
                tuple(self.roles),
                tuple((l.variant, l.grid_x, l.block_x) for l in self.launch),
                tuple(self.key))


class Stats(C.Structure):
    _fields_ = [("calls", C.c_uint64), ("hits", C.c_uint64), ("misses", C.c_uint64),
                ("errors", C.c_uint64), ("empty", C.c_uint64), ("installs", C.c_uint64),
                ("n_versions", C.c_uint32), ("capacity", C.c_uint32)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class ResidentInfo(C.Structure):
    _fields_ = [("enabled", C.c_int32), ("held", C.c_uint32), ("launches", C.c_uint64)]


class VersionInfo(C.Structure):
    _fields_ = [("key", C.c_uint64 * KEY_WORDS), ("variant", C.c_int32), ("roles", C.c_int32 * 3),
                ("hits", C.c_uint64), ("jit", C.c_int32), ("build_ms", C.c_float),
                ("n_launches", C.c_int32), ("kernels", C.c_int32 * 3),
                ("rope_slices", C.c_int32), ("candidate", C.c_int32),
                ("n_candidates", C.c_int32), ("tuned", C.c_int32), ("tune_ms", C.c_float),
                ("rope_tokens", C.c_int32), ("b_lo", C.c_int32), ("b_hi", C.c_int32),
                ("h_lo", C.c_uint32), ("h_hi", C.c_uint32), ("h_mod", C.c_int32)]


class RopeExt(C.Structure):
    _fields_ = [("rotary_dim", C.c_int32), ("interleaved", C.c_int32),
                ("pos_int64", C.c_int32), ("scaling", C.c_int32),
                ("factor", C.c_float), ("low_freq_factor", C.c_float),
                ("high_freq_factor", C.c_float), ("original_max_pos", C.c_int32),
                ("cos_sin", C.c_void_p), ("cos_sin_len", C.c_int64)]


class ChainArgs(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("nq", C.c_int32), ("nk", C.c_int32), ("hd", C.c_int32),
                ("T", C.c_int64), ("H", C.c_int64), ("I", C.c_int64),
                ("eps", C.c_float), ("base", C.c_float),
                ("x", C.c_void_p), ("x_rs", C.c_int64),
                ("res", C.c_void_p), ("res_rs", C.c_int64),
                ("w", C.c_void_p),
                ("y", C.c_void_p), ("y_rs", C.c_int64),
                ("res_out", C.c_void_p), ("ro_rs", C.c_int64),
                ("q", C.c_void_p), ("q_ts", C.c_int64),
                ("k", C.c_void_p), ("k_ts", C.c_int64),
                ("pos", C.c_void_p),
                ("gate", C.c_void_p), ("g_rs", C.c_int64),
                ("up", C.c_void_p), ("u_rs", C.c_int64),
                ("out", C.c_void_p), ("o_rs", C.c_int64),
                ("q_norm_w", C.c_void_p), ("k_norm_w", C.c_void_p),
                ("qk_eps", C.c_float), ("reserved", C.c_int32),
                ("rope_ext", C.POINTER(RopeExt))]


assert C.sizeof(Selection) == 120 and C.sizeof(ChainArgs) == 240 and C.sizeof(RopeExt) == 48
assert C.sizeof(VersionInfo) == 144 and C.sizeof(ResidentInfo) == 16

_P, _I64, _I32, _F, _U32 = C.c_void_p, C.c_int64, C.c_int32, C.c_float, C.c_uint32

SIGNATURES = {
    "tri_spec_cache_create": (C.c_int, [C.POINTER(C.c_void_p), _U32, _U32]),
    "tri_spec_cache_destroy": (None, [_P]),
    "tri_rmsnorm": (C.c_int, [_P, C.c_int, _P, _I64, _P, _P, _I64, _I64, _I64, _F, _P]),
    "tri_residual_rmsnorm": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _P, _I64, _P, _I64,
                                       _I64, _I64, _F, _P]),
    "tri_residual_rmsnorm_noalloc": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _P, _I64,
                                               _P, _I64, _I64, _I64, _F, _P]),
    "tri_rope_qk": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _I64, _I32, _I32, _I32, _F,
                              _P]),
    "tri_rope_qk_ext": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _I64, _I32, _I32, _I32,
                                  _F, C.POINTER(RopeExt), _P, _P, _F, _P]),
    "tri_qk_norm_rope": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _I64, _I32, _I32, _I32,
                                   _F, _P, _P, _F, _P]),
    "tri_swiglu": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _I64, _I64, _I64, _P]),
    "tri_silu": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _I64, _I64, _P]),
    "tri_add": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _P, _I64, _I64, _I64, _P]),
    "tri_masked_fill": (C.c_int, [_P, C.c_int, _P, _I64, _P, _I64, _F, _P, _I64, _I64, _I64,
                                  _P]),
    "tri_embedding": (C.c_int, [_P, C.c_int, _P, _I64, _I64, _P, _I32, _P, _I64, _I64, _I64,
                                _P]),
    "tri_decode_chain": (C.c_int, [_P, C.POINTER(ChainArgs), _P]),
    "tri_decode_chain_layers": (C.c_int, [_P, C.POINTER(ChainArgs), _U32, _P]),
    "tri_graph_build_layers": (C.c_int, [_P, C.POINTER(ChainArgs), _U32, C.POINTER(C.c_void_p)]),
    "tri_graph_launch": (C.c_int, [_P, _P]),
    "tri_graph_launch_count": (_U32, [_P]),
    "tri_graph_destroy": (None, [_P]),
    "tri_spec_install_last_miss": (C.c_int, [_P, C.POINTER(Selection)]),
    "tri_spec_last_selection": (C.c_int, [_P, C.POINTER(Selection)]),
    "tri_spec_stats": (C.c_int, [_P, C.POINTER(Stats)]),
    "tri_spec_resident_info": (C.c_int, [_P, C.POINTER(ResidentInfo)]),
    "tri_spec_version_info": (C.c_int, [_P, _U32, C.POINTER(VersionInfo)]),
    "tri_spec_version_constants": (C.c_int, [_P, _U32, C.POINTER(C.c_float), _U32,
                                             C.POINTER(C.c_uint32)]),
    "tri_launch_empty": (C.c_int, [_P, _P]),
    "tri_spec_set_code_dir": (C.c_int, [_P, C.c_char_p]),
    "tri_spec_export_keys": (C.c_int, [_P, C.POINTER(C.c_uint64), _U32, C.POINTER(C.c_uint32)]),
    "tri_spec_import_keys": (C.c_int, [_P, C.POINTER(C.c_uint64), _U32, C.POINTER(C.c_uint32)]),
    "tri_spec_install_key": (C.c_int, [_P, C.POINTER(C.c_uint64), _I32]),
    "tri_status_str": (C.c_char_p, [C.c_int]),
}


def declare(lib: C.CDLL) -> C.CDLL:
    """Attach argtypes / restype to every exported entry point."""
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load libtri.so (built in-tree). Raises if it has not been built."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise ImportError(
            f"libtri.so not found at {path}: build it first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = declare(C.CDLL(path))
    if path == LIB_PATH:
        _lib = lib
    return lib
