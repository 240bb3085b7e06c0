"""Locate / build the native libraries the tests load.

libtri.so (the product) is built by __graft_entry__.build(); the tests only
build it here when it is missing. libtri_fake.so is the cache core linked
with the recording backend in tests/native (CPU tests only).
"""
import ctypes as C
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_37241_amd")
LIBTRI = os.path.join(PKG, "libtri.so")
FAKE_SRC = os.path.join(ROOT, "tests", "native", "fake_backend.cpp")
FAKE_LIB = os.path.join(ROOT, "tests", "native", "libtri_fake.so")
# With TRI_FAKE_SANITIZE=1 the tests load a build of the same sources with
# AddressSanitizer and UndefinedBehaviorSanitizer (host code only; the
# process must preload the sanitizer runtimes, see test_host_sanitized.py).
SANITIZE = os.environ.get("TRI_FAKE_SANITIZE") == "1"
FAKE_ASAN_LIB = os.path.join(ROOT, "tests", "native", "libtri_fake_asan.so")
SANITIZE_FLAGS = ["-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=undefined"]


def _build_module():
    spec = importlib.util.spec_from_file_location("_tri_build", os.path.join(PKG, "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def ensure_libtri() -> str:
    if not os.path.exists(LIBTRI):
        _build_module().build()
    return LIBTRI


def ensure_fake() -> str:
    srcs = [FAKE_SRC] + [os.path.join(PKG, "csrc", n)
                         for n in ("api.cpp", "cache.cpp", "policy.cpp", "jit.cpp", "tune.cpp",
                                   "resident.cpp", "internal.h", "kernargs.h",
                                   "kernels/device.h")]
    out = FAKE_ASAN_LIB if SANITIZE else FAKE_LIB
    stale = (not os.path.exists(out)
             or any(os.path.getmtime(s) > os.path.getmtime(out) for s in srcs))
    if stale:
        _build_module().build_host_core(FAKE_SRC, out, SANITIZE_FLAGS if SANITIZE else None)
    return out


def load_fake():
    """The cache core + recording backend, with the ABI's signatures."""
    ensure_libtri()
    from paper_2609_37241_amd import _lib as L
    lib = L.declare(C.CDLL(ensure_fake()))
    lib.trifake_launch_count.restype = C.c_int64
    lib.trifake_upload_count.restype = C.c_int64
    lib.trifake_fail_at.argtypes = [C.c_int64]
    lib.trifake_init_status.argtypes = [C.c_int]
    lib.trifake_graph_launches.restype = C.c_int64
    lib.trifake_graph_destroys.restype = C.c_int64
    lib.trifake_capture_fail.argtypes = [C.c_int]
    lib.tri_graph_build_layers.argtypes = [C.c_void_p, C.c_void_p, C.c_uint32,
                                           C.POINTER(C.c_void_p)]
    lib.tri_graph_launch.argtypes = [C.c_void_p, C.c_void_p]
    lib.tri_graph_launch_count.argtypes = [C.c_void_p]
    lib.tri_graph_launch_count.restype = C.c_uint32
    lib.tri_graph_destroy.argtypes = [C.c_void_p]
    lib.tri_graph_destroy.restype = None
    lib.trifake_jit_count.restype = C.c_int64
    lib.trifake_compile_count.restype = C.c_int64
    lib.tri_spec_set_code_dir.argtypes = [C.c_void_p, C.c_char_p]
    lib.trifake_unload_count.restype = C.c_int64
    lib.trifake_jit_fail.argtypes = [C.c_int]
    lib.trifake_jit_source.restype = C.c_int64
    lib.trifake_jit_source.argtypes = [C.c_int64, C.c_char_p, C.c_int64]
    lib.trifake_set_cost.argtypes = [C.c_int32, C.c_int32, C.c_uint32, C.c_float]
    lib.trifake_scratch_fail.argtypes = [C.c_int]
    lib.trifake_set_arch.argtypes = [C.c_char_p]
    lib.trifake_tune_counts.argtypes = [C.POINTER(C.c_int64)]
    lib.trifake_get.argtypes = [C.c_int64, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                C.POINTER(C.c_int32), C.POINTER(C.c_uint32),
                                C.POINTER(C.c_uint32), C.POINTER(C.c_void_p),
                                C.c_char_p, C.c_int]
    lib.trifake_resident_check_fail.argtypes = [C.c_int]
    lib.trifake_resident_write_fail.argtypes = [C.c_int]
    lib.trifake_force_capturing.argtypes = [C.c_int]
    lib.trifake_resident_counts.argtypes = [C.POINTER(C.c_int64)]
    lib.trifake_resident_tag.argtypes = [C.c_int32, C.c_int32, C.c_int32,
                                         C.POINTER(C.c_uint32), C.POINTER(C.c_uint32)]
    lib.trifake_resident_tag.restype = C.c_int64
    lib.trifake_slot.argtypes = [C.c_int64]
    lib.trifake_slot.restype = C.c_int32
    return lib
