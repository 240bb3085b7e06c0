"""Build libtri.so in-tree: gfx950 kernels with hipcc, the host cache core
with the system C++ compiler, linked against the HIP runtime.

`build()` always recompiles everything (a few tens of seconds on 8 cores).
`build_host_core(backend_src, out)` links the same host sources against
another launch backend (the CPU tests use a recording one).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
from typing import List, Optional

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
KDIR = os.path.join(CSRC, "kernels")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libtri.so")
BENCH_LIB = os.path.join(PKG, "libtri_bench.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CXX = os.environ.get("CXX", "g++")

ARCH = "gfx950"
# Packed-FP32 instructions are disabled: hipcc may form v_pk_{add,mul,fma}_f32
# from ordinary float code, and we keep every float32 operation scalar.
HIP_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", INCLUDE, "-I", CSRC]
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-I", INCLUDE, "-I", CSRC]
HOST_SOURCES = ["api.cpp", "cache.cpp", "policy.cpp"]
HIP_BACKEND = "backend_hip.cpp"


def _run(cmd: List[str]) -> None:
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if out.strip():
        print(out, file=sys.stderr)


def _obj(src: str) -> str:
    return os.path.join(BUILD, os.path.basename(src) + ".o")


def hip_sources() -> List[str]:
    return sorted(os.path.join(KDIR, f) for f in os.listdir(KDIR) if f.endswith(".hip"))


def build(jobs: Optional[int] = None) -> str:
    """Compile and link libtri.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(16, os.cpu_count() or 4)
    cmds = []
    for src in hip_sources():
        cmds.append([HIPCC, *HIP_FLAGS, "-c", src, "-o", _obj(src)])
    for name in HOST_SOURCES:
        src = os.path.join(CSRC, name)
        cmds.append([CXX, *HOST_FLAGS, "-c", src, "-o", _obj(src)])
    src = os.path.join(CSRC, HIP_BACKEND)
    cmds.append([CXX, *HOST_FLAGS, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
                 "-c", src, "-o", _obj(src)])
    with cf.ThreadPoolExecutor(jobs) as ex:
        for f in [ex.submit(_run, c) for c in cmds]:
            f.result()
    objs = [c[-1] for c in cmds]
    rocm_lib = os.path.join(ROCM, "lib")
    tmp = LIB + ".tmp"
    _run([CXX, "-shared", "-o", tmp, *objs, "-L", rocm_lib, "-lamdhip64",
          "-Wl,-soname,libtri.so", f"-Wl,-rpath,{rocm_lib}", "-Wl,--no-undefined"])
    shutil.move(tmp, LIB)
    # the benchmark's native timing loops, linked against libtri.so
    harness = os.path.join(CSRC, "bench", "harness.cpp")
    tmp = BENCH_LIB + ".tmp"
    _run([CXX, *HOST_FLAGS, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
          "-shared", "-o", tmp, harness, "-L", PKG, "-ltri", "-L", rocm_lib, "-lamdhip64",
          "-Wl,-rpath,$ORIGIN", f"-Wl,-rpath,{rocm_lib}", "-Wl,--no-undefined"])
    shutil.move(tmp, BENCH_LIB)
    return LIB


def build_host_core(backend_src: str, out: str, extra_flags: Optional[List[str]] = None) -> str:
    """Link the host cache core with `backend_src` into shared library `out`."""
    srcs = [os.path.join(CSRC, n) for n in HOST_SOURCES] + [backend_src]
    tmp = out + ".tmp"
    _run([CXX, *HOST_FLAGS, *(extra_flags or []), "-shared", "-o", tmp, *srcs])
    shutil.move(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
