"""Build the native library ``libflowkv.so`` in-tree for gfx950.

``python -m paper_2504_03775_amd.build`` compiles the host C++ (allocator,
planner, scheduler, status) with g++ and the HIP translation unit (kernel + launcher)
with hipcc, then links them into ``paper_2504_03775_amd/libflowkv.so``.  In a
checkout with ``tests/native/abi_transfer.cpp`` it also builds that program,
which drives the library through the C ABI alone (no Python), next to its
source.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libflowkv.so")

HOST_SOURCES = ["flowkv_status.cpp", "flowkv_alloc.cpp", "flowkv_plan.cpp", "flowkv_sched.cpp",
                "flowkv_request.cpp"]
HIP_SOURCES = ["flowkv_transfer.hip", "flowkv_attention.hip"]

ARCH = "gfx950"
# packed-fp32 instructions are disabled for every HIP translation unit
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-command-line-argument"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True, extra_host_flags=(), lib_path: str = LIB,
          obj_tag: str = "") -> str:
    """Compile and link; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src.replace(".cpp", f"{obj_tag}.o"))
        _run(["g++", *HOST_FLAGS, *extra_host_flags, "-I", INCLUDE, "-I", CSRC,
              "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    hipcc = _hipcc()
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", f"{obj_tag}.o"))
        _run([hipcc, *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src),
              "-o", obj], verbose)
        objs.append(obj)
    tmp = lib_path + ".tmp"
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *extra_host_flags, *objs,
          "-o", tmp], verbose)
    os.replace(tmp, lib_path)
    if lib_path == LIB:
        build_abi_check(verbose)
    return lib_path


def build_abi_check(verbose: bool = True):
    """tests/native/abi_transfer: host C++ against include/flowkv.h and the
    HIP runtime API, linked to the in-tree library (found through its rpath)."""
    src = os.path.join(ROOT, "tests", "native", "abi_transfer.cpp")
    if not os.path.exists(src):
        return None
    exe = src[:-len(".cpp")]
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(_hipcc())))
    _run(["g++", "-O2", "-std=c++17", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
          "-I", INCLUDE, "-I", os.path.join(rocm, "include"), src,
          "-L", PKG, "-lflowkv", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
          "-Wl,-rpath,$ORIGIN/../../paper_2504_03775_amd",
          f"-Wl,-rpath,{os.path.join(rocm, 'lib')}", "-o", exe], verbose)
    return exe


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
