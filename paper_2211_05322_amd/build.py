"""Build libreshard.so (host planner + gfx950 kernel) in-tree with hipcc.

    python -m paper_2211_05322_amd.build

Compiles every source each time it is called; the result replaces the
library atomically so a process that already mapped the old file keeps it.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libreshard.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

ARCH = "gfx950"
COMMON = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-Wextra", "-Wno-unused-parameter"]
# packed-fp32 instructions are disabled for all device code
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_SOURCES = ["planner.cpp", "capi.cpp", "schedule.cpp", "pipeline.cpp"]
HIP_SOURCES = ["execute.hip"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose=False, extra_hip_flags=(), out=LIB):
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    tmp = tempfile.mkdtemp(prefix="reshard_build_")
    try:
        objs = []
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            _run(["g++", *COMMON, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
            objs.append(obj)
        for src in HIP_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *COMMON, *HIP_FLAGS, *extra_hip_flags, "-c", os.path.join(CSRC, src), "-o", obj],
                 verbose)
            objs.append(obj)
        tmp_lib = os.path.join(tmp, "libreshard.so")
        _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp_lib,
              f"-Wl,-rpath,{ROCM}/lib"], verbose)
        staged = out + ".tmp"
        shutil.copyfile(tmp_lib, staged)
        os.replace(staged, out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


ROOT = os.path.dirname(PKG)
C_CLIENT_SRC = os.path.join(ROOT, "tests", "c", "abi_gpu.c")
C_CLIENT = os.path.join(ROOT, "tests", "c", "abi_gpu")
ROOT_INCLUDE_HIP = os.path.join(ROCM, "include")


def build_c_client(verbose=False):
    """The C99 client of the C ABI that the GPU tests run (tests/c/abi_gpu.c):
    gcc against include/reshard.h, the in-tree library and the HIP runtime,
    no Python or torch in its process."""
    if not os.path.exists(C_CLIENT_SRC):  # a tree without tests
        return None
    staged = C_CLIENT + ".tmp"
    _run(["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic", "-D__HIP_PLATFORM_AMD__",
          "-I", os.path.join(ROOT, "include"), "-isystem", ROOT_INCLUDE_HIP, C_CLIENT_SRC,
          "-L", PKG, "-lreshard", "-L", f"{ROCM}/lib", "-lamdhip64",
          "-Wl,-rpath,$ORIGIN/../../paper_2211_05322_amd", f"-Wl,-rpath,{ROCM}/lib", "-o", staged], verbose)
    os.replace(staged, C_CLIENT)
    return C_CLIENT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_c_client(verbose="-v" in sys.argv))
