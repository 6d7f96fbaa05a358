"""Build libcurvadion.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

Usage: python -m paper_2512_13728_amd.build   (or build() from Python)
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libcurvadion.so")
OBJDIR = os.path.join(ROOT, "_build")

SOURCES = ["k_stream.hip", "k_gemm.hip", "k_gemm_bf.hip", "k_chol.hip", "k_colnorm.hip", "k_update_vec.hip", "k_small.hip", "k_gram.hip", "k_form_bq.hip", "k_nearid.hip", "api.cpp"]

# -packed-fp32-ops: keep the compiler from emitting packed fp32 arithmetic
# (v_pk_*_f32); scalar and vector fp32 code is compiled as plain VALU ops.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall",
             "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-munsafe-fp-atomics"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libcurvadion.so)")


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [hipcc(), *HIP_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
           os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


C_CLIENT_SRC = os.path.join(ROOT, "tests", "c", "cd_c_step.c")
C_CLIENT = os.path.join(ROOT, "tests", "c", "cd_c_step")


def build_c_client() -> str:
    """The plain-C99 client of the ABI that the tests run (gcc, no HIP
    compiler: the header and the HIP runtime's C API only)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(rocm, "include"), C_CLIENT_SRC,
           "-L", HERE, "-lcurvadion", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2512_13728_amd", "-Wl,-rpath," + os.path.join(rocm, "lib"),
           "-o", C_CLIENT]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"C client build failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return C_CLIENT


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library (then the C client
    the tests use); returns the library's path."""
    os.makedirs(OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    build_c_client()
    if verbose:
        print("built", LIB, "and", C_CLIENT)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
