"""Build libquake.so for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2412_00408_amd.build

Every source is compiled for gfx950 only, with fp contraction off (every
fused multiply-add of the method is an explicit fma), packed-fp32 VALU ops
disabled, denormals kept, then linked into one shared library.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libquake.so")
C_CLIENT_SRC = os.path.join(ROOT, "tests", "c", "abi_smoke.c")
C_CLIENT = os.path.join(ROOT, "tests", "c", "abi_smoke")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

SOURCES = ["elementwise.hip", "softmax.hip", "native16.hip", "gemm.hip", "attention.hip",
           "ceiling.hip", "abi.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument", "-I", INCLUDE, "-I", CSRC,
]


# Matrix-core accumulators in ordinary VGPRs: the attention kernel feeds them
# straight to VALU work, which cannot read the accumulation registers.
EXTRA_FLAGS = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd = [HIPCC, "-x", "hip", *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


def build_c_client(verbose: bool = False) -> str:
    """Compile the plain-C client of the ABI (gcc, include/quake.h and the HIP
    runtime only) that checks the library from C, without Python or torch."""
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE,
           "-I", os.path.join(ROCM, "include"), C_CLIENT_SRC, "-o", C_CLIENT + ".tmp",
           "-L", HERE, "-lquake", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2412_00408_amd",
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("gcc failed for the C client:\n%s\n%s" % (r.stdout, r.stderr))
    os.replace(C_CLIENT + ".tmp", C_CLIENT)
    if verbose:
        print("built", C_CLIENT)
    return C_CLIENT


if __name__ == "__main__":
    build(verbose=True)
    build_c_client(verbose=True)
    sys.exit(0)
