"""Build libmsao.so (the HIP kernels and the C ABI) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libmsao.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in
           ("msao_host.cpp", "msao_sched.cpp", "msao_kernels.hip", "msao_entropy.hip", "msao_simhash.hip",
            "msao_scratch.hip", "msao_calib.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep the compiler from forming packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"),
]


def build(verbose: bool = False) -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed to build libmsao.so")
    os.replace(tmp, LIB)
    return LIB


C_CLIENT_SRC = os.path.join(ROOT, "tests", "c", "abi_gpu_run.c")
C_CLIENT = os.path.join(ROOT, "tests", "c", "abi_gpu_run")


def build_c_client(verbose: bool = False) -> str:
    """The plain C client the GPU tests run (gcc, HIP C API, linked to libmsao.so)."""
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    tmp = C_CLIENT + f".tmp{os.getpid()}"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"), C_CLIENT_SRC, "-o", tmp,
           "-L", HERE, "-lmsao", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2604_02945_amd", "-Wl,-rpath," + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("gcc failed to build the C client")
    os.replace(tmp, C_CLIENT)
    return C_CLIENT


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_c_client(verbose=True))
