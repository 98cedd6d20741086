"""Builds the gfx950 HIP library in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
SOURCES = [os.path.join(PKG_DIR, "csrc", f)
           for f in ("rl_decode.hip", "rl_extend.hip", "rl_append.hip", "rl_weight_sync.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG_DIR, "librl_decode_attn.so")
# measurement-only kernels used by bench.py (stream-read ceiling, copy)
BENCH_SOURCES = [os.path.join(PKG_DIR, "csrc", "rl_bench_kernels.hip")]
BENCH_LIB_PATH = os.path.join(PKG_DIR, "librl_bench_kernels.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 VALU ops are kept out of generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _compile(sources, out, verbose):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + ["-I", INCLUDE] + sources + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_library(verbose: bool = False) -> str:
    """Compile the attention library (always), atomically replacing any
    previous build."""
    return _compile(SOURCES, LIB_PATH, verbose)


def build_bench_library(verbose: bool = False) -> str:
    return _compile(BENCH_SOURCES, BENCH_LIB_PATH, verbose)


def build_all(verbose: bool = False):
    return build_library(verbose), build_bench_library(verbose)


if __name__ == "__main__":
    print(build_all(verbose=True))
