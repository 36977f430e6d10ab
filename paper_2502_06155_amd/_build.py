"""Compile the gfx950 tile-attention library in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
REPO_DIR = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
LIB_NAME = "libtileattn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
SOURCES = [os.path.join(CSRC, f) for f in ("tile_attn_host.cpp", "tile_attn_kernels.hip", "tile_attn_bwd.hip",
                                               "tile_attn_noalloc.hip")]

HIP_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    # code object v5 loads in every ROCm 6.x/7.x runtime, including the one torch bundles
    "-mcode-object-version=5",
    # keep the compiler from emitting packed fp32 arithmetic (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(REPO_DIR, "include"),
]


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build_library(verbose: bool = True) -> str:
    """Build libtileattn.so next to this file and return its path."""
    fd, tmp = tempfile.mkstemp(prefix=".libtileattn.", suffix=".so.tmp", dir=PKG_DIR)
    os.close(fd)
    cmd = [hipcc(), *HIP_FLAGS, *SOURCES, "-o", tmp]
    if verbose:
        print("[build]", " ".join(cmd), flush=True)
    try:
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
        os.replace(tmp, LIB_PATH)
    finally:
        if os.path.exists(tmp):
            os.remove(tmp)
    return LIB_PATH


if __name__ == "__main__":
    print(build_library())
