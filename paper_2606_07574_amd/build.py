"""Build the HIP library libbirkhoff4.so for gfx950, in-tree (no JIT cache).

Usage: python -m paper_2606_07574_amd.build   (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "birkhoff4.hip")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libbirkhoff4.so")
ARCH = "gfx950"

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # keep packed-fp32 instructions out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # fp32 denormals flush to zero (the forward kernel relies on it, see csrc)
    "-fgpu-flush-denormals-to-zero",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


def build(extra_flags: list[str] | None = None, out: str = LIB, verbose: bool = False) -> str:
    """Compile csrc/birkhoff4.hip into ``out`` (always recompiles)."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *FLAGS, *(extra_flags or []), "-I", INCLUDE, "-o", tmp, SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
