"""Build libxgemm.so (the HIP library behind include/xgemm.h) for gfx950, in-tree."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "xgemm.hip")
DEPS = [SRC, os.path.join(PKG, "csrc", "gemm_kernel.hpp"), os.path.join(PKG, "csrc", "gemv_kernel.hpp"),
        os.path.join(PKG, "csrc", "pack_kernel.hpp"), os.path.join(PKG, "csrc", "sk_kernel.hpp"),
        os.path.join(ROOT, "include", "xgemm.h")]
LIB = os.path.join(PKG, "libxgemm.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 vector ops are disabled for all device code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++20", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    """Compile the library; always rebuilds.  Returns the path of the .so."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + [SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(d) > t for d in DEPS)


if __name__ == "__main__":
    print(build(verbose=True))
