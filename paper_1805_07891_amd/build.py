"""Builds the HIP library ``libphub.so`` in-tree for gfx950.

Every source is compiled by hipcc with contraction off, no fast-math and
subnormals kept, so that the kernel performs exactly the fp32 operations
the step defines; packed fp32 instructions are disabled.
"""

from __future__ import annotations

import os
import subprocess
import sys
from typing import Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libphub.so")

SOURCES = ["plan.cpp", "phub_api.cpp", "fused_step.hip"]
HEADERS = ["plan.hpp", "kernels.hpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",
    "-fno-fast-math",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def build(out: str = LIB, defines: Sequence[str] = (), extra: Sequence[str] = (),
          verbose: bool = False) -> str:
    """Compile and link the library; returns its path.  ``defines`` are
    extra -D settings (used for launch-shape sweeps)."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", *[f"-D{d}" for d in defines], *extra,
           *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
