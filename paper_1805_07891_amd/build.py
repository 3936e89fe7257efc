"""Builds the HIP libraries in-tree for gfx950: ``libphub.so`` (the
exchange step and its C interface) and ``libphub_probe.so`` (the bandwidth
probe that the benchmark times beside the step).

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
PROBE_LIB = os.path.join(PKG, "libphub_probe.so")
# Ablation build: the gradients loaded cache-allocating (run it with
# bench.py --library); not built by default.
GRADIENTS_CACHED_LIB = os.path.join(PKG, "libphub_gradients_cached.so")
PROBE_SOURCES = ["probe.hip"]

SOURCES = ["plan.cpp", "phub_api.cpp", "fused_step.hip", "step_noalloc.hip"]
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


def build_probe(out: str = PROBE_LIB, verbose: bool = False) -> str:
    """Compile the bandwidth probe library; returns its path."""
    srcs = [os.path.join(CSRC, s) for s in PROBE_SOURCES]
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, f"-I{INCLUDE}", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


def device_assembly(out: str, source: str = "fused_step.hip") -> str:
    """Compile one HIP source of the library to gfx950 device assembly (with
    its kernel metadata: registers, LDS, scratch, spills) at ``out``; the
    code-generation tests read it."""
    flags = [f for f in FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [HIPCC, *flags, f"-I{INCLUDE}", f"-I{CSRC}", "--cuda-device-only", "-S",
           os.path.join(CSRC, source), "-o", out]
    subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
    return out


def build_all(verbose: bool = False) -> None:
    build(verbose=verbose)
    build_probe(verbose=verbose)


def build_gradients_cached(verbose: bool = False) -> str:
    """The ablation library whose kernels load the gradients
    cache-allocating (PHUB_GRADIENT_LOADS_CACHED) instead of non-temporally."""
    return build(GRADIENTS_CACHED_LIB, defines=["PHUB_GRADIENT_LOADS_CACHED=1"], verbose=verbose)


if __name__ == "__main__":
    if "--gradients-cached" in sys.argv[1:]:
        build_gradients_cached(verbose=True)
    else:
        build_all(verbose=True)
    sys.exit(0)
