"""Build commands of the native library (gfx950 only)."""

from __future__ import annotations

import os
import subprocess
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libumap_layout.so")

SOURCES = ["api.hip", "kernels_prep.hip", "kernels_layout.hip", "kernels_hogwild.hip", "kernels_graph.hip",
           "kernels_probe.hip", "kernels_trust.hip", "fit_ab.cpp"]

HIPCC_FLAGS = [
    "-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 VALU ops stay off (only scalar fp32 arithmetic is emitted)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # IEEE fp32 division: the edge schedule is a floor of a quotient
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    # no implicit fma contraction: every kernel variant rounds identically
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build_library(verbose: bool = False) -> str:
    """Compile csrc/ into libumap_layout.so next to this file (always rebuilds)."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"),
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    t0 = time.time()
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} in {time.time() - t0:.1f}s")
    return LIB


if __name__ == "__main__":
    build_library(verbose=True)
