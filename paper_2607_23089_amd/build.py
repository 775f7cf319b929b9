"""Build the gfx950 row-softmax shared library (librowsm.so) in-tree.

``python -m paper_2607_23089_amd.build`` or ``build_library()``.  hipcc
cross-compiles for gfx950 without a GPU present.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librowsm.so")
SOURCES = [os.path.join(CSRC, "rowsm.hip")]
HEADERS = [os.path.join(CSRC, f) for f in
           ("rowsm_device.hpp", "small_row.hpp", "medium_row.hpp", "large_row.hpp",
            "split_row.hpp")]


def hipcc_command(out: str) -> list:
    # Packed-fp32 instructions are disabled for every HIP translation unit:
    # the host pass warns that it does not know the feature, which is harmless.
    return ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Wall", "-Wextra", "-Wno-unused-parameter",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC, "-o", out] + SOURCES


def build_library(verbose: bool = False) -> str:
    """Compile librowsm.so (always recompiles); returns its path."""
    tmp = LIB + ".tmp"
    cmd = hipcc_command(tmp)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
