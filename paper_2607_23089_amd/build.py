"""Build the gfx950 row-softmax shared library (librowsm.so) in-tree.

``python -m paper_2607_23089_amd.build`` or ``build_library()``.  hipcc
cross-compiles for gfx950 without a GPU present.  The kernel families live in
separate translation units (csrc/launch_*.hip), compiled in parallel and
linked together with the launcher (csrc/plan.hip) and the C ABI
(csrc/rowsm.hip).
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librowsm.so")
SOURCES = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
HEADERS = sorted(glob.glob(os.path.join(CSRC, "*.hpp")))

# Packed-fp32 instructions are disabled for every HIP translation unit: the
# host pass warns that it does not know the feature, which is harmless.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Wall", "-Wextra", "-Wno-unused-parameter",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", INCLUDE, "-I", CSRC]
NOISE = "is not a recognized feature for this target"


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if NOISE not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{err}")
    return err


def build_library(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile librowsm.so (always recompiles); returns its path."""
    jobs = jobs or min(8, os.cpu_count() or 1, len(SOURCES))
    with tempfile.TemporaryDirectory(prefix="rowsm_build_") as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in SOURCES]
        cmds = [["hipcc"] + HIP_FLAGS + ["-c", s, "-o", o] for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            errs = list(pool.map(_run, cmds))
        tmp_lib = LIB + ".tmp"
        errs.append(_run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp_lib]
                         + objs))
    if verbose:
        for e in errs:
            if e.strip():
                print(e, file=sys.stderr)
    os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
