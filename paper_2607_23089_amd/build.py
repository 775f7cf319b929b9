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
# host pass warns that it does not know the feature, which is harmless.  The
# device code objects are stored compressed (--offload-compress; the HIP
# runtime unpacks them when the library loads), which takes the library from
# about 23 MiB to about 8 MiB.
HIP_FLAGS = ["--offload-arch=gfx950", "--offload-compress", "-O3", "-std=c++17", "-fPIC",
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


# Translation units of the host-logic check build: the planner, the argument
# checks and C ABI, the exchange ring and the streaming copy.
HOST_CHECK_SOURCES = ["plan.hip", "rowsm.hip", "launch_split_common.hip", "stream_copy.hip"]
# Host-side sanitizers only; device code is built as usual.
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                 "-g"]


def build_host_check(out: str, stubs: str, jobs: int | None = None) -> str:
    """Build the host-logic check library at ``out``: HOST_CHECK_SOURCES plus
    ``stubs`` (launchers that launch nothing) with the host compiler's address
    and undefined-behaviour sanitizers.  Load it with the sanitizer runtime
    preloaded (sanitizer_runtime())."""
    srcs = [os.path.join(CSRC, f) for f in HOST_CHECK_SOURCES] + [stubs]
    flags = [f for f in HIP_FLAGS if f != "-O3"] + ["-O1"] + HOST_SANITIZE
    with tempfile.TemporaryDirectory(prefix="rowsm_check_") as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        cmds = [["hipcc"] + flags + ["-c", s, "-o", o] for s, o in zip(srcs, objs)]
        with ThreadPoolExecutor(max_workers=jobs or min(4, os.cpu_count() or 1)) as pool:
            list(pool.map(_run, cmds))
        _run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libasan", "-o", out]
             + HOST_SANITIZE + objs)
    return out


def sanitizer_runtime() -> str:
    """Path of the compiler's shared address-sanitizer runtime."""
    res = subprocess.run(["hipcc", "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True)
    return res.stdout.strip()


if __name__ == "__main__":
    print(build_library(verbose=True))
