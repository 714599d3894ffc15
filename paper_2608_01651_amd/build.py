"""Build libtreelin.so for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2608_01651_amd.build [-v]

Every HIP source is compiled with packed fp32 instructions disabled (hipcc's
host pass prints a harmless "not a recognized feature" warning for that
flag).  Object files go to _build/ at the repository root.

A second library, libtreelin_debug.so, is built from the same sources with
-DTL_DEBUG: its verify kernels fill their LDS with NaN before first use, so
that a test run against it shows any read of LDS a kernel has not written.
The package loads libtreelin.so; only that test loads the debug library.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libtreelin.so")
LIB_DEBUG = os.path.join(PKG, "libtreelin_debug.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["verify.hip", "verify_tiled.hip", "verify_gla_large.hip", "verify_gdn_dense.hip", "commit.hip", "topology.hip", "conv.hip", "budget.hip",
           "abi.cpp"]
COMMON = ["-std=c++17", "-O3", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}",
          "-Wall", "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-fno-gpu-flush-denormals-to-zero"]


def _compile(src, verbose, debug=False):
    objdir = os.path.join(OBJDIR, "debug") if debug else OBJDIR
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    cmd = [HIPCC, "-c"] + (["-x", "hip"] if src.endswith(".hip") else []) + \
        [os.path.join(CSRC, src), "-o", obj] + COMMON + (["-DTL_DEBUG"] if debug else [])
    if src.endswith(".hip"):
        cmd += DEVICE
    else:
        cmd += ["-D__HIP_PLATFORM_AMD__"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(line for line in (r.stderr or "").splitlines() if noise not in line)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{err}")
    if verbose and err.strip():
        print(err, flush=True)
    return obj


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking {os.path.basename(lib)} failed:\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose=False, debug=True):
    """Compile and link libtreelin.so (and, with debug, libtreelin_debug.so)."""
    os.makedirs(os.path.join(OBJDIR, "debug"), exist_ok=True)
    jobs = [(s, False) for s in SOURCES] + ([(s, True) for s in SOURCES] if debug else [])
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        objs = list(ex.map(lambda j: _compile(j[0], verbose, j[1]), jobs))
    _link(objs[:len(SOURCES)], LIB, verbose)
    if debug:
        _link(objs[len(SOURCES):], LIB_DEBUG, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv[1:]))
