"""Build ``libdisco.so`` for gfx950 with hipcc (in-tree, under ``_build/``).

Usage: ``python -m paper_2209_13603_amd.build [--debug-bounds]``.  Every call
recompiles; ``--debug-bounds`` writes ``libdisco_debug_bounds.so`` instead,
the kernels' psi-index range checks compiled in.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(BUILD_DIR, "libdisco.so")
# The same library with the kernels' psi-index range checks compiled in.
DEBUG_BOUNDS_LIB_PATH = os.path.join(BUILD_DIR, "libdisco_debug_bounds.so")

SOURCES = ["disco_plan.cpp", "disco_pack.cpp", "disco_spectral_plan.cpp", "disco_abi.cpp", "disco_kernels.hip",
           "disco_fused.hip", "disco_spectral.hip", "disco_sweep.hip", "disco_stencil.hip", "disco_grad.hip",
           "disco_noalloc.hip", "disco_mfma.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
# roctx ranges around plan creation and the ops (no-ops without a profiler).
LIBS = ["-L" + os.path.join(ROCM, "lib"), "-lrocprofiler-sdk-roctx"]
ARCH = "gfx950"

# Packed-fp32 VALU instructions stay disabled in all device code.
COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass reports the device-only feature flag as unknown: harmless.
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError("command failed (%d): %s\n%s" % (r.returncode, " ".join(cmd), out))
    if verbose and out.strip():
        print(out)


def build(verbose: bool = False, jobs: int = 5, debug_bounds: bool = False) -> str:
    """Compile the library for gfx950; with debug_bounds the build that
    checks the kernels' psi indices (DISCO_DEBUG_BOUNDS), written beside it."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs, procs = [], []
    defs = ["-DDISCO_DEBUG_BOUNDS"] if debug_bounds else []
    out_path = DEBUG_BOUNDS_LIB_PATH if debug_bounds else LIB_PATH
    with tempfile.TemporaryDirectory(dir=BUILD_DIR) as tmp:
        for src in SOURCES:
            obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
            lang = ["-x", "hip"] if src.endswith(".hip") else []
            cmd = [HIPCC, *COMMON, *defs, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
            objs.append(obj)
            procs.append(cmd)
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            list(ex.map(lambda c: _run(c, verbose), procs))
        tmp_lib = os.path.join(tmp, "libdisco.so")
        _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, *LIBS, "-o", tmp_lib], verbose)
        os.replace(tmp_lib, out_path)
    return out_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, debug_bounds="--debug-bounds" in sys.argv))
