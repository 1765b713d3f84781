"""Build libsqn.so (the C-ABI render library) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB_PATH = os.path.join(PKG, "libsqn.so")
SOURCES = [os.path.join(CSRC, "api.hip"), os.path.join(CSRC, "render.hip"),
           os.path.join(CSRC, "prepare.hip"), os.path.join(CSRC, "generate.hip")]
# memory-level ceilings for the benchmark's roofline (not part of the render ABI)
PROBE_PATH = os.path.join(PKG, "libsqn_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "probe.hip")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # ray, sample, index and termination arithmetic is specified as one
    # rounding per written operation: no contraction into FMA, IEEE binary32
    # division and square root, denormals kept
    "-ffp-contract=off",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    # the SLP vectorizer packs the six box comparisons into bit vectors;
    # scalar compares into lane masks are cheaper
    "-fno-slp-vectorize",
    # no packed binary32 VALU forms (v_pk_fma_f32 and the like) in device
    # code; the host pass warns that it does not know the feature, the
    # device pass applies it (tests/test_build_guard.py checks the assembly)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-command-line-argument",
]


OBJ_DIR = os.path.join(PKG, "_build")


def _hipcc():
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _compile_one(src, verbose):
    obj = os.path.join(OBJ_DIR, os.path.basename(src) + ".o")
    cmd = [_hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", "-o", obj, src]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return obj


def _compile(sources, path, verbose):
    """Each source to an object in parallel, then one shared library."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(OBJ_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(sources), os.cpu_count() or 1)) as pool:
        objs = list(pool.map(lambda src: _compile_one(src, verbose), sources))
    tmp = path + ".tmp"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)


def build(verbose: bool = False) -> str:
    """Compile libsqn.so and libsqn_probe.so (always recompiles)."""
    _compile(SOURCES, LIB_PATH, verbose)
    _compile(PROBE_SOURCES, PROBE_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
