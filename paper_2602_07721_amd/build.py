"""Build libpariskv.so in-tree for gfx950.

    python -m paper_2602_07721_amd.build [--jobs N] [--verbose]

Each HIP translation unit is compiled separately with hipcc (no relocatable
device code: every kernel is launched from its own file), the quad-precision
quantizer derivation with the host C++ compiler, and everything is linked
into ``paper_2602_07721_amd/libpariskv.so``.  Always recompiles.
"""

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpariskv.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX_HOST", "g++")

HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # Packed FP32 instructions are kept out of every kernel.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    f"-I{os.path.join(ROOT, 'include')}",
]
# Files whose float64 decision path is specified operation by operation.
EXACT_FP = {"encode.hip", "stage1.hip"}
HIP_SOURCES = ["api.hip", "encode.hip", "stage1.hip", "stage2.hip", "attend.hip", "group_attend.hip",
               "calib.hip"]
CXX_SOURCES = ["quantizer.cpp"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # hipcc's host pass does not know the packed-fp32 target feature; that warning is expected.
    noise = [ln for ln in r.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln
             and "not a recognized feature for this target" not in ln]
    if noise and verbose:
        print("\n".join(noise), file=sys.stderr)
    return r


def compile_hip(src, verbose=False):
    obj = os.path.join(BUILD, src + ".o")
    flags = list(HIP_FLAGS)
    if src in EXACT_FP:
        flags.append("-ffp-contract=off")
    _run([HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
    return obj


def compile_cxx(src, verbose=False):
    obj = os.path.join(BUILD, src + ".o")
    _run([CXX, "-O2", "-std=c++17", "-fPIC", "-c", os.path.join(CSRC, src), "-o", obj], verbose)
    return obj


def build(jobs=None, verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(8, len(HIP_SOURCES) + len(CXX_SOURCES))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(compile_hip, s, verbose) for s in HIP_SOURCES]
        futs += [ex.submit(compile_cxx, s, verbose) for s in CXX_SOURCES]
        objs = [f.result() for f in futs]
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs, "-lquadmath"], verbose)
    shutil.move(tmp, LIB)
    return LIB


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--verbose", action="store_true")
    args = ap.parse_args()
    print(build(args.jobs, args.verbose))


if __name__ == "__main__":
    main()
