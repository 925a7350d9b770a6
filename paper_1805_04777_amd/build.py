"""Build ``libconvcrf.so`` (the HIP library behind include/convcrf.h) for gfx950.

Every call compiles from source: each translation unit of ``csrc/`` goes to
its own object (the fused iteration, the fused blur iteration and the adjoint
message once per window side k), in parallel, and the objects are linked into ``paper_1805_04777_amd/libconvcrf.so``.  Objects
live in ``_build/`` at the repository root.

    python -m paper_1805_04777_amd.build [--jobs N] [--verbose]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libconvcrf.so")

WINDOW_SIDES = (1, 3, 5, 7, 9, 11, 13, 15)
ARCH = "gfx950"

# -packed-fp32-ops: no v_pk_*_f32 instructions are generated.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _units():
    units = []
    for k in WINDOW_SIDES:
        units.append((os.path.join(CSRC, "iter.hip"), os.path.join(BUILD, f"iter_k{k}.o"),
                      [f"-DCRF_K={k}"]))
        units.append((os.path.join(CSRC, "backward.hip"), os.path.join(BUILD, f"bwd_k{k}.o"),
                      [f"-DCRF_BWD_K={k}"]))
        units.append((os.path.join(CSRC, "blur.hip"), os.path.join(BUILD, f"blur_k{k}.o"),
                      [f"-DCRF_BLUR_K={k}"]))
    for name in ("aux", "backward", "features", "api"):
        units.append((os.path.join(CSRC, f"{name}.hip"), os.path.join(BUILD, f"{name}.o"), []))
    return units


def _compile(hipcc, src, obj, extra, verbose):
    cmd = [hipcc, *HIPCC_FLAGS, *extra, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature; that note is noise
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)} {extra}:\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return obj


def build(jobs: int | None = None, verbose: bool = False) -> str:
    """Compile every HIP source and link libconvcrf.so; returns its path."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(16, os.cpu_count() or 4)
    units = _units()
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda u: _compile(hipcc, *u, verbose), units))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--verbose", action="store_true")
    args = ap.parse_args(argv)
    print(build(args.jobs, args.verbose))


if __name__ == "__main__":
    main()
