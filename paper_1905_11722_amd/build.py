"""Compile the HIP libraries for gfx950 with hipcc.

All HIP sources under ``csrc/`` are compiled into one shared library,
``librcdp.so``, next to this file: the solver behind include/rc.h.  The
microbenchmarks of the chip's peaks under ``peak/`` (measurement only, not
part of the solver) go into ``libpeak.so``.  Packed-FP32 instruction
selection is disabled.
"""

import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "librcdp.so")
PEAK_LIB = os.path.join(HERE, "libpeak.so")
ARCH = os.environ.get("RCDP_OFFLOAD_ARCH", "gfx950")


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


OBJ_DIR = os.path.join(ROOT, "_build")
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]


def command(out, srcs=None):
    """One hipcc line that builds the shared library from the sources."""
    return ["hipcc"] + FLAGS + ["-shared"] + (sources() if srcs is None else srcs) + ["-o", out]


def _compile(lib, srcs, verbose):
    """Each source to an object (in parallel), then one shared library."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    objs = [os.path.join(OBJ_DIR, os.path.basename(src) + ".o") for src in srcs]

    def one(pair):
        src, obj = pair
        cmd = ["hipcc"] + FLAGS + ["-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)

    jobs = max(1, min(len(srcs), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4))))
    with ThreadPoolExecutor(jobs) as pool:
        list(pool.map(one, zip(srcs, objs)))
    tmp = lib + ".tmp"
    cmd = ["hipcc", f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, lib)


def build(verbose=False):
    _compile(LIB, sources(), verbose)
    _compile(PEAK_LIB, sorted(glob.glob(os.path.join(HERE, "peak", "*.hip"))), verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
