"""Compile the C oracle with gcc: ``oracle/librcoracle.so`` (single-threaded)
and ``oracle/librcoracle_omp.so`` (the same source with OpenMP: the targets of
one source are shared among threads, giving the same tables)."""

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rc_oracle.c")
LIB = os.path.join(HERE, "librcoracle.so")
LIB_OMP = os.path.join(HERE, "librcoracle_omp.so")


def _compile(out, extra, verbose):
    cmd = (["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC"] + extra
           + [SRC, "-o", out + ".tmp"])
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


def build(verbose=False):
    _compile(LIB, ["-Wno-unknown-pragmas"], verbose)
    _compile(LIB_OMP, ["-fopenmp"], verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
