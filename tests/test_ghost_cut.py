"""Host-side block cut of the ghost-zone fill (csrc/ghost_cut.h), on the CPU.

The cut splits targets 1..F-1 into runs of consecutive targets; the fill
relies on three properties, checked here independently of the cut's own
recurrence: every run has at most `max_rows` targets, every run's
dependency cone fits the halo (the heaviest chain of in-run pairs, summed
shifts, found by enumerating chains), and every run is maximal (the next
target would break one of the two), which makes the greedy cut the one with
the fewest runs.  The header is compiled with g++ into a test-local library
with its own wrapper; the product library exports nothing for it.
"""

import ctypes
import itertools
import os
import random
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1905_11722_amd", "csrc")

WRAPPER = r"""
#include "ghost_cut.h"
extern "C" int cut(int64_t F, const int32_t* near, int span, int max_rows, int32_t halo,
                   int32_t* out, int64_t cap) {
  std::vector<int32_t> nv(near, near + (F > 0 ? F * span : 0));
  const std::vector<int32_t> b = rcdp::ghost_cut_rows(F, nv, span, max_rows, halo);
  if ((int64_t)b.size() > cap) return -1;
  for (size_t i = 0; i < b.size(); i++) out[i] = b[i];
  return (int)b.size();
}
"""


@pytest.fixture(scope="module")
def cutlib(tmp_path_factory):
    d = tmp_path_factory.mktemp("ghost_cut")
    src = d / "wrap.cpp"
    src.write_text(WRAPPER)
    lib = d / "libcut.so"
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", "-I", CSRC,
                           str(src), "-o", str(lib)])
    h = ctypes.CDLL(str(lib))
    h.cut.restype = ctypes.c_int
    h.cut.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                      ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64]
    return h


def run_cut(h, F, near, span, max_rows, halo):
    near = np.ascontiguousarray(near, dtype=np.int32)
    out = np.zeros(F + 2, dtype=np.int32)
    k = h.cut(F, near.ctypes.data, span, max_rows, halo, out.ctypes.data, out.size)
    assert k > 0
    return [int(x) for x in out[:k]]


def shift(near, span, r, r2):
    d = r2 - r
    return int(near[r2 * span + d - 1]) if 1 <= d <= span else -1


def cone_by_chains(near, span, rows):
    """Heaviest chain r = a0 < a1 < ... < ak of in-run pairs, per start row,
    by enumerating every increasing sequence of rows."""
    best = {}
    for r in rows:
        later = [x for x in rows if x > r]
        top = 0
        for k in range(1, len(later) + 1):
            for seq in itertools.combinations(later, k):
                chain = (r,) + seq
                es = [shift(near, span, a, b) for a, b in zip(chain, chain[1:])]
                if all(e >= 0 for e in es):
                    top = max(top, sum(es))
        best[r] = top
    return best


def run_ok(near, span, rows, max_rows, halo):
    if len(rows) > max_rows:
        return False
    for i, r in enumerate(rows):                  # every in-run shift fits
        for r2 in rows[i + 1:]:
            if shift(near, span, r, r2) > halo:
                return False
    return max(cone_by_chains(near, span, rows).values()) <= halo


def check_cut(near, span, F, max_rows, halo, starts):
    assert starts[0] == 1 and starts[-1] == max(F, 1)
    assert all(a < b for a, b in zip(starts, starts[1:]))
    for a, b in zip(starts, starts[1:]):
        rows = list(range(a, b))
        assert run_ok(near, span, rows, max_rows, halo), (rows, halo)
        if b < F:                                  # maximal
            assert not run_ok(near, span, rows + [b], max_rows, halo), (rows, b)


def random_near(rng, F, span, p_pair, emax):
    near = np.full(F * span, -1, dtype=np.int32)
    for j in range(1, F):
        for d in range(1, min(span, j) + 1):
            if rng.random() < p_pair:
                near[j * span + d - 1] = rng.randint(0, emax)
    return near


@pytest.mark.parametrize("seed", range(12))
def test_random_shifts(cutlib, seed):
    rng = random.Random(seed)
    F = rng.randint(2, 70)
    span, max_rows = 8, 8
    halo = rng.choice([16, 64, 128])
    near = random_near(rng, F, span, rng.choice([0.2, 0.5, 0.9]), rng.choice([8, 40, 120]))
    starts = run_cut(cutlib, F, near, span, max_rows, halo)
    check_cut(near, span, F, max_rows, halo, starts)


def test_degenerate_sizes(cutlib):
    for F in (0, 1):
        assert run_cut(cutlib, F, np.zeros(0, np.int32), 8, 8, 64) == [1]
    assert run_cut(cutlib, 2, np.full(16, -1, np.int32), 8, 8, 64) == [1, 2]


def test_no_pairs_and_zero_shifts_fill_runs(cutlib):
    F = 30
    for value in (-1, 0):                           # no dependency / zero cones
        near = np.full(F * 8, value, dtype=np.int32)
        starts = run_cut(cutlib, F, near, 8, 8, 64)
        assert starts == [1, 9, 17, 25, 30]


def test_shift_above_halo_splits_every_pair(cutlib):
    F = 12
    near = np.full(F * 8, -1, dtype=np.int32)
    for j in range(2, F):
        near[j * 8 + 0] = 65                        # e(j-1, j) just above the halo
    starts = run_cut(cutlib, F, near, 8, 8, 64)
    assert starts == list(range(1, F + 1))
    near[:] = -1
    for j in range(2, F):
        near[j * 8 + 0] = 64                        # at the halo: pairs fit, chains do not
    starts = run_cut(cutlib, F, near, 8, 8, 64)
    assert starts == [1, 3, 5, 7, 9, 11, 12]        # targets 1..11 in pairs
    check_cut(near, 8, F, 8, 64, starts)


def test_chain_of_small_shifts_meets_the_halo(cutlib):
    """A chain of shifts 10: a run holds rows whose chained shift stays <= 64,
    i.e. 7 rows (cone 60), and the eighth would make 70."""
    F = 40
    near = np.full(F * 8, -1, dtype=np.int32)
    for j in range(2, F):
        near[j * 8 + 0] = 10
    starts = run_cut(cutlib, F, near, 8, 8, 64)
    check_cut(near, 8, F, 8, 64, starts)
    assert all(b - a == 7 for a, b in zip(starts[:-2], starts[1:-1]))
