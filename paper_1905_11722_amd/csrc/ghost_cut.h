// Host-side cut of the targets into blocks for the ghost-zone fill
// (ghost.hip).  Plain C++ with no device dependency, so that the CPU tests
// can compile it on its own.
//
// Targets 1..F-1 (family order) are cut greedily into runs of at most
// max_rows consecutive targets whose dependency cone fits `halo` cells:
// for the rows r of a run, cone(last) = 0 and cone(r) = max over later rows
// r2 of the run with a pair (r, r2) of cone(r2) + e(r, r2), where e is the
// pair's right-aligned shift; every cone must be at most `halo` (so every
// in-run shift is too).  A run grows while the next target still fits;
// since any part of a run that fits also fits, the greedy cut has the fewest
// runs.  near[j * near_span + d - 1] is e(j - d, j), or -1 when (L_{j-d},
// L_j) is no pair; near_span >= max_rows - 1.
#pragma once

#include <stdint.h>

#include <algorithm>
#include <vector>

namespace rcdp {

inline std::vector<int32_t> ghost_cut_rows(int64_t F, const std::vector<int32_t>& near,
                                           int near_span, int max_rows, int32_t halo) {
  std::vector<int32_t> bstart;
  bstart.push_back(1);
  if (F < 2) return bstart;
  auto shift = [&](int64_t r, int64_t r2) -> int32_t {   // e(r, r2), r < r2
    const int64_t d = r2 - r;
    return d >= 1 && d <= near_span ? near[r2 * near_span + d - 1] : -1;
  };
  std::vector<int32_t> cone((size_t)max_rows + 1);
  int64_t start = 1;
  for (int64_t j = 2; j < F; j++) {
    // would rows start .. j still fit?  cone(j) = 0, then backwards
    const int64_t len = j - start + 1;
    bool fits = len <= max_rows;
    for (int64_t r = len - 1; fits && r >= 0; r--) {
      int32_t cr = 0;
      for (int64_t r2 = r + 1; r2 < len && fits; r2++) {
        const int32_t e = shift(start + r, start + r2);
        if (e < 0) continue;
        if (e > halo) fits = false;
        cr = std::max(cr, cone[r2] + e);
      }
      cone[r] = cr;
      if (cr > halo) fits = false;
    }
    if (!fits) {
      start = j;
      bstart.push_back((int32_t)j);
    }
  }
  bstart.push_back((int32_t)F);
  return bstart;
}

}  // namespace rcdp
