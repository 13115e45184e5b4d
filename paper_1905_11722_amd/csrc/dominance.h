// The level fill with the dominance skip of Section 4.2 (fill.hip).
#pragma once

#include "rc_internal.h"

namespace rcdp {

// Algorithm 1 over the size levels with the skip: after each level its rows
// are reduced to their weak fronts (dominated cells stored as infinity) and
// we[L] (device, [F]) receives the end of row L's front; the next levels read
// source cells t < we[L] only.  sol->m must hold the initial condition.
hipError_t launch_fill_dominance(rc_solution sol, int32_t* we, hipStream_t s);

}  // namespace rcdp
