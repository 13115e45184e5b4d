// Traceback of the memory-indexed table (dual.hip).
#pragma once

#include "rc_internal.h"

namespace rcdp {

// Chain traced back through the table of launch_dual from st->t_sel /
// st->m_sel, and its strategy re-evaluated (Eq. 1, Eq. 2): chain[F], seg[n],
// cached[n], st->{k, overhead, peak, cache_mem}; st->error = 2 when the walk
// fails.
hipError_t launch_dual_trace(rc_family f, int32_t B, int32_t W, int objective, const uint32_t* D,
                             DevStatus* st, int32_t* chain, int32_t* seg, uint8_t* cached,
                             hipStream_t s);

}  // namespace rcdp
