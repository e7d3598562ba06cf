// Residency of the code cache's entries (locality.cpp), shared with the
// library's update step (api.cpp).
#pragma once

#include <cstdint>

#include "fcg.h"

namespace fcg {
// resident[n] = which entries stay in device memory under budget: pinned
// entries first, then descending locality score; with tau > 0 entries whose
// perplexity is below tau after all the others.  Errors: EINVAL.
fcg_status locality_residency(const fcg_locality* L, int64_t budget, const int64_t* cost, double tau,
                              const uint8_t* pinned, uint8_t* resident);
// number of functions the scorer tracks (0 for a null handle)
int32_t locality_size(const fcg_locality* L);
}  // namespace fcg
