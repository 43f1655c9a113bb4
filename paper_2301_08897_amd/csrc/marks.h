// marks.h -- range markers of the weighted aggregation (device code shared by
// the aggregation launch and the fused selection's decision launch).
#pragma once

#include "scadles_internal.h"

namespace scadles {

__device__ inline bool dense_device(const AggArgs& a, const AggCtx& c, uint32_t j)
{
  if (c.st) return c.st[j].sparse == 0u;
  return a.idx[j] == nullptr;
}

// lb[r] = number of entries of an ascending set with idx < r * kARange (the
// lower bound of the range start), for ranges r = t, t + nt, ... < nrange: a
// binary search over the set's idx. For any input the result is in [0, k].
__device__ inline void lb_ranges(const uint32_t* idx, uint32_t k, uint32_t* lb, uint32_t nrange, uint32_t t,
                                 uint32_t nt)
{
  for (uint32_t r = t; r < nrange; r += nt) {
    const uint64_t b = (uint64_t)r * kARange;
    uint32_t lo = 0, hi = k;
    while (lo < hi) {
      const uint32_t mid = lo + (hi - lo) / 2u;
      if ((uint64_t)idx[mid] < b) lo = mid + 1u;
      else hi = mid;
    }
    lb[r] = lo;
  }
}

}  // namespace scadles
