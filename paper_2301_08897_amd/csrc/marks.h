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

// Range markers: the first entry of device j in range r (positions
// [r * kARange, (r + 1) * kARange)) stores its position in rbeg[j][r], the last
// one stores its position + 1 in rend[j][r]; ranges without entries keep
// kNoEntry in rbeg. For ascending idx a range's entries are [rbeg, rend).
// Entries with idx >= n are skipped (only validation mode reports them).
// Each wave takes 1024 consecutive entries (16 per lane, all loads in flight);
// an entry's neighbours come from the adjacent lanes. Block bx of nbx for
// device j; check_dense: skip a device whose (final) decision is dense.
__device__ inline void mark_body(const AggArgs& a, const AggCtx& c, uint32_t j, uint32_t bx, uint32_t nbx,
                                 bool check_dense)
{
  constexpr int kPer = 16;
  const uint32_t* idx = a.idx[j];
  if (!idx || (check_dense && dense_device(a, c, j))) return;
  const uint64_t k = a.k[j];
  uint32_t* rb = c.rbeg + (uint64_t)j * c.nrange;
  uint32_t* re = c.rend + (uint64_t)j * c.nrange;
  const uint32_t l = lane_id();
  const uint64_t nwave = (uint64_t)nbx * kWaves;
  for (uint64_t b0 = ((uint64_t)bx * kWaves + (threadIdx.x >> 6)) * (64 * kPer); b0 < k;
       b0 += nwave * (64 * kPer)) {
    uint32_t x[kPer];
#pragma unroll
    for (int m = 0; m < kPer; ++m) {
      const uint64_t e = b0 + m * 64 + l;
      x[m] = e < k ? idx[e] : 0u;
    }
    const uint32_t before = b0 > 0 ? idx[b0 - 1] : 0u;
    const uint32_t after = b0 + 64 * kPer < k ? idx[b0 + 64 * kPer] : 0u;
#pragma unroll
    for (int m = 0; m < kPer; ++m) {
      const uint64_t e = b0 + m * 64 + l;
      uint32_t prev = __shfl_up(x[m], 1, 64);
      uint32_t next = __shfl_down(x[m], 1, 64);
      const uint32_t last_prev = m > 0 ? __builtin_amdgcn_readlane(x[m > 0 ? m - 1 : 0], 63) : before;
      const uint32_t first_next = m + 1 < kPer ? __builtin_amdgcn_readlane(x[m + 1 < kPer ? m + 1 : 0], 0) : after;
      if (l == 0) prev = last_prev;
      if (l == 63) next = first_next;
      const uint32_t i = x[m];
      if (e >= k || (uint64_t)i >= c.n) continue;
      const uint32_t r = i / (uint32_t)kARange;
      if (e == 0 || prev / (uint32_t)kARange != r) rb[r] = (uint32_t)e;
      if (e + 1 == k || next / (uint32_t)kARange != r) re[r] = (uint32_t)(e + 1);
    }
  }
}

}  // namespace scadles
