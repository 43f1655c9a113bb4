// frame.h -- how the selection kernels see a gradient: 16-byte vector loads in
// a 16-byte-aligned "virtual" frame, pad values outside the real range, and
// the ranking key of a magnitude. Internal to libscadles.
#pragma once

#include "scadles_internal.h"

namespace scadles {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));


// Pointers read from the device descriptors are generic; marking them global
// lets the compiler emit global_* instead of flat_* memory instructions.
// (The host compilation pass of this file sees plain pointers.)
#if defined(__HIP_DEVICE_COMPILE__)
#define GLOBAL __attribute__((address_space(1)))
#else
#define GLOBAL
#endif
template <class T>
__device__ inline const GLOBAL T* gptr(const T* p) { return (const GLOBAL T*)p; }
template <class T>
__device__ inline GLOBAL T* gptr(T* p) { return (GLOBAL T*)p; }

__device__ inline f4 ld_stream4(const GLOBAL float* p) { return __builtin_nontemporal_load((const GLOBAL f4*)p); }
__device__ inline f4 ld4(const GLOBAL float* p) { return *(const GLOBAL f4*)p; }
#if defined(__HIP_DEVICE_COMPILE__)
__device__ inline f4 ld_stream4(const float* p) { return ld_stream4(gptr(p)); }
__device__ inline f4 ld4(const float* p) { return ld4(gptr(p)); }
#endif
__device__ inline u4 ldu4(const uint32_t* p) { return *(const GLOBAL u4*)gptr(p); }

// A device's gradient seen in a 16-byte-aligned "virtual" frame: real element i
// sits at virtual position i + shift, shift = (address / 4) % 4, so every group
// of 4 virtual positions is one aligned 16-byte word. Positions outside the real
// range read as the pad pattern 0xFFFFFFFF, which rank_key maps to 0.
struct Row {
  const GLOBAL float* p;   // real element 0
  uint64_t shift;      // 0..3
  uint64_t n;          // real elements
};

constexpr uint32_t kPadBits = 0xFFFFFFFFu;

__device__ inline f4 load4(const Row& r, uint64_t v, bool stream)
{
  if (v >= r.shift && v + 4 <= r.shift + r.n) {
    const GLOBAL float* a = r.p + (v - r.shift);
    return stream ? ld_stream4(a) : ld4(a);
  }
  const float pad = __uint_as_float(kPadBits);
  f4 x = {pad, pad, pad, pad};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint64_t u = v + q;
    if (u >= r.shift && u < r.shift + r.n) x[q] = r.p[u - r.shift];
  }
  return x;
}

__device__ inline bool in_row(const Row& r, uint64_t v) { return v >= r.shift && v < r.shift + r.n; }

// Ranking key offset by one: 0 for the pad pattern, key + 1 for every finite
// value (finite keys are at most 0x7F7FFFFF, so nothing else wraps). Counting
// on it needs no validity masks: a pad is never above or equal to key + 1 >= 1.
__device__ inline uint32_t rank_key(float x) { return ((__float_as_uint(x) & kKeyMask) + 1u) & kKeyMask; }

}  // namespace scadles
