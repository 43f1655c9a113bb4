// aggregate.hip -- weighted aggregation (Eqn 4b) and SGD update (Eqn 4c) for gfx950.
//
// g~[i] = sum_{j=0..K-1} r_j * v_j(i) over the devices' sparse (or dense)
// contributions. The positions are cut into tiles of kATile; one workgroup
// owns a tile and accumulates it in LDS in double, device by device in
// ascending order, one fused multiply-add per term (r_j * v is exact in
// double, so every term is rounded once, exactly as a serial double sum in
// device order would round it). No atomics: the result is bit-reproducible
// and independent of the launch shape. Nothing here is a dense contraction,
// so there is no MFMA: the bound is HBM traffic (sparse pairs in, dense out).
#include "scadles_internal.h"

namespace scadles {

typedef float f4 __attribute__((ext_vector_type(4)));

// Survivor offsets of each tile start, per device: off[j][t] = first position p
// of device j's sorted idx with idx[p] >= t * kATile; off[j][ntile] = k_j.
// Each entry is written by exactly one survivor when idx is strictly
// ascending. Optionally flags idx that is not strictly ascending or >= n.
__global__ __launch_bounds__(kBlock) void k_offsets(AggArgs a, AggCtx c, uint32_t validate)
{
  const uint32_t j = blockIdx.y;
  const uint32_t* idx = a.idx[j];
  if (!idx) return;
  const uint64_t k = a.k[j];
  uint32_t* off = c.off + (uint64_t)j * (c.ntile + 1);
  const uint32_t nt = c.ntile;
  if (k == 0) {
    if (blockIdx.x == 0)
      for (uint32_t t = threadIdx.x; t <= nt; t += kBlock) off[t] = 0u;
    return;
  }
  const uint64_t p0 = ((uint64_t)blockIdx.x * kBlock + threadIdx.x) * 4;
  for (uint64_t p = p0; p < p0 + 4 && p < k; ++p) {
    const uint32_t cur_i = idx[p];
    uint32_t cur = cur_i / kATile;
    if (cur > nt) cur = nt;
    int64_t prev = -1;
    if (p > 0) {
      const uint32_t prev_i = idx[p - 1];
      uint32_t pt = prev_i / kATile;
      prev = pt > nt ? nt : pt;
      if (validate && prev_i >= cur_i) atomicOr(c.err, 1u);
    }
    if (validate && cur_i >= c.n) atomicOr(c.err, 1u);
    for (int64_t t = prev + 1; t <= (int64_t)cur; ++t) off[t] = (uint32_t)p;
    if (p == k - 1)
      for (uint32_t t = cur + 1; t <= nt; ++t) off[t] = (uint32_t)k;
  }
}

__device__ inline bool dense_device(const AggArgs& a, const AggCtx& c, uint32_t j)
{
  if (c.st) return c.st[j].sparse == 0u;
  return a.idx[j] == nullptr;
}

// One tile: stage every device's entries of the tile (flattened in device
// order) into LDS with all loads in flight, then apply them device by device.
__global__ __launch_bounds__(kBlock) void k_aggregate(AggArgs a, AggCtx c)
{
  __shared__ double acc[kATile];
  __shared__ uint16_t s_pos[kAStage];
  __shared__ float s_val[kAStage];
  __shared__ uint32_t s_lo[kMaxK];
  __shared__ uint32_t s_pref[kMaxK + 1];
  __shared__ uint32_t s_dense[kMaxK];
  const uint32_t t = blockIdx.x, tid = threadIdx.x;
  const uint64_t base = (uint64_t)t * kATile;
  const uint32_t len = (uint32_t)((c.n - base < (uint64_t)kATile) ? c.n - base : (uint64_t)kATile);
  const uint32_t K = c.K;

  for (uint32_t e = tid; e < kATile; e += kBlock) acc[e] = 0.0;
  if (tid < K) {
    const uint32_t j = tid;
    uint32_t lo = 0, cnt = 0, dn = 0;
    if (dense_device(a, c, j)) {
      dn = 1;
      cnt = len;
    } else {
      const uint32_t* off = c.off + (uint64_t)j * (c.ntile + 1);
      const uint32_t kj = a.k[j];
      uint32_t l0 = off[t], l1 = off[t + 1];
      l0 = l0 > kj ? kj : l0;
      l1 = l1 > kj ? kj : l1;
      if (l1 < l0) l1 = l0;
      lo = l0;
      cnt = l1 - l0;
    }
    s_lo[j] = lo;
    s_dense[j] = dn;
    s_pref[j + 1] = cnt;
  }
  __syncthreads();
  if (tid == 0) {
    s_pref[0] = 0;
    for (uint32_t j = 0; j < K; ++j) s_pref[j + 1] += s_pref[j];
  }
  __syncthreads();
  const uint32_t total = s_pref[K];

  for (uint32_t c0 = 0; c0 < total; c0 += kAStage) {
    const uint32_t c1 = (c0 + kAStage < total) ? c0 + kAStage : total;
    // Stage: find the device of each flattened entry, load its position and value.
    for (uint32_t q = c0 + tid; q < c1; q += kBlock) {
      uint32_t lo = 0, hi = K;       // largest j with s_pref[j] <= q
      while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (s_pref[mid] <= q) lo = mid;
        else hi = mid;
      }
      const uint32_t j = lo;
      const uint32_t r = q - s_pref[j];
      uint32_t pos;
      float v;
      if (s_dense[j]) {
        pos = r;
        v = a.dense[j][base + r];
      } else {
        const uint64_t p = (uint64_t)s_lo[j] + r;
        const uint64_t i = a.idx[j][p];
        pos = (i >= base && i - base < len) ? (uint32_t)(i - base) : 0xFFFFu;
        v = a.val[j][p];
      }
      s_pos[q - c0] = (uint16_t)pos;
      s_val[q - c0] = v;
    }
    __syncthreads();
    // Apply in device order; a barrier between devices keeps the order per position.
    for (uint32_t j = 0; j < K; ++j) {
      const uint32_t b0 = s_pref[j] > c0 ? s_pref[j] : c0;
      const uint32_t b1 = s_pref[j + 1] < c1 ? s_pref[j + 1] : c1;
      if (b0 >= b1) continue;
      const double w = (double)a.w[j];
      for (uint32_t q = b0 + tid; q < b1; q += kBlock) {
        const uint32_t pos = s_pos[q - c0];
        if (pos < len) acc[pos] = __builtin_fma(w, (double)s_val[q - c0], acc[pos]);
      }
      __syncthreads();
    }
    __syncthreads();
  }

  // Round once to float; optionally the SGD update of Eqn 4c on the float aggregate.
  for (uint32_t e = tid * 4; e < len; e += kRound) {
    if (e + 4 <= len) {
      f4 g = {(float)acc[e], (float)acc[e + 1], (float)acc[e + 2], (float)acc[e + 3]};
      *reinterpret_cast<f4*>(c.out + base + e) = g;
      if (c.params) {
        f4 p = *reinterpret_cast<const f4*>(c.params + base + e);
        const double nlr = -(double)c.lr;
        p.x = (float)__builtin_fma(nlr, (double)g.x, (double)p.x);
        p.y = (float)__builtin_fma(nlr, (double)g.y, (double)p.y);
        p.z = (float)__builtin_fma(nlr, (double)g.z, (double)p.z);
        p.w = (float)__builtin_fma(nlr, (double)g.w, (double)p.w);
        *reinterpret_cast<f4*>(c.params + base + e) = p;
      }
    } else {
      for (uint32_t q = e; q < len; ++q) {
        const float g = (float)acc[q];
        c.out[base + q] = g;
        if (c.params)
          c.params[base + q] = (float)__builtin_fma(-(double)c.lr, (double)g, (double)c.params[base + q]);
      }
    }
  }
}

// Eqn 4c on its own: p <- p - lr * g, one fused multiply-add in double.
__global__ __launch_bounds__(kBlock) void k_sgd(float* p, const float* g, uint64_t n, float lr)
{
  const double nlr = -(double)lr;
  const uint64_t n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n4; i += stride) {
    f4 pv = *reinterpret_cast<const f4*>(p + 4 * i);
    const f4 gv = __builtin_nontemporal_load(reinterpret_cast<const f4*>(g + 4 * i));
    pv.x = (float)__builtin_fma(nlr, (double)gv.x, (double)pv.x);
    pv.y = (float)__builtin_fma(nlr, (double)gv.y, (double)pv.y);
    pv.z = (float)__builtin_fma(nlr, (double)gv.z, (double)pv.z);
    pv.w = (float)__builtin_fma(nlr, (double)gv.w, (double)pv.w);
    *reinterpret_cast<f4*>(p + 4 * i) = pv;
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const uint64_t i = 4 * n4 + threadIdx.x;
    p[i] = (float)__builtin_fma(nlr, (double)g[i], (double)p[i]);
  }
}

__global__ void k_zero_u32(uint32_t* p) { *p = 0u; }

hipError_t launch_aggregate(const AggArgs& a, const AggCtx& c, uint32_t validate, hipStream_t s)
{
  if (validate) k_zero_u32<<<1, 1, 0, s>>>(c.err);
  const uint32_t bx = c.kmax ? (uint32_t)((c.kmax + kRound - 1) / kRound) : 1u;
  if (c.K) k_offsets<<<dim3(bx, c.K), kBlock, 0, s>>>(a, c, validate);
  k_aggregate<<<c.ntile, kBlock, 0, s>>>(a, c);
  return hipGetLastError();
}

hipError_t launch_sgd(float* p, const float* g, uint64_t n, float lr, hipStream_t s)
{
  uint64_t blocks = (n / 4 + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 8192) blocks = 8192;
  k_sgd<<<(uint32_t)blocks, kBlock, 0, s>>>(p, g, n, lr);
  return hipGetLastError();
}

}  // namespace scadles
