// aggregate.hip -- weighted aggregation (Eqn 4b) and SGD update (Eqn 4c) for gfx950.
//
// g~[i] = sum_{j=0..K-1} r_j * v_j(i) over the devices' sparse (or dense)
// contributions. One wave owns a tile of kATile positions at a time and
// accumulates it in LDS in double, device by device in ascending order, one
// rounding per term (r_j * v is exact in double, so every term is rounded
// once, exactly as a serial double sum in device order rounds it). The order
// needs no barrier: a wave's LDS operations (plain and atomic) execute in
// program order. No global atomics and no cross-wave races, so the result is
// bit-reproducible and independent of the launch shape. Nothing here is a dense contraction, so there is no MFMA: the bound is
// HBM traffic (sparse pairs in, dense aggregate out, parameters in and out).
#include "scadles_internal.h"

namespace scadles {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ inline bool dense_device(const AggArgs& a, const AggCtx& c, uint32_t j)
{
  if (c.st) return c.st[j].sparse == 0u;
  return a.idx[j] == nullptr;
}

// start[j][r] = first position p of device j's ascending idx with
// idx[p] >= r * kARange * kATile (binary search; any input gives a value in [0, k_j]).
__global__ __launch_bounds__(kBlock) void k_starts(AggArgs a, AggCtx c)
{
  const uint32_t per = c.nrange + 1;
  const uint64_t gid = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (gid >= (uint64_t)c.K * per) return;
  const uint32_t j = (uint32_t)(gid / per), r = (uint32_t)(gid - (uint64_t)j * per);
  const uint32_t* idx = a.idx[j];
  uint32_t lo = 0;
  if (idx) {
    const uint64_t target = (uint64_t)r * kARange * kATile;
    uint32_t hi = a.k[j];
    while (lo < hi) {
      const uint32_t mid = lo + (hi - lo) / 2;
      if ((uint64_t)idx[mid] < target) lo = mid + 1;
      else hi = mid;
    }
  }
  c.start[gid] = lo;
}

// Flags a set whose idx is not strictly ascending or reaches n (validation mode).
__global__ __launch_bounds__(kBlock) void k_validate(AggArgs a, AggCtx c)
{
  const uint32_t j = blockIdx.y;
  const uint32_t* idx = a.idx[j];
  if (!idx) return;
  const uint64_t p = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (p >= a.k[j]) return;
  const uint32_t cur = idx[p];
  if (cur >= c.n || (p > 0 && idx[p - 1] >= cur)) atomicOr(c.err, 1u);
}

// acc += p as one LDS read-modify-write. The LDS executes a wave's operations
// in program order, so device j's additions to a position precede device
// j+1's; p = r_j * v is exact in double, so acc + p rounds once, exactly like
// fma(r_j, v, acc).
__device__ inline void lds_add(double* a, double p)
{
  __hip_atomic_fetch_add(a, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// One wave per range of kARange tiles. Lane j < K keeps device j's survivor
// pointer; for each tile the wave loads the next 64 entries of kABatch devices
// at once (all loads in flight), then applies them device by device: the
// entries below the tile's end are consumed (for ascending idx they are a
// prefix of the lanes), the pointer advances by their count, and a device with
// 64 or more entries in the tile loops on. Dense devices add the whole tile.
__global__ __launch_bounds__(64) void k_aggregate(AggArgs a, AggCtx c)
{
  __shared__ double acc[kATile];
  const uint32_t l = threadIdx.x;
  const uint32_t K = c.K;
  const uint32_t rg = blockIdx.x;
  uint32_t ptr = 0, kj = 0, dn = 0;
  if (l < K) {
    kj = a.k[l];
    dn = dense_device(a, c, l) ? 1u : 0u;
    ptr = dn ? 0u : c.start[(uint64_t)l * (c.nrange + 1) + rg];
  }
  const uint32_t t0 = rg * kARange;
  const uint32_t t1 = (t0 + kARange < c.ntile) ? t0 + kARange : c.ntile;
  for (uint32_t t = t0; t < t1; ++t) {
    const uint64_t base = (uint64_t)t * kATile;
    const uint64_t tend = base + kATile;
    const uint32_t len = (uint32_t)((c.n - base < (uint64_t)kATile) ? c.n - base : (uint64_t)kATile);
    // Parameters of a full tile are fetched now, used after the accumulation.
    f4 pp[kATile / 256];
    const bool pre = c.params && len == (uint32_t)kATile;
    if (pre) {
#pragma unroll
      for (int m = 0; m < kATile / 256; ++m) pp[m] = *reinterpret_cast<const f4*>(c.params + base + m * 256 + l * 4);
    }
#pragma unroll
    for (int m = 0; m < kATile / 64; ++m) acc[m * 64 + l] = 0.0;

    for (uint32_t jb = 0; jb < K; jb += kABatch) {
      uint32_t ri[kABatch];
      float rv[kABatch];
      bool ok[kABatch];
#pragma unroll
      for (int jj = 0; jj < kABatch; ++jj) {
        const uint32_t j = jb + jj;
        ok[jj] = false;
        ri[jj] = 0u;
        rv[jj] = 0.f;
        if (j < K) {
          const uint32_t pj = __builtin_amdgcn_readlane(ptr, j);
          const uint32_t kk = __builtin_amdgcn_readlane(kj, j);
          const uint32_t dj = __builtin_amdgcn_readlane(dn, j);
          if (!dj && (uint64_t)pj + l < kk) {
            ok[jj] = true;
            ri[jj] = a.idx[j][pj + l];
            rv[jj] = a.val[j][pj + l];
          }
        }
      }
#pragma unroll
      for (int jj = 0; jj < kABatch; ++jj) {
        const uint32_t j = jb + jj;
        if (j >= K) break;
        const double w = (double)a.w[j];
        if (__builtin_amdgcn_readlane(dn, j)) {
          const float* g = a.dense[j] + base;
#pragma unroll 4
          for (int m = 0; m < kATile / 64; ++m) {
            const uint32_t e = m * 64 + l;
            if (e < len) lds_add(&acc[e], w * (double)g[e]);
          }
          continue;
        }
        bool take = ok[jj] && (uint64_t)ri[jj] < tend;
        uint32_t i = ri[jj];
        float v = rv[jj];
        while (true) {
          if (take && (uint64_t)i >= base) {
            const uint32_t pos = (uint32_t)(i - base);
            if (pos < len) lds_add(&acc[pos], w * (double)v);
          }
          const uint32_t cnt = (uint32_t)__builtin_popcountll(ballot(take));
          if (l == j) ptr += cnt;
          if (cnt < 64u) break;
          // 64 entries of this device fell in the tile: fetch the next 64.
          const uint32_t pj = __builtin_amdgcn_readlane(ptr, j);
          const uint32_t kk = __builtin_amdgcn_readlane(kj, j);
          const bool okn = (uint64_t)pj + l < kk;
          i = okn ? a.idx[j][pj + l] : 0u;
          v = okn ? a.val[j][pj + l] : 0.f;
          take = okn && (uint64_t)i < tend;
        }
      }
    }

    // Round once to float; optionally the SGD update of Eqn 4c on the float aggregate.
    if (pre) {
      const double nlr = -(double)c.lr;
#pragma unroll
      for (int m = 0; m < kATile / 256; ++m) {
        const uint32_t e = m * 256 + l * 4;
        const f4 g = {(float)acc[e], (float)acc[e + 1], (float)acc[e + 2], (float)acc[e + 3]};
        *reinterpret_cast<f4*>(c.out + base + e) = g;
        f4 p = pp[m];
        p.x = (float)__builtin_fma(nlr, (double)g.x, (double)p.x);
        p.y = (float)__builtin_fma(nlr, (double)g.y, (double)p.y);
        p.z = (float)__builtin_fma(nlr, (double)g.z, (double)p.z);
        p.w = (float)__builtin_fma(nlr, (double)g.w, (double)p.w);
        *reinterpret_cast<f4*>(c.params + base + e) = p;
      }
      continue;
    }
    for (uint32_t e = l * 4; e < len; e += 256) {
      if (e + 4 <= len) {
        const f4 g = {(float)acc[e], (float)acc[e + 1], (float)acc[e + 2], (float)acc[e + 3]};
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
  if (c.K) {
    if (validate) {
      k_zero_u32<<<1, 1, 0, s>>>(c.err);
      const uint32_t bx = c.kmax ? (uint32_t)((c.kmax + kBlock - 1) / kBlock) : 1u;
      k_validate<<<dim3(bx, c.K), kBlock, 0, s>>>(a, c);
    }
    const uint64_t ns = (uint64_t)c.K * (c.nrange + 1);
    k_starts<<<(uint32_t)((ns + kBlock - 1) / kBlock), kBlock, 0, s>>>(a, c);
  }
  k_aggregate<<<c.nrange, 64, 0, s>>>(a, c);
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
