// aggregate.hip -- weighted aggregation (Eqn 4b) and SGD update (Eqn 4c) for gfx950.
//
// g~[i] = sum_{j=0..K-1} r_j * v_j(i) over the devices' sparse (or dense)
// contributions. One wave owns a range of kARange positions and accumulates it
// in LDS in double, device by device in ascending order, one rounding per term
// (r_j * v is exact in double, so every term is rounded once, exactly as a
// serial double sum in device order rounds it). The order needs no barrier: a
// wave's LDS operations (plain and atomic) execute in program order, and one
// device never has two entries at one position. No global atomics and no
// cross-wave races, so the result is bit-reproducible and independent of the
// launch shape. Nothing here is a dense contraction, so there is no MFMA: the
// bound is HBM traffic (sparse pairs in, dense aggregate out, parameters in
// and out).
#include "marks.h"

namespace scadles {

typedef float f4 __attribute__((ext_vector_type(4)));

// Range markers of every sparse device (one thread per range).
__global__ __launch_bounds__(kBlock) void k_lb(AggArgs a, AggCtx c)
{
  const uint32_t j = blockIdx.y;
  if (!a.idx[j] || dense_device(a, c, j)) return;
  lb_ranges(a.idx[j], a.k[j], c.lb + (uint64_t)j * c.nrange, c.nrange, blockIdx.x * kBlock + threadIdx.x,
            gridDim.x * kBlock);
}

// Range markers of sets this library built (ascending by construction) in one
// streaming pass over their idx instead of a search per range: position p
// (0 <= p <= k) is the marker of every range start in (idx[p-1], idx[p]],
// with idx[-1] below and idx[k] above every index, so each marker is written
// exactly once. A lane writes an interval of up to kMarkShort ranges itself;
// longer ones (sparse sets) are written by the whole wave. Writes stay below
// nrange for any input; for a set that is not ascending some markers keep
// older values, which the aggregation's clamping keeps in bounds.
constexpr uint32_t kMarkBatch = 8;    // positions per lane per pass
constexpr uint32_t kMarkShort = 4;
__global__ __launch_bounds__(kBlock) void k_marks(AggArgs a, AggCtx c)
{
  const uint32_t j = blockIdx.y;
  if (!a.idx[j] || dense_device(a, c, j)) return;
  const uint32_t* idx = a.idx[j];
  const uint32_t k = a.k[j];
  uint32_t* lb = c.lb + (uint64_t)j * c.nrange;
  const uint32_t l = lane_id();
  const uint32_t rlast = c.nrange - 1u;
  constexpr uint32_t kSpan = kMarkBatch * 64;
  const uint64_t np = (uint64_t)k + 1u;
  const uint64_t step = (uint64_t)gridDim.x * (kBlock / 64) * kSpan;
  for (uint64_t w0 = ((uint64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)) * kSpan; w0 < np; w0 += step) {
    uint32_t cur[kMarkBatch];
#pragma unroll
    for (int m = 0; m < (int)kMarkBatch; ++m) {
      const uint64_t p = w0 + m * 64 + l;
      cur[m] = p < k ? idx[p] : 0u;
    }
    uint32_t last = w0 > 0 ? idx[w0 - 1] : 0u;
#pragma unroll
    for (int m = 0; m < (int)kMarkBatch; ++m) {
      const uint64_t p = w0 + m * 64 + l;
      const uint32_t up = __shfl_up(cur[m], 1, 64);
      const uint32_t prev = l ? up : last;
      last = __builtin_amdgcn_readlane(cur[m], 63);
      const uint32_t ra = p ? prev / kARange + 1u : 0u;
      uint32_t rb = p < k ? cur[m] / kARange : rlast;
      if (rb > rlast) rb = rlast;
      const bool live = p < np && ra <= rb;
      const uint32_t pv = (uint32_t)p;
      if (live && rb - ra < kMarkShort)
        for (uint32_t r = ra; r <= rb; ++r) lb[r] = pv;
      uint64_t lm = ballot(live && rb - ra >= kMarkShort);
      while (lm) {
        const int q = __builtin_ctzll(lm);
        lm &= lm - 1;
        const uint32_t qa = __builtin_amdgcn_readlane(ra, q), qb = __builtin_amdgcn_readlane(rb, q);
        const uint32_t qp = __builtin_amdgcn_readlane(pv, q);
        for (uint32_t r = qa + l; r <= qb; r += 64) lb[r] = qp;
      }
    }
  }
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

// Adds one sparse entry (position i, value v) of weight w to the range at base.
__device__ inline void add_entry(double* acc, uint32_t i, float v, uint64_t base, double w)
{
  const uint64_t pos = (uint64_t)i - base;     // wraps for i < base: rejected below
  if (pos < (uint64_t)kARange) lds_add(&acc[pos], w * (double)v);
}

// First 64 entries of devices jb .. jb + kABatch - 1 in the range.
__device__ inline void load_batch(const AggArgs& a, uint32_t jb, uint32_t K, uint32_t eb, uint32_t em,
                                  uint32_t (&ri)[kABatch], float (&rv)[kABatch])
{
  const uint32_t l = lane_id();
#pragma unroll
  for (int jj = 0; jj < kABatch; ++jj) {
    const uint32_t j = jb + jj;
    ri[jj] = 0u;
    rv[jj] = 0.f;
    if (j < K) {
      const uint32_t b = __builtin_amdgcn_readlane(eb, j);
      const uint32_t m = __builtin_amdgcn_readlane(em, j);
      if (l < m) {
        ri[jj] = a.idx[j][b + l];
        rv[jj] = a.val[j][b + l];
      }
    }
  }
}

// Adds devices jb .. jb + kABatch - 1 in ascending order: the loaded first 64
// entries, then any further entries in rounds of four 64-entry windows, or the
// whole range of a dense device.
__device__ inline void add_batch(const AggArgs& a, double* acc, uint32_t jb, uint32_t K, uint32_t eb, uint32_t em,
                                 uint64_t dmask, uint64_t base, uint32_t len, const uint32_t (&ri)[kABatch],
                                 const float (&rv)[kABatch])
{
  const uint32_t l = lane_id();
#pragma unroll
  for (int jj = 0; jj < kABatch; ++jj) {
    const uint32_t j = jb + jj;
    if (j >= K) break;
    const double w = (double)a.w[j];
    if ((dmask >> j) & 1ull) {
      const float* g = a.dense[j] + base;
#pragma unroll 8
      for (int m = 0; m < kARange / 64; ++m) {
        const uint32_t e = m * 64 + l;
        if (e < len) lds_add(&acc[e], w * (double)g[e]);
      }
      continue;
    }
    const uint32_t b = __builtin_amdgcn_readlane(eb, j);
    const uint32_t m = __builtin_amdgcn_readlane(em, j);
    if (l < m) add_entry(acc, ri[jj], rv[jj], base, w);
    // Entries of one device hit distinct positions, so their order is free.
    for (uint32_t o = 64; o < m; o += 256) {
      uint32_t xi[4];
      float xv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t q = o + u * 64 + l;
        xi[u] = 0u;
        xv[u] = 0.f;
        if (q < m) {
          xi[u] = a.idx[j][b + q];
          xv[u] = a.val[j][b + q];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (o + u * 64 + l < m) add_entry(acc, xi[u], xv[u], base, w);
    }
  }
}

constexpr uint32_t kAGroup = 16;   // consecutive ranges per XCD turn

// One wave per range. Lane j < K holds device j's entry interval [eb, eb + em)
// in the range (from the range markers). Devices are added in ascending order,
// kABatch at a time (see load_batch / add_batch). Dense devices add the whole
// range from their gradient.
__global__ __launch_bounds__(64) void k_aggregate(AggArgs a, AggCtx c)
{
  __shared__ double acc[kARange];
  const uint32_t l = threadIdx.x;
  const uint32_t K = c.K;
  // Workgroups are dealt to the GPU's 8 XCDs in turn; consecutive groups of
  // kAGroup ranges go to one XCD, so the cache lines that neighbouring ranges
  // share (the markers, the ends of every device's entry window) are fetched
  // into one XCD's L2 rather than into several (1.14 -> 1.02 x the
  // algorithmic bytes fetched at the largest workload, same time).
  const uint32_t bq = blockIdx.x >> 3;
  const uint32_t r = (bq / kAGroup) * (8 * kAGroup) + (blockIdx.x & 7u) * kAGroup + bq % kAGroup;
  if (r >= c.nrange) return;
  const uint64_t base = (uint64_t)r * kARange;
  const uint32_t len = (uint32_t)((c.n - base < (uint64_t)kARange) ? c.n - base : (uint64_t)kARange);
  uint32_t eb = 0, em = 0;
  bool dn = false;
  if (l < K) {
    // both markers in one round trip
    const uint64_t at = (uint64_t)l * c.nrange + r;
    const uint32_t kk = a.k[l];
    const uint32_t b0 = c.lb[at];
    uint32_t e0 = r + 1 < c.nrange ? c.lb[at + 1] : kk;
    dn = dense_device(a, c, l);
    if (e0 > kk) e0 = kk;       // keeps any input in bounds; ascending input never needs it
    if (!dn && b0 < e0) {
      eb = b0;
      em = e0 - b0;
    }
  }
  const uint64_t dmask = ballot(dn);
  // Parameters (and momentum buffer) of a full range are fetched now, used after the accumulation.
  f4 pp[kARange / 256], vv[kARange / 256];
  const bool pre = c.params && len == (uint32_t)kARange;
  if (pre) {
#pragma unroll
    for (int m = 0; m < kARange / 256; ++m) pp[m] = *reinterpret_cast<const f4*>(c.params + base + m * 256 + l * 4);
    if (c.mbuf) {
#pragma unroll
      for (int m = 0; m < kARange / 256; ++m) vv[m] = *reinterpret_cast<const f4*>(c.mbuf + base + m * 256 + l * 4);
    }
  }
#pragma unroll
  for (int m = 0; m < kARange / 64; ++m) acc[m * 64 + l] = 0.0;

  // Batches of kABatch devices, double-buffered: the next batch's loads are in
  // flight while the current batch is added.
  uint32_t ia[kABatch], ib[kABatch];
  float va[kABatch], vb[kABatch];
  load_batch(a, 0, K, eb, em, ia, va);
  for (uint32_t jb = 0; jb < K; jb += 2 * kABatch) {
    if (jb + kABatch < K) load_batch(a, jb + kABatch, K, eb, em, ib, vb);
    add_batch(a, acc, jb, K, eb, em, dmask, base, len, ia, va);
    if (jb + kABatch >= K) break;
    if (jb + 2 * kABatch < K) load_batch(a, jb + 2 * kABatch, K, eb, em, ia, va);
    add_batch(a, acc, jb + kABatch, K, eb, em, dmask, base, len, ib, vb);
  }

  // Round once to float; optionally the SGD update of Eqn 4c (or momentum SGD
  // with weight decay) on the float aggregate. The aggregate and the momentum
  // buffer go out with nontemporal stores: nothing in the step reads them
  // again (0.03 and 0.025 ms less per step at the largest workload than plain
  // stores; the parameters' plain stores are faster than nontemporal ones).
  const double nlr = -(double)c.lr, mom = (double)c.mom, wd = (double)c.wd;
  if (pre) {
#pragma unroll
    for (int m = 0; m < kARange / 256; ++m) {
      const uint32_t e = m * 256 + l * 4;
      const f4 g = {(float)acc[e], (float)acc[e + 1], (float)acc[e + 2], (float)acc[e + 3]};
      __builtin_nontemporal_store(g, reinterpret_cast<f4*>(c.out + base + e));
      f4 p = pp[m];
      if (c.mbuf) {
        f4 v = vv[m];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float pq = p[q], vq = v[q];
          momentum_step(pq, vq, g[q], nlr, mom, wd);
          p[q] = pq;
          v[q] = vq;
        }
        __builtin_nontemporal_store(v, reinterpret_cast<f4*>(c.mbuf + base + e));
      } else {
        p.x = (float)__builtin_fma(nlr, (double)g.x, (double)p.x);
        p.y = (float)__builtin_fma(nlr, (double)g.y, (double)p.y);
        p.z = (float)__builtin_fma(nlr, (double)g.z, (double)p.z);
        p.w = (float)__builtin_fma(nlr, (double)g.w, (double)p.w);
      }
      *reinterpret_cast<f4*>(c.params + base + e) = p;
    }
    return;
  }
  for (uint32_t e = l * 4; e < len; e += 256) {
    if (e + 4 <= len) {
      const f4 g = {(float)acc[e], (float)acc[e + 1], (float)acc[e + 2], (float)acc[e + 3]};
      __builtin_nontemporal_store(g, reinterpret_cast<f4*>(c.out + base + e));
      if (c.params) {
        f4 p = *reinterpret_cast<const f4*>(c.params + base + e);
        if (c.mbuf) {
          f4 v = *reinterpret_cast<const f4*>(c.mbuf + base + e);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float pq = p[q], vq = v[q];
            momentum_step(pq, vq, g[q], nlr, mom, wd);
            p[q] = pq;
            v[q] = vq;
          }
          __builtin_nontemporal_store(v, reinterpret_cast<f4*>(c.mbuf + base + e));
        } else {
          p.x = (float)__builtin_fma(nlr, (double)g.x, (double)p.x);
          p.y = (float)__builtin_fma(nlr, (double)g.y, (double)p.y);
          p.z = (float)__builtin_fma(nlr, (double)g.z, (double)p.z);
          p.w = (float)__builtin_fma(nlr, (double)g.w, (double)p.w);
        }
        *reinterpret_cast<f4*>(c.params + base + e) = p;
      }
    } else {
      for (uint32_t q = e; q < len; ++q) {
        const float g = (float)acc[q];
        c.out[base + q] = g;
        if (c.params && c.mbuf) {
          float p = c.params[base + q], v = c.mbuf[base + q];
          momentum_step(p, v, g, nlr, mom, wd);
          c.mbuf[base + q] = v;
          c.params[base + q] = p;
        } else if (c.params) {
          c.params[base + q] = (float)__builtin_fma(nlr, (double)g, (double)c.params[base + q]);
        }
      }
    }
  }
}

// Eqn 4c on its own: p <- p - lr * g, one fused multiply-add in double. One
// float4 of each operand per thread and no loop: every load of the launch is
// independent, which keeps the most bytes in flight (a grid-stride loop with
// the same arithmetic measured 25% slower on the largest workload's size).
__global__ __launch_bounds__(kBlock) void k_sgd(float* p, const float* g, uint64_t n, float lr)
{
  const double nlr = -(double)lr;
  const uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n / 4) {
    f4 pv = *reinterpret_cast<const f4*>(p + 4 * i);
    const f4 gv = __builtin_nontemporal_load(reinterpret_cast<const f4*>(g + 4 * i));
    pv.x = (float)__builtin_fma(nlr, (double)gv.x, (double)pv.x);
    pv.y = (float)__builtin_fma(nlr, (double)gv.y, (double)pv.y);
    pv.z = (float)__builtin_fma(nlr, (double)gv.z, (double)pv.z);
    pv.w = (float)__builtin_fma(nlr, (double)gv.w, (double)pv.w);
    *reinterpret_cast<f4*>(p + 4 * i) = pv;
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const uint64_t t = (n & ~3ull) + threadIdx.x;
    p[t] = (float)__builtin_fma(nlr, (double)g[t], (double)p[t]);
  }
}

__global__ void k_zero_u32(uint32_t* p) { *p = 0u; }

// Range markers of every sparse device.
hipError_t launch_marks(const AggArgs& a, const AggCtx& c, hipStream_t s)
{
  if (!c.K || !c.nrange) return hipSuccess;
  uint32_t bx = (c.nrange + kBlock - 1) / kBlock;
  if (bx > 64) bx = 64;
  k_lb<<<dim3(bx, c.K), kBlock, 0, s>>>(a, c);
  return hipGetLastError();
}

// Range markers of sets this library built, by a streaming pass (k_marks).
hipError_t launch_marks_built(const AggArgs& a, const AggCtx& c, hipStream_t s)
{
  if (!c.K || !c.nrange) return hipSuccess;
  constexpr uint64_t kPerBlock = (kBlock / 64) * kMarkBatch * 64;
  uint64_t bx = ((uint64_t)c.kmax + kPerBlock) / kPerBlock;
  if (bx > 1024) bx = 1024;
  k_marks<<<dim3((uint32_t)bx, c.K), kBlock, 0, s>>>(a, c);
  return hipGetLastError();
}

// marks_done: the range markers of every device were built earlier on this stream.
hipError_t launch_aggregate(const AggArgs& a, const AggCtx& c, uint32_t validate, bool marks_done, hipStream_t s)
{
  if (c.K) {
    if (validate) {
      k_zero_u32<<<1, 1, 0, s>>>(c.err);
      const uint32_t bx = c.kmax ? (uint32_t)((c.kmax + kBlock - 1) / kBlock) : 1u;
      k_validate<<<dim3(bx, c.K), kBlock, 0, s>>>(a, c);
    }
    if (!marks_done) {
      const hipError_t e = launch_marks(a, c, s);
      if (e != hipSuccess) return e;
    }
  }
  k_aggregate<<<(c.nrange + 8 * kAGroup - 1) / (8 * kAGroup) * (8 * kAGroup), 64, 0, s>>>(a, c);
  return hipGetLastError();
}

// Momentum SGD with weight decay on its own (same arithmetic as the fused
// update), one float4 of each operand per thread like k_sgd.
__global__ __launch_bounds__(kBlock) void k_momentum_sgd(float* p, float* v, const float* g, uint64_t n, float lr,
                                                         float mom, float wd)
{
  const double nlr = -(double)lr, mu = (double)mom, dw = (double)wd;
  const uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n / 4) {
    f4 pv = *reinterpret_cast<const f4*>(p + 4 * i);
    f4 vv = *reinterpret_cast<const f4*>(v + 4 * i);
    const f4 gv = __builtin_nontemporal_load(reinterpret_cast<const f4*>(g + 4 * i));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float pq = pv[q], vq = vv[q];
      momentum_step(pq, vq, gv[q], nlr, mu, dw);
      pv[q] = pq;
      vv[q] = vq;
    }
    *reinterpret_cast<f4*>(v + 4 * i) = vv;
    *reinterpret_cast<f4*>(p + 4 * i) = pv;
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const uint64_t t = (n & ~3ull) + threadIdx.x;
    float pt = p[t], vt = v[t];
    momentum_step(pt, vt, g[t], nlr, mu, dw);
    v[t] = vt;
    p[t] = pt;
  }
}

// One thread per float4 (at least one workgroup, for the tail of n < 4).
static uint32_t elementwise_blocks(uint64_t n)
{
  const uint64_t b = (n / 4 + kBlock - 1) / kBlock;
  return (uint32_t)(b < 1 ? 1 : b);
}

hipError_t launch_momentum_sgd(float* p, float* v, const float* g, uint64_t n, float lr, float mom, float wd,
                               hipStream_t s)
{
  k_momentum_sgd<<<elementwise_blocks(n), kBlock, 0, s>>>(p, v, g, n, lr, mom, wd);
  return hipGetLastError();
}

hipError_t launch_sgd(float* p, const float* g, uint64_t n, float lr, hipStream_t s)
{
  k_sgd<<<elementwise_blocks(n), kBlock, 0, s>>>(p, g, n, lr);
  return hipGetLastError();
}

}  // namespace scadles
