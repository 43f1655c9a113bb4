// rows.hip -- per-layer Top-k of short layers (the per-layer reading of the
// Top-k of §IV, ScaDLES arXiv 2301.08897): every (device, layer) row whose
// layer has at most a few million elements is selected by one workgroup, all
// such rows of all devices in one launch, instead of one multi-launch
// selection per layer.
//
// A row's k-th largest key (31-bit magnitude key, ties to the lower index) is
// found digit by digit, 12 + 10 + 9 bits: a histogram of the top digit over
// the row (one read, with sum g^2); once the keys that share the decided
// digits fit in LDS they are collected there (a second read) and the remaining
// digits are decided in LDS; a bin too large for LDS is refined by another
// histogram read instead. A last read writes the kept entries in index order:
// keys above the threshold, and keys equal to it while fewer than `need` came
// before.
#include "frame.h"

namespace scadles {

namespace {

constexpr int kRowWaves = kRowBlock / 64;
constexpr int kRowLevels = 3;
// digit `level` of a key: bits [shift, shift + width)
__device__ inline uint32_t level_shift(int level) { return level == 0 ? 19u : (level == 1 ? 9u : 0u); }
__device__ inline uint32_t level_width(int level) { return level == 0 ? 12u : (level == 1 ? 10u : 9u); }
constexpr uint32_t kRowBins = 1u << 12;
constexpr uint64_t kNotShort = ~0ull;

// Inclusive scan of one value per thread in thread order over the workgroup;
// `total` receives the sum. Contains two barriers.
__device__ inline uint32_t row_scan(uint32_t v, uint32_t* s_w, uint32_t& total)
{
  const uint32_t w = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v);
  if (lane_id() == 63) s_w[w] = incl;
  __syncthreads();
  uint32_t base = 0, tot = 0;
  for (uint32_t i = 0; i < (uint32_t)kRowWaves; ++i) {
    const uint32_t x = s_w[i];
    base += i < w ? x : 0u;
    tot += x;
  }
  total = tot;
  __syncthreads();
  return base + incl;
}

// Fixed-order sum of one double per thread over the workgroup.
__device__ inline double row_sum_f64(double v, double* s_d)
{
  v = wave_sum_f64(v);
  if (lane_id() == 0) s_d[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
  for (int i = 0; i < kRowWaves; ++i) r += s_d[i];
  __syncthreads();
  return r;
}

// The bin of `hist` (2^width bins) holding the rank-th largest key, counting
// from the top bin: s_res = {bin, keys in higher bins, keys in the bin}.
__device__ inline void row_select_bin(const uint32_t* hist, uint32_t width, uint32_t rank, uint32_t* s_w,
                                      uint32_t* s_res)
{
  const uint32_t bins = 1u << width;
  const uint32_t per = bins > (uint32_t)kRowBlock ? bins / kRowBlock : 1u;
  const uint32_t t = threadIdx.x;
  const bool owns = t * per < bins;
  uint32_t v = 0;
  if (owns)
    for (uint32_t i = 0; i < per; ++i) v += hist[bins - 1 - (t * per + i)];
  uint32_t tot;
  const uint32_t incl = row_scan(v, s_w, tot);
  const uint32_t excl = incl - v;
  if (owns && excl < rank && rank <= incl) {
    uint32_t above = excl;
    for (uint32_t i = 0; i < per; ++i) {
      const uint32_t b = bins - 1 - (t * per + i);
      const uint32_t h = hist[b];
      if (rank <= above + h) {
        s_res[0] = b;
        s_res[1] = above;
        s_res[2] = h;
        break;
      }
      above += h;
    }
  }
  __syncthreads();
}

struct PutArgs {
  uint64_t v[kPutWords];
  uint64_t* dst;
  uint32_t count;
};

// Copies a table chunk from the kernel arguments to device memory.
__global__ __launch_bounds__(256) void k_put(PutArgs a)
{
  for (uint32_t i = threadIdx.x; i < a.count; i += blockDim.x) a.dst[i] = a.v[i];
}

// One workgroup per device: every layer's k (the same rule as the host's),
// the exclusive prefix of k over the layers (where the layer's entries start
// in the device's output), and the row descriptors of the short layers.
__global__ __launch_bounds__(256) void k_rows_prep(RowsCtx rc, RowsPrep rp)
{
  __shared__ uint64_t s_w[4];
  const uint32_t j = blockIdx.x, tid = threadIdx.x;
  const double ratio = rp.ratio[j];
  uint64_t run = 0;
  for (uint32_t l0 = 0; l0 < rc.L; l0 += 256) {
    const uint32_t l = l0 + tid;
    uint64_t off = 0, nl = 0, kl = 0;
    if (l < rc.L) {
      off = rc.table[l];
      nl = rc.table[l + 1] - off;
      kl = k_of(nl, ratio);
    }
    uint64_t incl = kl;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t t = __shfl_up(incl, d, 64);
      if (lane_id() >= (uint32_t)d) incl += t;
    }
    if (lane_id() == 63) s_w[tid >> 6] = incl;
    __syncthreads();
    uint64_t pre = run + incl - kl;
    for (uint32_t i = 0; i < (tid >> 6); ++i) pre += s_w[i];
    const uint64_t chunk = s_w[0] + s_w[1] + s_w[2] + s_w[3];
    __syncthreads();
    if (l < rc.L) {
      const uint64_t q = rc.table[rc.L + 1 + l];
      if (q != kNotShort) {
        RowDesc d;
        d.grad = rp.grad[j] + off;
        d.idx_out = rp.idx[j] + pre;
        d.val_out = rp.val[j] + pre;
        d.n = (uint32_t)nl;
        d.k = (uint32_t)kl;
        d.base = (uint32_t)off;
        d.eslot = j * rc.L + l;
        rc.rows[q * rc.K + j] = d;
      }
    }
    run += chunk;
  }
}

// The selection of one row (see the top of this file).
__global__ __launch_bounds__(kRowBlock) __attribute__((amdgpu_waves_per_eu(8, 8))) void k_rows(RowsCtx rc)
{
  __shared__ uint32_t hist[kRowBins];
  __shared__ uint32_t cand[kRowCand];
  __shared__ uint32_t s_w[kRowWaves];
  __shared__ uint32_t s_res[4];
  __shared__ double s_d[kRowWaves];
  const RowDesc d = rc.rows[blockIdx.x];
  const uint32_t tid = threadIdx.x;
  const Row row{gptr(d.grad), ((uint64_t)d.grad >> 2) & 3u, d.n};
  const uint64_t vend = (uint64_t)d.n + row.shift;
  constexpr uint64_t kStep = (uint64_t)kRowBlock * 4;

  // top digit over the row, and sum g^2
  for (uint32_t i = tid; i < kRowBins; i += kRowBlock) hist[i] = 0u;
  __syncthreads();
  double e_all = 0.0;
  for (uint64_t v = (uint64_t)tid * 4; v < vend; v += kStep) {
    const f4 x = load4(row, v, false);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (in_row(row, v + q)) {
        atomicAdd(&hist[key_of(x[q]) >> level_shift(0)], 1u);
        e_all = __builtin_fma((double)x[q], (double)x[q], e_all);
      }
    }
  }
  {
    const double ea = row_sum_f64(e_all, s_d);  // (its barriers also complete the histogram)
    if (tid == 0) rc.row_e[2ull * d.eslot] = ea;
  }

  uint32_t rank = d.k, prefix = 0, pbits = 0, m = 0;
  bool in_lds = false;
  for (int level = 0;; ++level) {
    if (tid == 0) s_res[0] = s_res[1] = s_res[2] = 0u;
    row_select_bin(hist, level_width(level), rank, s_w, s_res);
    const uint32_t b = s_res[0], above = s_res[1], h = s_res[2];
    rank -= above;
    prefix = (prefix << level_width(level)) | b;
    pbits += level_width(level);
    if (level + 1 == kRowLevels) break;
    const uint32_t pshift = 31u - pbits;
    if (!in_lds && h <= (uint32_t)kRowCand) {
      // the keys sharing the decided digits fit in LDS: collect them
      if (tid == 0) s_res[3] = 0u;
      __syncthreads();
      for (uint64_t v = (uint64_t)tid * 4; v < vend; v += kStep) {
        const f4 x = load4(row, v, false);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t key = key_of(x[q]);
          if (in_row(row, v + q) && (key >> pshift) == prefix) {
            const uint32_t at = atomicAdd(&s_res[3], 1u);
            if (at < (uint32_t)kRowCand) cand[at] = key;
          }
        }
      }
      __syncthreads();
      m = s_res[3] < (uint32_t)kRowCand ? s_res[3] : (uint32_t)kRowCand;
      in_lds = true;
    }
    // histogram of the next digit over the keys sharing the decided digits
    const uint32_t nshift = level_shift(level + 1), nmask = (1u << level_width(level + 1)) - 1u;
    __syncthreads();
    for (uint32_t i = tid; i < kRowBins; i += kRowBlock) hist[i] = 0u;
    __syncthreads();
    if (in_lds) {
      for (uint32_t i = tid; i < m; i += kRowBlock) {
        const uint32_t key = cand[i];
        if ((key >> pshift) == prefix) atomicAdd(&hist[(key >> nshift) & nmask], 1u);
      }
    } else {
      for (uint64_t v = (uint64_t)tid * 4; v < vend; v += kStep) {
        const f4 x = load4(row, v, false);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t key = key_of(x[q]);
          if (in_row(row, v + q) && (key >> pshift) == prefix) atomicAdd(&hist[(key >> nshift) & nmask], 1u);
        }
      }
    }
    __syncthreads();
  }
  const uint32_t thr = prefix, need = rank;

  // ordered output: 4096 positions per round, kept positions by a workgroup scan
  uint32_t run_g = 0, run_e = 0;
  double e_kept = 0.0;
  GLOBAL uint32_t* oi = gptr(d.idx_out);
  GLOBAL float* ov = gptr(d.val_out);
#pragma unroll 1
  for (uint64_t v0 = 0; v0 < vend; v0 += kStep) {
    const uint64_t v = v0 + (uint64_t)tid * 4;
    const f4 x = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
    bool g[4], e[4];
    uint32_t cg = 0, ce = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool valid = v < vend && in_row(row, v + q);
      const uint32_t key = key_of(x[q]);
      g[q] = valid && key > thr;
      e[q] = valid && key == thr;
      cg += g[q] ? 1u : 0u;
      ce += e[q] ? 1u : 0u;
    }
    const uint32_t mine = cg | (ce << 16);
    uint32_t tot;
    const uint32_t ex = row_scan(mine, s_w, tot) - mine;
    uint32_t gb = run_g + (ex & 0xFFFFu), eb = run_e + (ex >> 16);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (g[q] || (e[q] && eb < need)) {
        const uint32_t pos = gb + (eb < need ? eb : need);
        if (pos < d.k) {
          oi[pos] = (uint32_t)(v + q - row.shift) + d.base;
          ov[pos] = x[q];
        }
        e_kept = __builtin_fma((double)x[q], (double)x[q], e_kept);
      }
      gb += g[q] ? 1u : 0u;
      eb += e[q] ? 1u : 0u;
    }
    run_g += tot & 0xFFFFu;
    run_e += tot >> 16;
  }
  const double ek = row_sum_f64(e_kept, s_d);
  if (tid == 0) rc.row_e[2ull * d.eslot + 1] = ek;
}

// Per device: the energies of its short layers summed in layer order.
__global__ __launch_bounds__(64) void k_rows_energy(RowsCtx rc, double* energies)
{
  if (threadIdx.x != 0) return;
  const uint32_t j = blockIdx.x;
  double ea = 0.0, ek = 0.0;
  for (uint32_t l = 0; l < rc.L; ++l) {
    if (rc.table[rc.L + 1 + l] == kNotShort) continue;
    ea += rc.row_e[2ull * ((uint64_t)j * rc.L + l)];
    ek += rc.row_e[2ull * ((uint64_t)j * rc.L + l) + 1];
  }
  energies[2 * j] = ea;
  energies[2 * j + 1] = ek;
}

}  // namespace

hipError_t launch_put_table(const uint64_t* src, uint64_t count, uint64_t* dst, hipStream_t s)
{
  for (uint64_t at = 0; at < count; at += kPutWords) {
    PutArgs a;
    a.count = (uint32_t)(count - at < (uint64_t)kPutWords ? count - at : (uint64_t)kPutWords);
    for (uint32_t i = 0; i < a.count; ++i) a.v[i] = src[at + i];
    a.dst = dst + at;
    k_put<<<1, 256, 0, s>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_rows(const RowsCtx& rc, const RowsPrep& rp, double* energies, hipStream_t s)
{
  k_rows_prep<<<rc.K, 256, 0, s>>>(rc, rp);
  if (rc.Ls > 0) {
    k_rows<<<rc.Ls * rc.K, kRowBlock, 0, s>>>(rc);
    if (energies) k_rows_energy<<<rc.K, 64, 0, s>>>(rc, energies);
  }
  return hipGetLastError();
}

}  // namespace scadles
