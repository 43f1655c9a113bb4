// rows.hip -- per-layer Top-k of short layers (the per-layer reading of the
// Top-k of §IV, ScaDLES arXiv 2301.08897): every (device, layer) row whose
// layer has at most a few million elements is selected by one workgroup, all
// such rows of all devices in one launch, instead of one multi-launch
// selection per layer.
//
// Per row (31-bit magnitude keys, ties to the lower index): a systematic
// sample brackets the k-th largest key; one read counts the keys above the
// bracket, gathers the keys inside it into LDS and tallies every wave's chunk;
// the exact key is selected among the gathered keys digit by digit (12 + 10 +
// 9 bits) in LDS; a last read writes the kept entries in index order -- keys
// above the threshold, and keys equal to it while fewer than `need` came
// before -- each wave at the positions its chunk tallies give. When the
// bracket misses or overflows LDS, the digits are decided over the whole row
// (a histogram read per digit until the remaining keys fit in LDS) and the
// output positions come from a workgroup scan per round.
#include "frame.h"

namespace scadles {

namespace {

constexpr int kRowWaves = kRowBlock / 64;
constexpr int kRowLevels = 3;
// digit `level` of a key: bits [shift, shift + width)
__device__ inline uint32_t level_shift(int level) { return level == 0 ? 19u : (level == 1 ? 9u : 0u); }
__device__ inline uint32_t level_width(int level) { return level == 0 ? 12u : (level == 1 ? 10u : 9u); }
constexpr uint32_t kRowBins = 1u << 12;
constexpr int kRowSampleBits = 13;           // digit of the sample histogram
constexpr uint32_t kRowSampleStride = 4096;  // one 256-element sample chunk per this many elements
constexpr uint32_t kRowWholeMax = 65536;     // rows up to this long are their own sample
// The full reads take kRowR rounds of 256 contiguous elements per wave at once
// (every lane loads its 4 elements of each round before any is used): wave w
// of a workgroup round covers [w, w + 1) * 256 * kRowR of it.
constexpr int kRowR = 8;
constexpr uint64_t kRowRound = (uint64_t)kRowBlock * 4 * kRowR;
// Per-wave chunks of a row whose tallies fit in LDS (rows up to 2^21 + 32768 elements)
constexpr uint32_t kRowChunks = 65 * kRowWaves;
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

// First virtual position of lane l's 4 elements in round r of wave w.
__device__ inline uint64_t row_pos(uint64_t v0, uint32_t w, int r, uint32_t l)
{
  return v0 + (uint64_t)w * (256u * kRowR) + (uint64_t)r * 256u + 4u * l;
}

// One round of the ordered output in a wave: its kept entries (keys above the
// threshold, and keys equal to it while fewer than `need` came before) at
// their positions; run_g / run_e count the wave's keys above / equal so far.
__device__ inline void row_write_round(const f4& x, uint64_t v, uint64_t vend, const Row& row, uint32_t base,
                                       uint32_t thr, uint32_t need, uint32_t k, GLOBAL uint32_t* oi,
                                       GLOBAL float* ov, uint32_t& run_g, uint32_t& run_e, double& e2)
{
  bool fg[4], fe[4];
  uint64_t bg[4], be[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool valid = v < vend && in_row(row, v + q);
    const uint32_t key = key_of(x[q]);
    fg[q] = valid && key > thr;
    fe[q] = valid && key == thr;
    bg[q] = ballot(fg[q]);
    be[q] = ballot(fe[q]);
  }
  if ((bg[0] | bg[1] | bg[2] | bg[3] | be[0] | be[1] | be[2] | be[3]) == 0ull) return;
  uint32_t gt_b = run_g + mbcnt(bg[0]) + mbcnt(bg[1]) + mbcnt(bg[2]) + mbcnt(bg[3]);
  uint32_t eq_b = run_e + mbcnt(be[0]) + mbcnt(be[1]) + mbcnt(be[2]) + mbcnt(be[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (fg[q] || (fe[q] && eq_b < need)) {
      const uint32_t pos = gt_b + (eq_b < need ? eq_b : need);
      if (pos < k) {
        oi[pos] = (uint32_t)(v + q - row.shift) + base;
        ov[pos] = x[q];
      }
      e2 = __builtin_fma((double)x[q], (double)x[q], e2);
    }
    gt_b += fg[q] ? 1u : 0u;
    eq_b += fe[q] ? 1u : 0u;
  }
  run_g += (uint32_t)(__builtin_popcountll(bg[0]) + __builtin_popcountll(bg[1]) + __builtin_popcountll(bg[2]) +
                      __builtin_popcountll(bg[3]));
  run_e += (uint32_t)(__builtin_popcountll(be[0]) + __builtin_popcountll(be[1]) + __builtin_popcountll(be[2]) +
                      __builtin_popcountll(be[3]));
}

// Radix selection, digit by digit, of the rank-th largest key among the keys
// with prefix `prefix` of `pbits` bits, starting at digit level `level`, over
// the m keys in cand (LDS). Returns the key; `rank` ends as the number of keys
// equal to it that are kept (the rank within the equal keys).
__device__ inline uint32_t row_select_lds(const uint32_t* cand, uint32_t m, uint32_t& rank, uint32_t* hist,
                                          uint32_t* s_w, uint32_t* s_res)
{
  const uint32_t tid = threadIdx.x;
  uint32_t prefix = 0, pbits = 0;
  for (int level = 0; level < kRowLevels; ++level) {
    const uint32_t sh = level_shift(level), mask = (1u << level_width(level)) - 1u;
    const uint32_t pshift = 31u - pbits;
    for (uint32_t i = tid; i < kRowBins; i += kRowBlock) hist[i] = 0u;
    if (tid == 0) s_res[0] = s_res[1] = s_res[2] = 0u;
    __syncthreads();
    for (uint32_t i = tid; i < m; i += kRowBlock) {
      const uint32_t key = cand[i];
      if (pbits == 0 || (key >> pshift) == prefix) atomicAdd(&hist[(key >> sh) & mask], 1u);
    }
    __syncthreads();
    row_select_bin(hist, level_width(level), rank, s_w, s_res);
    rank -= s_res[1];
    prefix = (prefix << level_width(level)) | s_res[0];
    pbits += level_width(level);
    __syncthreads();
  }
  return prefix;
}

// The same over the whole row in global memory, for rows whose sampled
// bracket missed: a histogram read per digit until the keys sharing the
// decided digits fit in LDS, then the rest in LDS.
__device__ inline uint32_t row_select_global(const Row& row, uint64_t vend, uint32_t& rank, uint32_t* hist,
                                             uint32_t* cand, uint32_t* s_w, uint32_t* s_res)
{
  const uint32_t tid = threadIdx.x;
  constexpr uint64_t kStep = (uint64_t)kRowBlock * 4;
  uint32_t prefix = 0, pbits = 0, m = 0;
  bool in_lds = false;
  for (int level = 0; level < kRowLevels; ++level) {
    const uint32_t sh = level_shift(level), mask = (1u << level_width(level)) - 1u;
    const uint32_t pshift = 31u - pbits;
    for (uint32_t i = tid; i < kRowBins; i += kRowBlock) hist[i] = 0u;
    if (tid == 0) s_res[0] = s_res[1] = s_res[2] = 0u;
    __syncthreads();
    if (in_lds) {
      for (uint32_t i = tid; i < m; i += kRowBlock) {
        const uint32_t key = cand[i];
        if ((key >> pshift) == prefix) atomicAdd(&hist[(key >> sh) & mask], 1u);
      }
    } else {
      for (uint64_t v = (uint64_t)tid * 4; v < vend; v += kStep) {
        const f4 x = load4(row, v, false);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t key = key_of(x[q]);
          if (in_row(row, v + q) && (pbits == 0 || (key >> pshift) == prefix))
            atomicAdd(&hist[(key >> sh) & mask], 1u);
        }
      }
    }
    __syncthreads();
    row_select_bin(hist, level_width(level), rank, s_w, s_res);
    const uint32_t h = s_res[2];
    rank -= s_res[1];
    prefix = (prefix << level_width(level)) | s_res[0];
    pbits += level_width(level);
    __syncthreads();
    if (level + 1 < kRowLevels && !in_lds && h <= (uint32_t)kRowCand) {
      // the keys sharing the decided digits fit in LDS: collect them
      const uint32_t ps = 31u - pbits;
      if (tid == 0) s_res[3] = 0u;
      __syncthreads();
      for (uint64_t v = (uint64_t)tid * 4; v < vend; v += kStep) {
        const f4 x = load4(row, v, false);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t key = key_of(x[q]);
          if (in_row(row, v + q) && (key >> ps) == prefix) {
            const uint32_t at = atomicAdd(&s_res[3], 1u);
            if (at < (uint32_t)kRowCand) cand[at] = key;
          }
        }
      }
      __syncthreads();
      m = s_res[3] < (uint32_t)kRowCand ? s_res[3] : (uint32_t)kRowCand;
      in_lds = true;
      __syncthreads();
    }
  }
  return prefix;
}

// The bracket [t_lo, t_hi) of a row from a systematic sample (256-element
// chunks every kRowSampleStride elements; the whole row when it is short):
// the bins of its 13-bit histogram (in shist, kRowCand words of LDS) around
// k's expected sample rank, six standard deviations and 8 ranks either side.
__device__ inline void row_bracket(const RowDesc& d, const Row& row, uint64_t vend, uint32_t* shist, uint32_t* s_w,
                                   uint32_t* s_res, uint32_t& t_lo, uint32_t& t_hi)
{
  static_assert((1 << kRowSampleBits) <= kRowCand, "the sample histogram fits the candidate array");
  const uint32_t tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const bool whole = d.n <= (uint32_t)kRowWholeMax;
  const uint64_t stride = whole ? 256u : (uint64_t)kRowSampleStride;
  for (uint32_t i = tid; i < (1u << kRowSampleBits); i += kRowBlock) shist[i] = 0u;
  __syncthreads();
  uint32_t s_cnt = 0;
  for (uint64_t c0 = w; c0 * stride < vend; c0 += 4 * kRowWaves) {
    f4 x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint64_t v = (c0 + r * kRowWaves) * stride + 4u * lane;
      x[r] = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint64_t v = (c0 + r * kRowWaves) * stride + 4u * lane;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (v < vend && in_row(row, v + q)) {
          atomicAdd(&shist[key_of(x[r][q]) >> (31 - kRowSampleBits)], 1u);
          ++s_cnt;
        }
      }
    }
  }
  uint32_t s_n;
  row_scan(s_cnt, s_w, s_n);
  // sample ranks bracketing the k-th largest key
  uint32_t r_lo, r_hi;
  if (whole) {
    r_lo = r_hi = d.k;
  } else {
    const double kf = (double)d.k * (double)s_n / (double)d.n, sd = __builtin_sqrt(kf);
    double lo = __builtin_ceil(kf + 6.0 * sd + 8.0), hi = __builtin_floor(kf - 6.0 * sd - 8.0);
    lo = lo > (double)s_n ? (double)s_n : (lo < 1.0 ? 1.0 : lo);
    r_lo = (uint32_t)lo;
    r_hi = hi < 1.0 ? 0u : (uint32_t)hi;
  }
  if (tid == 0) s_res[0] = s_res[1] = s_res[2] = 0u;
  row_select_bin(shist, kRowSampleBits, r_lo, s_w, s_res);
  t_lo = s_res[0] << (31 - kRowSampleBits);
  __syncthreads();
  t_hi = kKeyInf;
  if (r_hi >= 1) {
    if (tid == 0) s_res[0] = s_res[1] = s_res[2] = 0u;
    row_select_bin(shist, kRowSampleBits, r_hi, s_w, s_res);
    t_hi = (s_res[0] + 1u) << (31 - kRowSampleBits);
    __syncthreads();
  }
}

// Ordered output of a whole row by one workgroup, without chunk tallies: per
// workgroup round the waves' counts give each wave's starting position. Returns
// this thread's share of the kept sum of squares.
__device__ inline double row_write_ordered(const RowDesc& d, const Row& row, uint64_t vend, uint32_t thr,
                                           uint32_t need, GLOBAL uint32_t* oi, GLOBAL float* ov, uint32_t* s_w)
{
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  double e_kept = 0.0;
  uint32_t run_g = 0, run_e = 0;
#pragma unroll 1
  for (uint64_t v0 = 0; v0 < vend; v0 += kRowRound) {
    f4 x[kRowR];
#pragma unroll
    for (int r = 0; r < kRowR; ++r) {
      const uint64_t v = row_pos(v0, w, r, lane);
      x[r] = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
    }
    uint32_t cnt = 0;
#pragma unroll
    for (int r = 0; r < kRowR; ++r) {
      const uint64_t v = row_pos(v0, w, r, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool valid = v < vend && in_row(row, v + q);
        const uint32_t key = key_of(x[r][q]);
        cnt += (valid && key > thr) ? 1u : 0u;
        cnt += (valid && key == thr) ? 0x10000u : 0u;
      }
    }
    uint32_t wt = cnt;
#pragma unroll
    for (int dd = 32; dd >= 1; dd >>= 1) wt += __shfl_xor(wt, dd, 64);
    if (lane == 0) s_w[w] = wt;
    __syncthreads();
    uint32_t wex = 0, tot = 0;
    for (uint32_t i = 0; i < (uint32_t)kRowWaves; ++i) {
      const uint32_t y = s_w[i];
      wex += i < w ? y : 0u;
      tot += y;
    }
    __syncthreads();
    uint32_t rg = run_g + (wex & 0xFFFFu), re = run_e + (wex >> 16);
#pragma unroll
    for (int r = 0; r < kRowR; ++r)
      row_write_round(x[r], row_pos(v0, w, r, lane), vend, row, d.base, thr, need, d.k, oi, ov, rg, re, e_kept);
    run_g += tot & 0xFFFFu;
    run_e += tot >> 16;
  }
  return e_kept;
}

// The selection of one row. A systematic sample (256-element chunks every
// kRowSampleStride elements; the whole row when it is short) gives a bracket
// [t_lo, t_hi) that holds the k-th largest key with high probability: the
// bins of its 13-bit histogram around k's expected sample rank, six standard
// deviations and 8 ranks either side. One read of the row then counts the keys
// at or above t_hi, gathers the keys inside the bracket into LDS and sums g^2;
// the k-th largest key is selected among the gathered ones. If the bracket
// missed or overflowed LDS, the digits are decided over the whole row instead.
// A last read writes the kept entries in index order.
__global__ __launch_bounds__(kRowBlock) void k_rows(RowsCtx rc)
{
  __shared__ uint32_t hist[kRowBins];
  __shared__ uint32_t cand[kRowCand];
  __shared__ uint32_t s_w[kRowWaves];
  __shared__ uint32_t s_res[4];
  __shared__ double s_d[kRowWaves];
  __shared__ uint32_t s_chunk[2 * kRowChunks];
  const RowDesc d = rc.rows[rc.Lb * rc.K + blockIdx.x];
  const uint32_t tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const Row row{gptr(d.grad), ((uint64_t)d.grad >> 2) & 3u, d.n};
  const uint64_t vend = (uint64_t)d.n + row.shift;

  // 1. bracket from the sample
  uint32_t t_lo, t_hi;
  row_bracket(d, row, vend, cand, s_w, s_res, t_lo, t_hi);

  // 2. one read: keys >= t_hi counted, keys in [t_lo, t_hi) gathered, sum g^2
  if (tid == 0) s_res[3] = 0u;
  __syncthreads();
  double e_all = 0.0;
  uint32_t sure = 0;
  const uint64_t nchunk = (vend + kRowRound - 1) / kRowRound * kRowWaves;
  const bool tally = nchunk <= (uint64_t)kRowChunks;
  for (uint64_t v0 = 0; v0 < vend; v0 += kRowRound) {
    f4 x[kRowR];
#pragma unroll
    for (int r = 0; r < kRowR; ++r) {
      const uint64_t v = row_pos(v0, w, r, lane);
      x[r] = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
    }
    // count this lane's keys in the bracket, then one wave-wide slot
    // reservation for all of them (one LDS atomic per wave and round)
    uint32_t nb = 0, sure_w = 0;
#pragma unroll
    for (int r = 0; r < kRowR; ++r) {
      const uint64_t v = row_pos(v0, w, r, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool valid = v < vend && in_row(row, v + q);
        const uint32_t key = key_of(x[r][q]);
        const bool above = valid && key >= t_hi;
        sure += above ? 1u : 0u;
        sure_w += (uint32_t)__builtin_popcountll(ballot(above));
        nb += (valid && key >= t_lo && key < t_hi) ? 1u : 0u;
        if (valid) e_all = __builtin_fma((double)x[r][q], (double)x[r][q], e_all);
      }
    }
    // this wave's chunk of the round: keys at or above t_hi, and where its
    // bracket keys start in cand and how many there are
    const uint64_t chunk = v0 / kRowRound * kRowWaves + w;
    if (!ballot(nb != 0u)) {
      if (tally && lane == 0) {
        s_chunk[2 * chunk] = sure_w;
        s_chunk[2 * chunk + 1] = 0u;
      }
    } else {
      const uint32_t incl = wave_incl_scan(nb);
      const uint32_t total = __shfl(incl, 63, 64);
      uint32_t at = 0;
      if (lane == 0) {
        at = atomicAdd(&s_res[3], total);
        if (tally) {
          s_chunk[2 * chunk] = sure_w | (total << 16);
          s_chunk[2 * chunk + 1] = at;
        }
      }
      at = __shfl(at, 0, 64) + incl - nb;
#pragma unroll
      for (int r = 0; r < kRowR; ++r) {
        const uint64_t v = row_pos(v0, w, r, lane);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const bool valid = v < vend && in_row(row, v + q);
          const uint32_t key = key_of(x[r][q]);
          if (valid && key >= t_lo && key < t_hi) {
            if (at < (uint32_t)kRowCand) cand[at] = key;
            ++at;
          }
        }
      }
    }
  }
  uint32_t sure_all;
  row_scan(sure, s_w, sure_all);
  const uint32_t nband = s_res[3];
  {
    const double ea = row_sum_f64(e_all, s_d);
    if (tid == 0) rc.row_e[2ull * d.eslot] = ea;
  }

  // 3. the threshold key and the number of keys equal to it that are kept
  uint32_t thr, need;
  const bool in_band = sure_all < d.k && d.k - sure_all <= nband && nband <= (uint32_t)kRowCand;
  if (in_band) {
    need = d.k - sure_all;
    thr = row_select_lds(cand, nband, need, hist, s_w, s_res);
  } else {
    need = d.k;
    thr = row_select_global(row, vend, need, hist, cand, s_w, s_res);
  }

  // 4. ordered output
  double e_kept = 0.0;
  GLOBAL uint32_t* oi = gptr(d.idx_out);
  GLOBAL float* ov = gptr(d.val_out);
  if (tally && in_band) {
    // every chunk's keys above / equal to the threshold from its tallies and
    // bracket keys, their exclusive prefix in index order, then each wave
    // writes its chunks on its own
    const uint32_t per = (uint32_t)((nchunk + kRowBlock - 1) / kRowBlock);
    const uint32_t c0 = tid * per, c1 = c0 + per < (uint32_t)nchunk ? c0 + per : (uint32_t)nchunk;
    uint32_t gsum = 0, esum = 0;
    for (uint32_t c = c0; c < c1; ++c) {
      const uint32_t tl = s_chunk[2 * c], st = s_chunk[2 * c + 1], nbc = tl >> 16;
      uint32_t g = tl & 0xFFFFu, e = 0;
      for (uint32_t i = 0; i < nbc; ++i) {
        const uint32_t key = cand[st + i];
        g += key > thr ? 1u : 0u;
        e += key == thr ? 1u : 0u;
      }
      s_chunk[2 * c] = g;
      s_chunk[2 * c + 1] = e;
      gsum += g;
      esum += e;
    }
    uint32_t tg, te;
    const uint32_t gex = row_scan(gsum, s_w, tg) - gsum;
    const uint32_t eex = row_scan(esum, s_w, te) - esum;
    {
      uint32_t rg = gex, re = eex;
      for (uint32_t c = c0; c < c1; ++c) {
        const uint32_t g = s_chunk[2 * c], e = s_chunk[2 * c + 1];
        s_chunk[2 * c] = rg;
        s_chunk[2 * c + 1] = re;
        rg += g;
        re += e;
      }
    }
    __syncthreads();
#pragma unroll 1
    for (uint64_t v0 = 0; v0 < vend; v0 += kRowRound) {
      const uint64_t chunk = v0 / kRowRound * kRowWaves + w;
      f4 x[kRowR];
#pragma unroll
      for (int r = 0; r < kRowR; ++r) {
        const uint64_t v = row_pos(v0, w, r, lane);
        x[r] = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
      }
      uint32_t rg = s_chunk[2 * chunk], re = s_chunk[2 * chunk + 1];
#pragma unroll
      for (int r = 0; r < kRowR; ++r)
        row_write_round(x[r], row_pos(v0, w, r, lane), vend, row, d.base, thr, need, d.k, oi, ov, rg, re, e_kept);
    }
  } else {
    e_kept = row_write_ordered(d, row, vend, thr, need, oi, ov, s_w);
  }
  const double ek = row_sum_f64(e_kept, s_d);
  if (tid == 0) rc.row_e[2ull * d.eslot + 1] = ek;
}

// ---- split rows --------------------------------------------------------------------------
// A row longer than the split threshold is read by one workgroup per part:
//   k_big_bracket  one workgroup per row: the sampled bracket [t_lo, t_hi)
//                  (as k_rows computes it);
//   k_big_gather   one workgroup per part, the one read of the row: sum of
//                  g^2 and, per chunk, the keys >= t_hi counted and the
//                  candidates (keys >= t_lo) staged in index order in the
//                  wave's own region of the row's candidate list;
//   k_big_select   one workgroup per row: the selection-interval keys (the
//                  candidates below t_hi) collected in LDS, the threshold
//                  selected among them, then every chunk's kept entries above /
//                  equal to it (counted on its candidates) and their exclusive
//                  prefix in index order. A row whose bracket missed, or whose
//                  candidates overflowed a wave's region, is selected and
//                  written here, by this workgroup alone, as k_rows does it;
//   k_big_write    one workgroup per part: every chunk's kept entries, from its
//                  candidates, at the positions from its prefix;
//   k_big_finish   the kept energy of each row from its waves' sums, in order.
// No workgroup waits for another inside a launch, and the part kernels have
// no barrier and no atomic but the rare overflow flag.
constexpr int kPartWaves = (int)kRowPartWaves;
// selection-interval keys a split row's select workgroup holds in LDS (one
// workgroup per row: it can take most of a compute unit's 160 KiB)
constexpr int kBigCand = 32768;
static_assert(kBigCand >= kRowCand, "the whole-row path of the select kernel uses kRowCand keys of the array");
constexpr int kPartBlock = 64 * kPartWaves;
constexpr int kWaveChunks = kRowPartChunks / kPartWaves;    // chunks of one wave, loaded at once
static_assert(kRowChunkLen == 256u * kRowR, "a chunk is one wave's kRowR rounds");
static_assert(kWaveChunks * kPartWaves == (int)kRowPartChunks, "a part's chunks are split evenly over its waves");

// Part workgroup g: its row (index into rc.rows), part, the row's first part
// workgroup and number of parts.
struct PartOf {
  uint32_t b, p, g0, np;
};

__device__ inline PartOf part_of(const RowsCtx& rc, uint32_t g)
{
  const uint64_t* pre = rc.table + 2ull * rc.L + 1;
  uint32_t lo = 0, hi = rc.Lb;     // pre[lo] * K <= g < pre[hi] * K
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (pre[mid] * rc.K <= g) lo = mid;
    else hi = mid;
  }
  const uint32_t np = (uint32_t)(pre[lo + 1] - pre[lo]);
  const uint32_t rel = g - (uint32_t)(pre[lo] * rc.K);
  const uint32_t j = rel / np;
  PartOf r;
  r.b = lo * rc.K + j;
  r.p = rel - j * np;
  r.g0 = g - r.p;
  r.np = np;
  return r;
}

// Split row b's first part workgroup and number of parts.
__device__ inline void row_parts(const RowsCtx& rc, uint32_t b, uint32_t& g0, uint32_t& np)
{
  const uint64_t* pre = rc.table + 2ull * rc.L + 1;
  const uint32_t q = b / rc.K, j = b - q * rc.K;
  np = (uint32_t)(pre[q + 1] - pre[q]);
  g0 = (uint32_t)(pre[q] * rc.K) + j * np;
}

// Split row b's candidate list: its first entry and the capacity of one wave's region.
__device__ inline void row_cands(const RowsCtx& rc, uint32_t b, uint64_t& off, uint32_t& wcap)
{
  const uint64_t* pre = rc.table + 2ull * rc.L + 1;             // part_pre, then cand_pre
  const uint64_t* cpre = pre + rc.Lb + 1;
  const uint32_t q = b / rc.K, j = b - q * rc.K;
  const uint64_t per_row = cpre[q + 1] - cpre[q];
  off = cpre[q] * rc.K + (uint64_t)j * per_row;
  wcap = (uint32_t)(per_row / ((pre[q + 1] - pre[q]) * kPartWaves));
}

// Fixed-order sum of n doubles by one wave (lane l adds l, l + 64, ...).
__device__ inline double wave_sum_list(const double* a, uint32_t n)
{
  double v = 0.0;
  for (uint32_t i = lane_id(); i < n; i += 64) v += a[i];
  return wave_sum_f64(v);
}

__global__ __launch_bounds__(kRowBlock) void k_big_bracket(RowsCtx rc)
{
  __shared__ uint32_t shist[1 << kRowSampleBits];
  __shared__ uint32_t s_w[kRowWaves];
  __shared__ uint32_t s_res[4];
  const RowDesc d = rc.rows[blockIdx.x];
  const Row row{gptr(d.grad), ((uint64_t)d.grad >> 2) & 3u, d.n};
  uint32_t t_lo, t_hi;
  row_bracket(d, row, (uint64_t)d.n + row.shift, shist, s_w, s_res, t_lo, t_hi);
  if (threadIdx.x == 0) {
    BigRowState st;
    __builtin_memset(&st, 0, sizeof(st));
    st.t_lo = t_lo;
    st.t_hi = t_hi;
    rc.bst[blockIdx.x] = st;
  }
}

// Gather-pass counts of one chunk in one wave (x holds its kRowR rounds: lane
// l has elements v0 + r * 256 + 4 l .. + 3 of round r): keys >= t_hi and
// candidates (keys >= t_lo); e_all accumulates g^2. kFull: every element is in
// the row.
template <bool kFull>
__device__ inline void gather_count(const f4 (&x)[kRowR], uint64_t v0, uint64_t vend, const Row& row, uint32_t t_lo,
                                    uint32_t t_hi, uint32_t& nsure, uint32_t& ncand, uint32_t& nband, double& e_all)
{
  nsure = ncand = nband = 0;
#pragma unroll
  for (int r = 0; r < kRowR; ++r) {
    const uint64_t v = v0 + r * 256u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool valid = kFull || (v < vend && in_row(row, v + q));
      const uint32_t key = key_of(x[r][q]);
      nsure += (uint32_t)__builtin_popcountll(ballot(valid && key >= t_hi));
      ncand += (uint32_t)__builtin_popcountll(ballot(valid && key >= t_lo));
      nband += (uint32_t)__builtin_popcountll(ballot(valid && key >= t_lo && key < t_hi));
      if (kFull) e_all = __builtin_fma((double)x[r][q], (double)x[r][q], e_all);
      else if (valid) e_all = __builtin_fma((double)x[r][q], (double)x[r][q], e_all);
    }
  }
}

// Stages one chunk's candidates at cand[at ..] (index order: round, lane,
// component), at most up to position cap.
template <bool kFull>
__device__ inline void gather_write(const f4 (&x)[kRowR], uint64_t v0, uint64_t vend, const Row& row, uint32_t t_lo,
                                    uint32_t at, GLOBAL uint64_t* cand, uint32_t cap)
{
#pragma unroll
  for (int r = 0; r < kRowR; ++r) {
    const uint64_t v = v0 + r * 256u;
    bool f[4];
    uint64_t bc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool valid = kFull || (v < vend && in_row(row, v + q));
      f[q] = valid && key_of(x[r][q]) >= t_lo;
      bc[q] = ballot(f[q]);
    }
    if ((bc[0] | bc[1] | bc[2] | bc[3]) == 0ull) continue;
    uint32_t cp = at + mbcnt(bc[0]) + mbcnt(bc[1]) + mbcnt(bc[2]) + mbcnt(bc[3]);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (f[q]) {
        if (cp < cap) cand[cp] = (uint64_t)(uint32_t)(v + q - row.shift) | ((uint64_t)__float_as_uint(x[r][q]) << 32);
        ++cp;
      }
    }
    at += (uint32_t)(__builtin_popcountll(bc[0]) + __builtin_popcountll(bc[1]) + __builtin_popcountll(bc[2]) +
                     __builtin_popcountll(bc[3]));
  }
}

// Each wave loads its kWaveChunks consecutive chunks at once, counts them and
// stages their candidates in its region.
__global__ __launch_bounds__(kPartBlock) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_big_gather(RowsCtx rc)
{
  const PartOf po = part_of(rc, blockIdx.x);
  const RowDesc d = rc.rows[po.b];
  GLOBAL BigRowState* st = gptr(rc.bst) + po.b;
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  const Row row{gptr(d.grad), ((uint64_t)d.grad >> 2) & 3u, d.n};
  const uint64_t vend = (uint64_t)d.n + row.shift;
  const uint32_t c0 = w * kWaveChunks;
  const uint64_t vw = (uint64_t)po.p * kRowPartLen + (uint64_t)c0 * kRowChunkLen;   // the wave's first element
  const bool full = vw >= row.shift && vw + (uint64_t)kWaveChunks * kRowChunkLen <= vend;
  const uint64_t v0 = vw + 4u * lane;
  f4 x[kWaveChunks][kRowR];
  if (full) {
    const GLOBAL float* p = row.p + (vw - row.shift) + 4u * lane;
#pragma unroll
    for (int c = 0; c < kWaveChunks; ++c)
#pragma unroll
      for (int r = 0; r < kRowR; ++r) x[c][r] = ld_stream4(p + c * kRowChunkLen + r * 256u);
  } else {
#pragma unroll
    for (int c = 0; c < kWaveChunks; ++c)
#pragma unroll
      for (int r = 0; r < kRowR; ++r) {
        const uint64_t v = v0 + (uint64_t)c * kRowChunkLen + r * 256u;
        x[c][r] = v < vend ? load4(row, v, false) : f4{0.f, 0.f, 0.f, 0.f};
      }
  }
  const uint32_t t_lo = st->t_lo, t_hi = st->t_hi;
  uint64_t coff;
  uint32_t wcap;
  row_cands(rc, po.b, coff, wcap);
  const uint32_t wbase = (po.p * kPartWaves + w) * wcap;       // the wave's region in the row's list
  GLOBAL uint64_t* cand = gptr(rc.cand) + coff + wbase;
  GLOBAL uint32_t* rec = gptr(rc.chunk) + ((uint64_t)blockIdx.x * kRowPartChunks + c0) * kChunkWords;
  double e_all = 0.0;
  uint32_t at = 0;
#pragma unroll
  for (int c = 0; c < kWaveChunks; ++c) {
    const uint64_t vc = v0 + (uint64_t)c * kRowChunkLen;
    uint32_t nsure, ncand, nband;
    if (full) gather_count<true>(x[c], vc, vend, row, t_lo, t_hi, nsure, ncand, nband, e_all);
    else gather_count<false>(x[c], vc, vend, row, t_lo, t_hi, nsure, ncand, nband, e_all);
    if (ncand) {
      if (full) gather_write<true>(x[c], vc, vend, row, t_lo, at, cand, wcap);
      else gather_write<false>(x[c], vc, vend, row, t_lo, at, cand, wcap);
    }
    if (lane == 0) {
      const u4 w4 = {nsure, nband, wbase + at, ncand};
      *reinterpret_cast<GLOBAL u4*>(rec + c * kChunkWords) = w4;
    }
    at += ncand;
  }
  if (at > wcap && lane == 0) __hip_atomic_fetch_or(&st->ovf, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const double e = wave_sum_f64(e_all);
  if (lane == 0) rc.part_e[(uint64_t)blockIdx.x * kPartWaves + w] = e;
}

__global__ __launch_bounds__(kRowBlock) void k_big_select(RowsCtx rc)
{
  __shared__ uint32_t hist[kRowBins];
  __shared__ uint32_t cand[kBigCand];
  __shared__ uint32_t s_w[kRowWaves];
  __shared__ uint32_t s_res[4];
  __shared__ double s_d[kRowWaves];
  const uint32_t b = blockIdx.x, tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const RowDesc d = rc.rows[b];
  GLOBAL BigRowState* st = gptr(rc.bst) + b;
  uint32_t g0, np;
  row_parts(rc, b, g0, np);
  uint64_t coff;
  uint32_t wcap;
  row_cands(rc, b, coff, wcap);
  const GLOBAL uint64_t* list = gptr(rc.cand) + coff;
  const uint32_t nch = np * kRowPartChunks;
  GLOBAL uint32_t* ch = gptr(rc.chunk) + (uint64_t)g0 * kRowPartChunks * kChunkWords;
  const Row row{gptr(d.grad), ((uint64_t)d.grad >> 2) & 3u, d.n};
  const uint64_t vend = (uint64_t)d.n + row.shift;
  const uint32_t t_hi = st->t_hi;
  if (w == 0) {
    const double ea = wave_sum_list(rc.part_e + (uint64_t)g0 * kPartWaves, np * kPartWaves);
    if (lane == 0) rc.row_e[2ull * d.eslot] = ea;
  }
  // each thread a run of consecutive chunks (one chunk per thread for rows up
  // to kRowBlock chunks); their records stay in registers for the first run
  const uint32_t per = (nch + kRowBlock - 1) / kRowBlock;
  const uint32_t c0 = tid * per < nch ? tid * per : nch, c1 = c0 + per < nch ? c0 + per : nch;
  uint32_t sure = 0, band = 0;
  for (uint32_t c = c0; c < c1; ++c) {
    sure += ch[kChunkWords * c];
    band += ch[kChunkWords * c + 1];
  }
  uint32_t sure_all, nband;
  row_scan(sure, s_w, sure_all);
  const uint32_t boff = row_scan(band, s_w, nband) - band;   // the thread's chunks' keys start here in LDS
  const bool in_band = st->ovf == 0u && sure_all < d.k && d.k - sure_all <= nband && nband <= (uint32_t)kBigCand;
  if (in_band) {
    // the selection-interval keys (the candidates below t_hi) into LDS, each
    // thread's chunks in order from boff: the only read of the candidates
    uint32_t pos = boff;
    for (uint32_t c = c0; c < c1; ++c) {
      const uint32_t at = ch[kChunkWords * c + 2], n = ch[kChunkWords * c + 3];
      for (uint32_t e0 = 0; e0 < n; e0 += 8) {
        uint32_t kv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) kv[i] = e0 + i < n ? (uint32_t)(list[at + e0 + i] >> 32) & kKeyMask : kKeyInf;
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (kv[i] < t_hi) {
            if (pos < (uint32_t)kBigCand) cand[pos] = kv[i];
            ++pos;
          }
      }
    }
    __syncthreads();
    uint32_t need = d.k - sure_all;
    const uint32_t thr = row_select_lds(cand, nband, need, hist, s_w, s_res);
    // every chunk's kept entries above / equal to the threshold (its keys >=
    // t_hi and its band keys in LDS), then their exclusive prefix in index order
    uint32_t gsum = 0, esum = 0;
    pos = boff;
    for (uint32_t c = c0; c < c1; ++c) {
      const uint32_t nb = ch[kChunkWords * c + 1];
      uint32_t g = ch[kChunkWords * c], e = 0;
      for (uint32_t i = 0; i < nb; ++i) {
        const uint32_t key = cand[pos + i];
        g += key > thr ? 1u : 0u;
        e += key == thr ? 1u : 0u;
      }
      pos += nb;
      ch[kChunkWords * c] = g;
      ch[kChunkWords * c + 1] = e;
      gsum += g;
      esum += e;
    }
    uint32_t tg, te;
    uint32_t rg = row_scan(gsum, s_w, tg) - gsum;
    uint32_t re = row_scan(esum, s_w, te) - esum;
    for (uint32_t c = c0; c < c1; ++c) {
      const uint32_t g = ch[kChunkWords * c], e = ch[kChunkWords * c + 1];
      ch[kChunkWords * c] = rg;
      ch[kChunkWords * c + 1] = re;
      rg += g;
      re += e;
    }
    if (tid == 0) {
      st->thr = thr;
      st->need = need;
      st->slow = 0u;
    }
  } else {
    // the bracket missed or a wave's candidates overflowed: this workgroup
    // selects and writes the row on its own
    uint32_t need = d.k;
    const uint32_t thr = row_select_global(row, vend, need, hist, cand, s_w, s_res);
    const double ek =
        row_sum_f64(row_write_ordered(d, row, vend, thr, need, gptr(d.idx_out), gptr(d.val_out), s_w), s_d);
    if (tid == 0) {
      rc.row_e[2ull * d.eslot + 1] = ek;
      st->slow = 1u;
    }
  }
}

// Kept entries of one chunk from its staged candidates (index order): n of
// them at cand, run_g / run_e the kept entries above / equal to the threshold
// before the chunk.
__device__ inline void write_staged(const GLOBAL uint64_t* cand, uint32_t n, uint32_t base, uint32_t thr,
                                    uint32_t need, uint32_t k, GLOBAL uint32_t* oi, GLOBAL float* ov, uint32_t run_g,
                                    uint32_t run_e, double& e2)
{
  const uint32_t lane = lane_id();
  for (uint32_t e0 = 0; e0 < n; e0 += 4 * 64) {
    uint64_t w4[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint32_t e = e0 + m * 64 + lane;
      w4[m] = e < n ? cand[e] : 0ull;
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (e0 + m * 64 >= n) break;
      const bool valid = e0 + m * 64 + lane < n;
      const uint32_t vb = (uint32_t)(w4[m] >> 32), key = vb & kKeyMask;
      const bool fg = valid && key > thr, fe = valid && key == thr;
      const uint64_t bg = ballot(fg), be = ballot(fe);
      const uint32_t gt_b = run_g + mbcnt(bg), eq_b = run_e + mbcnt(be);
      if (fg || (fe && eq_b < need)) {
        const uint32_t pos = gt_b + (eq_b < need ? eq_b : need);
        const float v = __uint_as_float(vb);
        if (pos < k) {
          oi[pos] = (uint32_t)w4[m] + base;
          ov[pos] = v;
        }
        e2 = __builtin_fma((double)v, (double)v, e2);
      }
      run_g += (uint32_t)__builtin_popcountll(bg);
      run_e += (uint32_t)__builtin_popcountll(be);
    }
  }
}

__global__ __launch_bounds__(kPartBlock) void k_big_write(RowsCtx rc)
{
  const PartOf po = part_of(rc, blockIdx.x);
  const GLOBAL BigRowState* st = gptr(rc.bst) + po.b;
  const uint32_t lane = lane_id(), w = threadIdx.x >> 6;
  double e_kept = 0.0;
  if (!st->slow) {
    const RowDesc d = rc.rows[po.b];
    const uint32_t thr = st->thr, need = st->need;
    uint64_t coff;
    uint32_t wcap;
    row_cands(rc, po.b, coff, wcap);
    const GLOBAL uint64_t* list = gptr(rc.cand) + coff;
    const GLOBAL uint32_t* rec = gptr(rc.chunk) + (uint64_t)blockIdx.x * kRowPartChunks * kChunkWords;
    GLOBAL uint32_t* oi = gptr(d.idx_out);
    GLOBAL float* ov = gptr(d.val_out);
#pragma unroll
    for (int c = 0; c < kWaveChunks; ++c) {
      const u4 r4 = *reinterpret_cast<const GLOBAL u4*>(rec + (w * kWaveChunks + c) * kChunkWords);
      if (r4[3]) write_staged(list + r4[2], r4[3], d.base, thr, need, d.k, oi, ov, r4[0], r4[1], e_kept);
    }
  }
  const double e = wave_sum_f64(e_kept);
  if (lane == 0) rc.part_e[((uint64_t)rc.nparts + blockIdx.x) * kPartWaves + w] = e;
}

__global__ __launch_bounds__(64) void k_big_finish(RowsCtx rc)
{
  const uint32_t b = blockIdx.x;
  if (rc.bst[b].slow) return;
  uint32_t g0, np;
  row_parts(rc, b, g0, np);
  const double ek = wave_sum_list(rc.part_e + ((uint64_t)rc.nparts + g0) * kPartWaves, np * kPartWaves);
  if (threadIdx.x == 0) rc.row_e[2ull * rc.rows[b].eslot + 1] = ek;
}

// Per device: the energies of all its layers, short and long (each lane a
// strided subset in layer order, then the lanes in a fixed tree).
__global__ __launch_bounds__(64) void k_rows_energy(RowsCtx rc, double* energies)
{
  // lane i adds layers i, i + 64, ... in order, then the lanes in a fixed tree
  const uint32_t j = blockIdx.x;
  double ea = 0.0, ek = 0.0;
  for (uint32_t l = threadIdx.x; l < rc.L; l += 64) {
    ea += rc.row_e[2ull * ((uint64_t)j * rc.L + l)];
    ek += rc.row_e[2ull * ((uint64_t)j * rc.L + l) + 1];
  }
  ea = wave_sum_f64(ea);
  ek = wave_sum_f64(ek);
  if (threadIdx.x != 0) return;
  energies[2 * j] = ea;
  energies[2 * j + 1] = ek;
}

// The adaptive rule of §IV per device on its whole-gradient energies after a
// per-layer selection (and the moving average and accounting options).
__global__ __launch_bounds__(64) void k_layers_decide(DecideArgs a)
{
  const uint32_t j = blockIdx.x * 64 + threadIdx.x;
  if (j >= a.K) return;
  const double ea = a.e[2 * j], ek = a.e[2 * j + 1];
  const uint32_t sp = adaptive_rule(ea, ek, a.ewma ? a.ewma + 2 * (uint64_t)j : nullptr, a.beta, a.delta);
  a.st[j].sparse = sp;
  if (a.counters) account(a.counters + 3 * (uint64_t)j, sp, a.k[j], a.n);
  if (a.energies_out) {
    a.energies_out[2 * j] = ea;
    a.energies_out[2 * j + 1] = ek;
  }
  if (a.compressed_out) a.compressed_out[j] = (uint8_t)sp;
}

}  // namespace

hipError_t launch_layers_decide(const DecideArgs& a, hipStream_t s)
{
  k_layers_decide<<<(a.K + 63) / 64, 64, 0, s>>>(a);
  return hipGetLastError();
}

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
  if (rc.Lb > 0) {
    const uint32_t nb = rc.Lb * rc.K;
    k_big_bracket<<<nb, kRowBlock, 0, s>>>(rc);
    k_big_gather<<<rc.nparts, kPartBlock, 0, s>>>(rc);
    k_big_select<<<nb, kRowBlock, 0, s>>>(rc);
    k_big_write<<<rc.nparts, kPartBlock, 0, s>>>(rc);
    k_big_finish<<<nb, 64, 0, s>>>(rc);
  }
  if (rc.Ls > rc.Lb) k_rows<<<(rc.Ls - rc.Lb) * rc.K, kRowBlock, 0, s>>>(rc);
  if (rc.Ls > 0 && energies) k_rows_energy<<<rc.K, 64, 0, s>>>(rc, energies);
  return hipGetLastError();
}

// Clears n words (a fill kernel rather than a memset node, so that the call
// stays safe to capture in a graph).
__global__ __launch_bounds__(256) void k_zero_words(uint32_t* p, uint32_t n)
{
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

hipError_t launch_zero_words(uint32_t* p, uint32_t n, hipStream_t s)
{
  k_zero_words<<<1, 256, 0, s>>>(p, n);
  return hipGetLastError();
}

hipError_t launch_rows_energy(const RowsCtx& rc, double* energies, hipStream_t s)
{
  k_rows_energy<<<rc.K, 64, 0, s>>>(rc, energies);
  return hipGetLastError();
}

}  // namespace scadles
