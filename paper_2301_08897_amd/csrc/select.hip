// select.hip -- Top-k selection kernels for gfx950.
//
// Top-k sparsification (§III-C, §IV "High communication cost" of ScaDLES,
// arXiv 2301.08897) keeps, per device, the k entries of largest |g| (ties to
// the lower index) in ascending index order. Magnitudes are ranked as the
// 31-bit integer key bits(g) & 0x7FFFFFFF, whose order is that of |g| for
// finite values, so every decision below is exact integer work.
//
// Fast path (one read of every gradient):
//   1. bracket   : a systematic sample (256-element chunks at a fixed stride)
//                  is radix-selected at two ranks around k * (sample/n), giving
//                  keys t_lo <= (k-th largest key) < t_hi with high probability;
//   2. main pass : every gradient is read once; each wave stages the keys >= t_lo
//                  of its 4096-element chunk ("slot": index, value pairs in
//                  index order) with counts of keys >= t_lo and >= t_hi; sum g^2
//                  is fused in; a scan of the counts gives every slot's offsets;
//   3. threshold : the keys of the selection interval ([t_lo, t_hi), or above
//                  t_hi when that already holds k keys) are copied to a short
//                  list, and the exact k-th largest key is radix-selected on it;
//   4. output    : per group of slots, the kept entries -- keys above the
//                  threshold plus the lowest-indexed `need` keys equal to it --
//                  are counted, scanned and written in index order.
// If the bracket missed (fewer than k candidates) or the candidates overflow
// their region, the device falls back to the exact path: a radix select over
// all of its data, then an ordered compaction over its data.
#include "frame.h"
#include "marks.h"

namespace scadles {

constexpr uint32_t kNoDevice = 0xFFFFFFFFu;

// ---- radix-selection digit view ------------------------------------------------------------
struct SelView {
  uint32_t lo, hi, shift, width, prefix;
};

// Width of the pending digit. The sample selections take 11-bit digits from
// the top (their bracket stops after kBracketPasses digits); the exact
// selections take the remainder bits first and 11-bit digits after, the same
// number of passes with the smallest histogram in the first pass, which sees
// the most keys and flushes the most bins.
__device__ inline uint32_t digit_width(uint32_t bits, bool remainder_first)
{
  if (bits <= (uint32_t)kDigitBits) return bits;
  if (!remainder_first) return (uint32_t)kDigitBits;
  const uint32_t r = bits % (uint32_t)kDigitBits;
  return r ? r : (uint32_t)kDigitBits;
}

__device__ inline SelView view_of(const Sel& s, bool remainder_first)
{
  SelView v;
  v.lo = s.lo;
  v.hi = s.hi;
  v.width = digit_width(s.bits, remainder_first);
  v.shift = s.bits - v.width;
  v.prefix = s.prefix;
  return v;
}

// Digit of `key` for the pending pass, if the key is in the band and matches the
// digits decided so far.
__device__ inline bool sel_digit(const SelView& v, uint32_t key, uint32_t& d)
{
  if (key < v.lo || key >= v.hi) return false;
  const uint32_t o = key - v.lo;
  if ((o >> (v.shift + v.width)) != v.prefix) return false;
  d = (o >> v.shift) & ((1u << v.width) - 1u);
  return true;
}

// Threshold, count above it and ties kept, from whichever selection decided it.
__device__ inline bool threshold_of(const DevState& s, uint32_t& thr, uint64_t& need)
{
  const Sel& sel = s.fallback ? s.sel[kSlotFull] : s.sel[kSlotCand];
  if (!sel.found) {
    thr = kKeyInf;
    need = 0;
    return false;
  }
  thr = sel.result;
  need = sel.rank;
  return true;
}

__device__ inline void flush_hist(const uint32_t* h, uint32_t* g, int nb)
{
  for (int b = threadIdx.x; b < nb; b += kBlock) {
    uint32_t v = h[b];
    if (v) atomicAdd(g + b, v);
  }
}

// ---- block-wide rank selection over a histogram -----------------------------------------------
// Among nb bins (nb a multiple of NT) holding counts of keys by digit, finds the
// bin of the key of 1-based descending rank `rank` (the largest digit is the
// top bin) and the number of keys in the bins above it. Every thread returns
// the same result; false (bin 0, above = total) when rank exceeds the total.
// The histogram must be complete (a barrier before the call); s_w holds
// NT / 64 + 3 words of LDS.
template <int NT>
__device__ inline bool block_find(const uint32_t* h, int nb, uint64_t rank, uint32_t* s_w, uint32_t& bin,
                                  uint64_t& above)
{
  constexpr int kW = NT / 64;
  const int per = nb / NT;
  const uint32_t tid = threadIdx.x, w = tid >> 6;
  const int b_hi = nb - (int)tid * per;               // this thread's bins [b_hi - per, b_hi), top first
  uint32_t sum = 0;
  for (int i = 0; i < per; ++i) sum += h[b_hi - 1 - i];
  const uint32_t incl = wave_incl_scan(sum);
  if (lane_id() == 63) s_w[w] = incl;
  if (tid == 0) s_w[kW + 2] = 0u;
  __syncthreads();
  uint64_t excl = incl - sum;
  for (uint32_t i = 0; i < w; ++i) excl += s_w[i];
  if (excl < rank && rank <= excl + sum) {
    uint64_t cum = excl;
    for (int i = 0; i < per; ++i) {
      const uint32_t v = h[b_hi - 1 - i];
      if (cum + v >= rank) {
        s_w[kW] = (uint32_t)(b_hi - 1 - i);
        s_w[kW + 1] = (uint32_t)(cum - excl);       // within this thread's share: < 2^32
        s_w[kW + 2] = 1u + tid;
        break;
      }
      cum += v;
    }
  }
  __syncthreads();
  const uint32_t who = s_w[kW + 2];
  const bool ok = who != 0u;
  if (ok) {
    bin = s_w[kW];
    // the finder's exclusive prefix: the wave totals before its wave, then the
    // bins of the lanes before it in its wave, then its own bins above the hit
    const uint32_t ft = who - 1u, fw = ft >> 6;
    uint64_t pre = 0;
    for (uint32_t i = 0; i < fw; ++i) pre += s_w[i];
    for (int b = nb - (int)(fw * 64) * per - 1; b >= nb - (int)ft * per; --b) pre += h[b];
    above = pre + s_w[kW + 1];
  } else {
    bin = 0;
    uint64_t tot = 0;
    for (int i = 0; i < kW; ++i) tot += s_w[i];
    above = tot;
  }
  __syncthreads();
  return ok;
}

// Bracket of the main pass from the sample selections. The bracket only has to
// be conservative (t_lo at or below the sample key of rank r_lo, t_hi above the
// one of rank r_hi), so the selections stop after kBracketPasses digits: the
// rank's bin [B, B + 2^bits) gives t_lo = B and t_hi = B + 2^bits. A selection
// that missed gives t_lo = 0 (every key a candidate) or no upper bracket.
constexpr int kBracketPasses = 2;

__device__ inline void bracket_of(const DevDesc& d, const DevState& s, uint32_t& tlo, uint32_t& thi)
{
  if (d.mode != kModeFast) {
    tlo = thi = kKeyInf;
    return;
  }
  const Sel& a = s.sel[kSlotSampleLo];
  const Sel& b = s.sel[kSlotSampleHi];
  tlo = a.found ? a.result : (a.active ? a.lo + (a.prefix << a.bits) : 0u);
  if (b.found) {
    thi = b.result + 1u;
  } else if (b.active) {
    const uint64_t top = (uint64_t)b.lo + ((uint64_t)(b.prefix + 1u) << b.bits);
    thi = top < (uint64_t)kKeyInf ? (uint32_t)top : kKeyInf;
  } else {
    thi = kKeyInf;
  }
  if (thi <= tlo) thi = kKeyInf;
}

// ---- 0. per-call preparation -----------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_prep(Ctx c, PrepArgs a)
{
  const uint32_t K = c.K;
  if (blockIdx.x == 0 && threadIdx.x < K) {
    const uint32_t j = threadIdx.x;
    uint64_t off = 0;
    for (uint32_t i = 0; i < j; ++i) off += a.cap[i];
    DevDesc d;
    d.grad = a.grad[j];
    d.idx_out = a.idx[j];
    d.val_out = a.val[j];
    d.cand_off = off;
    d.k = a.k[j];
    d.cap = a.cap[j];
    d.mode = a.mode[j];
    d.r_lo = a.r_lo[j];
    d.r_hi = a.r_hi[j];
    d.shift = (uint32_t)((reinterpret_cast<uintptr_t>(a.grad[j]) >> 2) & 3u);
    c.desc[j] = d;
    DevState s;
    __builtin_memset(&s, 0, sizeof(s));
    s.t_lo = s.t_hi = kKeyInf;
    s.thr = kKeyInf;
    if (d.mode == kModeFast) {
      Sel& lo = s.sel[kSlotSampleLo];
      lo.active = 1;
      lo.lo = 0;
      lo.hi = kKeyInf;
      lo.bits = 31;
      lo.rank = d.r_lo;
      if (d.r_hi >= 1) {
        Sel& hi = s.sel[kSlotSampleHi];
        hi.active = 1;
        hi.lo = 0;
        hi.hi = kKeyInf;
        hi.bits = 31;
        hi.rank = d.r_hi;
      }
    }
    c.st[j] = s;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *c.fb_count = 0u;
  const uint64_t nh = (uint64_t)K * kSlots * kBins;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < nh; i += stride) c.hist[i] = 0u;
}

// ---- 1. bracket: histogram pass over the systematic sample (two selections) ----------------
__global__ __launch_bounds__(kBlock) void k_hist_sample(Ctx c)
{
  __shared__ uint32_t h[2][kBins];
  const uint32_t j = blockIdx.y;
  const DevDesc& d = c.desc[j];
  if (d.mode != kModeFast) return;
  const Sel s0 = c.st[j].sel[kSlotSampleLo];
  const Sel s1 = c.st[j].sel[kSlotSampleHi];
  if (!s0.active && !s1.active) return;
  const uint64_t e0 = (uint64_t)blockIdx.x * kSBlk;
  if (e0 >= c.s_n) return;
  const SelView v0 = view_of(s0, false), v1 = view_of(s1, false);
  // both selections at the same digit (always in the first pass): one histogram
  const bool same = s0.active && s1.active && v0.lo == v1.lo && v0.hi == v1.hi && v0.shift == v1.shift &&
                    v0.width == v1.width && v0.prefix == v1.prefix;
  for (int b = threadIdx.x; b < 2 * kBins; b += kBlock) (&h[0][0])[b] = 0u;
  constexpr int kR = kSBlk / kRound;
  const uint64_t e1 = (e0 + kSBlk < c.s_n) ? e0 + kSBlk : c.s_n;
  f4 x[kR];
#pragma unroll
  for (int r = 0; r < kR; ++r) {
    const uint64_t e = e0 + (uint64_t)r * kRound + threadIdx.x * 4;
    const uint64_t chunk = e / kSChunk, within = e % kSChunk;
    const uint64_t i = chunk * c.s_stride + within;     // real position of sample element e
    if (d.shift == 0 && e + 4 <= e1) x[r] = ld4(d.grad + i);
    else
      for (int q = 0; q < 4; ++q) x[r][q] = (e + q < e1) ? gptr(d.grad)[i + q] : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kR; ++r) {
    const uint64_t e = e0 + (uint64_t)r * kRound + threadIdx.x * 4;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (e + q >= e1) break;
      const uint32_t key = key_of(x[r][q]);
      uint32_t dg;
      if (s0.active && sel_digit(v0, key, dg)) atomicAdd(&h[0][dg], 1u);
      if (!same && s1.active && sel_digit(v1, key, dg)) atomicAdd(&h[1][dg], 1u);
    }
  }
  __syncthreads();
  if (s0.active) flush_hist(h[0], c.hist + ((uint64_t)j * kSlots + kSlotSampleLo) * kBins, kBins);
  if (s1.active) flush_hist(same ? h[0] : h[1], c.hist + ((uint64_t)j * kSlots + kSlotSampleHi) * kBins, kBins);
}

// ---- radix digit decision for slots [s0, s1) of one device (one wave) -----------------------
// With `bracket` set (the last pass of the sampling stage), the device's
// bracket [t_lo, t_hi) is then stored in its state for the main pass.
__global__ __launch_bounds__(64) void k_find(Ctx c, int s_begin, int s_end, int bracket)
{
  const uint32_t j = c.j0 + blockIdx.x, l = lane_id();
  for (int s = s_begin; s < s_end; ++s) {
    Sel sel = c.st[j].sel[s];
    if (!sel.active) continue;
    uint32_t* h = c.hist + ((uint64_t)j * kSlots + s) * kBins;
    const uint32_t w = digit_width(sel.bits, s >= kSlotCand);
    const int nb = 1 << w;
    const int per = (nb + 63) / 64;                // bins per lane, at most 32
    const int b_hi = nb - (int)l * per;           // this lane covers bins [b_lo, b_hi), top first
    const int b_lo = b_hi - per > 0 ? b_hi - per : 0;
    uint32_t hv[32];
    uint32_t sum = 0;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int b = b_hi - 1 - i;
      hv[i] = (i < per && b >= b_lo) ? h[b] : 0u;
      sum += hv[i];
    }
    const uint32_t incl = wave_incl_scan(sum);
    const uint32_t excl = incl - sum;
    const bool hit = (uint64_t)excl < sel.rank && sel.rank <= (uint64_t)incl;
    const uint64_t m = ballot(hit);
    uint32_t dsel = 0, cum = excl;
    if (hit) {
      bool done = false;
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        if (!done && (uint64_t)cum + hv[i] >= sel.rank) {
          dsel = (uint32_t)(b_hi - 1 - i);
          done = true;
        }
        if (!done) cum += hv[i];
      }
    }
    const int src = m ? __builtin_ctzll(m) : 0;
    dsel = __shfl(dsel, src, 64);
    cum = __shfl(cum, src, 64);
    if (l == 0) {
      if (!m) {
        sel.active = 0;
        sel.found = 0;
        c.st[j].err |= s < kSlotCand ? kErrBracket : kErrSelect;   // a bracket miss sends the device to the exact path
      } else {
        sel.rank -= cum;
        sel.above += cum;
        sel.prefix = (sel.prefix << w) | dsel;
        sel.bits -= w;
        if (sel.bits == 0) {
          sel.active = 0;
          sel.found = 1;
          sel.result = sel.lo + sel.prefix;
        }
      }
      c.st[j].sel[s] = sel;
    }
    for (int b = l; b < kBins; b += 64) h[b] = 0u;
  }
  if (bracket && l == 0) {
    uint32_t tlo, thi;
    bracket_of(c.desc[j], c.st[j], tlo, thi);
    c.st[j].t_lo = tlo;
    c.st[j].t_hi = thi;
  }
}

// ---- 2. main pass: one read of every gradient ------------------------------------------------
// No workgroup waits on another: wave w of tile t of device j stages its
// candidates (keys >= t_lo) in index order and writes them to its own slot
// (kWaveCap entries) with a count; a per-device scan of the slot counts then
// gives every slot its offset in the device's candidate list.
template <int R>
__device__ inline uint64_t elem_of(uint32_t w, int r, uint32_t l)
{
  return (uint64_t)w * (R * 256) + (uint64_t)r * 256 + l * 4;
}

// Exclusive per-wave prefix and block total of one packed (lo16 | hi16 << 16)
// per-lane count; lds needs 8 words.
__device__ inline uint32_t wave_prefix_of_block(uint32_t packed_lane, uint32_t* lds, uint32_t& total)
{
  const uint32_t w = threadIdx.x >> 6;
  uint32_t t = packed_lane;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) t += __shfl_xor(t, d, 64);
  if (lane_id() == 0) lds[w] = t;
  __syncthreads();
  uint32_t ex = 0;
  for (uint32_t i = 0; i < w; ++i) ex += lds[i];
  total = lds[0] + lds[1] + lds[2] + lds[3];
  __syncthreads();
  return ex;
}

// One round of phase 1 for one wave: sum of squares, counts of candidates
// (key >= tlo) and sure keys (key >= thi), and the round's candidates staged in
// LDS in index order (lane, then component) after the `wc` already staged, the
// keys of those below thi (the selection interval) likewise in s_b.
// kEdge: the round may hold pads (pattern 0xFFFFFFFF), so keys are compared as
// rank keys (key + 1, pads 0) and fmax drops the pads' NaN from the squares.
// Counts are wave totals from ballots (scalar popcounts).
// A staged candidate: its index in the low word, its value's bits in the high word.
// A tile's slot region (kSlotWords words, consecutive tiles back to back):
// words 0 .. band - 1 hold the keys of the candidates below t_hi (the
// selection interval), word band + e candidate e's value bits, and the 16-bit
// word (2 * kSlotWords - 1 - e) candidate e's offset in the tile (index = tile
// * kTile - shift + offset). The keys start at a fixed place, so their readers
// load them before the counts arrive. Both ends are written as whole 16-byte
// chunks; a tile whose two parts would meet overflows.
static_assert((kSlotWords & (kSlotWords - 1)) == 0, "slot positions wrap inside a power-of-two region");
__device__ inline uint32_t slot_off16_at(uint32_t e) { return 2u * kSlotWords - 1u - e; }

__device__ inline uint64_t pack_cand(uint32_t i, float v) { return (uint64_t)i | ((uint64_t)__float_as_uint(v) << 32); }

template <bool kEdge>
__device__ inline void main_stage(const f4& x, uint32_t i0, uint32_t tlo, uint32_t thi, double (&e2)[2], uint32_t& wc,
                                  uint32_t& ws, uint64_t* s_c, uint32_t* s_b)
{
  uint64_t b[4], bb[4];
  bool f[4], fb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const double xd = (double)x[q];
    if (kEdge) e2[q & 1] += __builtin_fmax(xd * xd, 0.0);
    else e2[q & 1] = __builtin_fma(xd, xd, e2[q & 1]);
    const uint32_t key = kEdge ? rank_key(x[q]) : key_of(x[q]);
    const uint32_t lo = kEdge ? tlo + 1u : tlo, hi = kEdge ? thi + 1u : thi;
    f[q] = key >= lo;
    fb[q] = f[q] && key < hi;
    b[q] = ballot(f[q]);
    bb[q] = ballot(fb[q]);
  }
  const uint64_t any = b[0] | b[1] | b[2] | b[3];
  if (any == 0ull) return;
  const uint32_t nb = (uint32_t)(__builtin_popcountll(bb[0]) + __builtin_popcountll(bb[1]) +
                                 __builtin_popcountll(bb[2]) + __builtin_popcountll(bb[3]));
  const uint32_t nc = (uint32_t)(__builtin_popcountll(b[0]) + __builtin_popcountll(b[1]) +
                                 __builtin_popcountll(b[2]) + __builtin_popcountll(b[3]));
  // wb, the wave's staged selection keys so far, is wc - ws
  uint32_t pos = wc + mbcnt(b[0]) + mbcnt(b[1]) + mbcnt(b[2]) + mbcnt(b[3]);
  uint32_t bpos = (wc - ws) + mbcnt(bb[0]) + mbcnt(bb[1]) + mbcnt(bb[2]) + mbcnt(bb[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (f[q]) {
      if (pos < (uint32_t)kWaveCap) s_c[pos] = pack_cand(i0 + q, x[q]);
      ++pos;
    }
    if (fb[q]) {
      if (bpos < (uint32_t)kWaveCap) s_b[bpos] = key_of(x[q]);
      ++bpos;
    }
  }
  wc += nc;
  ws += nc - nb;
}

// Each workgroup reads one tile of kTile gradient elements (workgroup b: device
// b / tpd, tile b % tpd). Wave w owns elements [w*4096, (w+1)*4096) of the tile
// and stages its candidates in LDS; the tile's slot is written at the end (the
// only barrier). The gradient pointers come as kernel arguments so that the
// tile's loads issue before anything is read from the workspace.
__global__ __launch_bounds__(kBlock) void k_main(Ctx c, GradArgs ga)
{
  __shared__ uint64_t s_c[kWaves][kWaveCap];
  __shared__ uint32_t s_b[kWaves][kWaveCap];
  const uint32_t l = lane_id(), w = threadIdx.x >> 6;
  const uint32_t jr = blockIdx.x / c.tpd, tile = blockIdx.x - jr * c.tpd;
  const uint32_t j = c.j0 + jr;
  const float* grad = ga.grad[j];
  const uint64_t shift = (reinterpret_cast<uintptr_t>(grad) >> 2) & 3u;
  const uint64_t vbase = (uint64_t)tile * kTile;      // virtual position of the tile
  const Row row{gptr(grad), shift, c.n};
  // Interior tiles hold only real elements: plain aligned loads kept in
  // registers. The (at most two) edge tiles of a device reload per round.
  const bool full = vbase >= row.shift && vbase + kTile <= row.shift + row.n;
  const uint32_t wv0 = (uint32_t)(w * (kTileRounds * 256) + l * 4);   // this lane's first element in the tile
  // real index of virtual position vbase + wv0 (may wrap for leading pads; never written)
  const uint32_t i_base = (uint32_t)(vbase + wv0 - row.shift);

  double e2[2] = {0.0, 0.0};
  uint32_t wc = 0, ws = 0;
  if (full) {
    const GLOBAL float* p = row.p + (vbase - row.shift) + wv0;
    f4 v[kTileRounds];
#pragma unroll
    for (int r = 0; r < kTileRounds; ++r) v[r] = ld_stream4(p + r * 256);
    const uint32_t tlo = c.st[j].t_lo, thi = c.st[j].t_hi;
#pragma unroll
    for (int r = 0; r < kTileRounds; ++r) {
      main_stage<false>(v[r], i_base + r * 256, tlo, thi, e2, wc, ws, s_c[w], s_b[w]);
      __builtin_amdgcn_sched_barrier(0);    // keep rounds apart: bounds the live ballot masks
    }
  } else {
    const uint32_t tlo = c.st[j].t_lo, thi = c.st[j].t_hi;
    for (int r = 0; r < kTileRounds; ++r)
      main_stage<true>(load4(row, vbase + wv0 + r * 256, false), i_base + r * 256, tlo, thi, e2, wc, ws, s_c[w],
                     s_b[w]);
  }
  // The tile's slot: the waves' staged candidates one after the other (index
  // order), then the keys of the candidates below t_hi (the selection
  // interval [t_lo, t_hi)), two per entry, as one contiguous rotated run; its
  // counts and sum of squares. A tile with a wave chunk over kWaveCap
  // candidates, or whose run would not fit the region, stages nothing and is
  // recorded for k_overflow, which re-scans it once the slot offsets are known;
  // its region then holds the per-chunk counts.
  __shared__ uint32_t s_cnt[kWaves];
  __shared__ double s_e[kWaves];
  const double es = wave_sum_f64(e2[0] + e2[1]);
  if (l == 0) {
    s_cnt[w] = wc | (ws << 16);
    s_e[w] = es;
  }
  __syncthreads();
  // cb[i] / kb[i]: candidates / selection keys of the waves before wave i
  uint32_t cb[kWaves + 1], kb[kWaves + 1];
  bool ovf = false;
  cb[0] = kb[0] = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    const uint32_t v = s_cnt[i], wci = v & 0xFFFFu;
    cb[i + 1] = cb[i] + wci;
    kb[i + 1] = kb[i] + wci - (v >> 16);
    ovf |= wci > (uint32_t)kWaveCap;
  }
  const uint32_t cand = cb[kWaves], band = kb[kWaves], sure = cand - band;
  const uint32_t na = (cand + band + 3u) / 4u, nbk = ((cand + 1u) / 2u + 3u) / 4u;   // 16-byte chunks of both ends
  ovf |= 4u * (na + nbk) > (uint32_t)kSlotWords;
  const uint64_t slot = (uint64_t)j * c.nslot + tile;
  if (threadIdx.x == 0) {
    c.slot_cnt[slot] = cand | (ovf ? 0x8000u : 0u) | (sure << 16);
    c.epart[slot] = (s_e[0] + s_e[1]) + (s_e[2] + s_e[3]);
    if (ovf) {
      const uint32_t i = atomicAdd(&c.st[j].ovf_n, 1u);
      c.ovf_list[(uint64_t)j * c.nslot + i] = tile;
    }
  }
  GLOBAL uint32_t* reg = gptr(c.slot) + slot * kSlotWords;
  if (ovf) {
    // per-chunk candidate and selection-key counts for k_overflow
    if (threadIdx.x < 2 * kWaves) {
      const uint32_t v = s_cnt[threadIdx.x & (kWaves - 1)];
      reg[threadIdx.x] = threadIdx.x < kWaves ? (v & 0xFFFFu) : (v & 0xFFFFu) - (v >> 16);
    }
    return;
  }
  // The whole workgroup writes both ends, 16 bytes per thread (nontemporal:
  // the slots are read only after the whole pass).
  const uint32_t* c32 = reinterpret_cast<const uint32_t*>(&s_c[0][0]);
  const uint32_t* b32 = &s_b[0][0];
  auto cand_word = [&](uint32_t e, uint32_t half) -> uint32_t {    // half 0: index, 1: value bits
    const uint32_t wi = (uint32_t)(e >= cb[1]) + (uint32_t)(e >= cb[2]) + (uint32_t)(e >= cb[3]);
    const uint32_t base = wi == 0 ? cb[0] : (wi == 1 ? cb[1] : (wi == 2 ? cb[2] : cb[3]));
    return c32[wi * (2 * kWaveCap) + 2u * (e - base) + half];
  };
  auto low_word = [&](uint32_t q) -> uint32_t {
    if (q < band) {
      const uint32_t wi = (uint32_t)(q >= kb[1]) + (uint32_t)(q >= kb[2]) + (uint32_t)(q >= kb[3]);
      const uint32_t base = wi == 0 ? kb[0] : (wi == 1 ? kb[1] : (wi == 2 ? kb[2] : kb[3]));
      return b32[wi * kWaveCap + (q - base)];
    }
    const uint32_t e = q - band;
    return e < cand ? cand_word(e, 1u) : 0u;
  };
  const uint32_t ibase = (uint32_t)(vbase - row.shift);   // index of tile position 0 (mod 2^32)
  auto off16 = [&](uint32_t e) -> uint32_t { return e < cand ? (cand_word(e, 0u) - ibase) & 0xFFFFu : 0u; };
  for (uint32_t t = threadIdx.x; t < na + nbk; t += kBlock) {
    u4 v;
    uint32_t p0;
    if (t < na) {
      p0 = 4u * t;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = low_word(p0 + i);
    } else {
      p0 = kSlotWords - 4u * nbk + 4u * (t - na);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t e_lo = slot_off16_at(2u * (p0 + i));     // candidate in the word's low half
        v[i] = off16(e_lo) | (off16(e_lo - 1u) << 16);
      }
    }
    __builtin_nontemporal_store(v, reinterpret_cast<GLOBAL u4*>(reg + p0));
  }
}

// ---- after the main pass: energies, slot offsets, candidate totals, path decision ----------
__device__ inline uint64_t wave_incl_scan_u64(uint64_t v)
{
  const uint32_t l = lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint64_t t = __shfl_up(v, d, 64);
    if (l >= (uint32_t)d) v += t;
  }
  return v;
}

// One workgroup per device: the exclusive prefix of the tiles' candidate | sure
// << 32 counts (each thread takes a run of consecutive tiles), the sum of
// squares over all tiles in a fixed order, then the path decision: the exact
// path (fallback) or the radix selection on the selection interval. NT = 1024
// when it runs alone; 256 when it runs beside another selection's main pass,
// whose stream of small workgroups rarely leaves 16 waves of a compute unit
// free at once.
constexpr int kScanBlockLarge = 1024, kScanBlockSmall = 256;
template <int kScanBlock>
__global__ __launch_bounds__(kScanBlock) void k_scan(Ctx c)
{
  constexpr int kW = kScanBlock / 64;
  __shared__ uint64_t s_w[kW];
  __shared__ double s_e[kW];
  const uint32_t j = c.j0 + blockIdx.x, tid = threadIdx.x, w = tid >> 6;
  const DevDesc d = c.desc[j];
  const bool fast = d.mode == kModeFast;
  const uint32_t per = (c.nslot + kScanBlock - 1) / kScanBlock;
  const uint32_t t0 = tid * per < c.nslot ? tid * per : c.nslot;
  const uint32_t t1 = t0 + per < c.nslot ? t0 + per : c.nslot;
  const uint32_t* cnt = c.slot_cnt + (uint64_t)j * c.nslot;
  const double* ep = c.epart + (uint64_t)j * c.nslot;
  uint64_t sum = 0;
  double e = 0.0;
  for (uint32_t t = t0; t < t1; ++t) {
    e += ep[t];
    if (fast) {
      const uint32_t v = cnt[t];
      sum += (uint64_t)(v & 0x7FFFu) | ((uint64_t)(v >> 16) << 32);
    }
  }
  // energies: per thread in tile order, then lanes and waves in a fixed pattern
  const double ew = wave_sum_f64(e);
  const uint64_t incl = wave_incl_scan_u64(sum);
  if (lane_id() == 63) s_w[w] = incl;
  if (lane_id() == 0) s_e[w] = ew;
  __syncthreads();
  uint64_t run = incl - sum;
  for (uint32_t i = 0; i < w; ++i) run += s_w[i];
  if (fast) {
    uint64_t* off = c.slot_off + (uint64_t)j * c.nslot;
    for (uint32_t t = t0; t < t1; ++t) {
      off[t] = run;
      const uint32_t v = cnt[t];
      run += (uint64_t)(v & 0x7FFFu) | ((uint64_t)(v >> 16) << 32);
    }
  }
  if (tid != 0) return;
  uint64_t tot = 0;
  double e_all = 0.0;
  for (int i = 0; i < kW; ++i) {
    tot += s_w[i];
    e_all += s_e[i];
  }
  DevState& s = c.st[j];
  s.e_all = e_all;
  bool fb = !fast || c.force_fallback;
  const uint32_t tlo = s.t_lo, thi = s.t_hi;
  if (fast) {
    s.cand = tot & 0xFFFFFFFFull;
    s.sure = tot >> 32;
    if (s.err) fb = true;
    // the selection interval must hold the k-th largest key: fewer than k sure keys
    if (s.cand < d.k || s.cand > d.cap || s.sure >= d.k) fb = true;
  }
  Sel sel;
  __builtin_memset(&sel, 0, sizeof(sel));
  sel.active = 1;
  if (fb) {
    s.fallback = 1;
    atomicAdd(c.fb_count, 1u);
    sel.lo = 0;
    sel.hi = kKeyInf;
    sel.bits = 31;
    sel.rank = d.k;
    s.sel[kSlotFull] = sel;
  } else {
    s.fallback = 0;
    sel.lo = tlo;
    sel.hi = thi;
    sel.rank = d.k - s.sure;
    const uint32_t b = bitlen32(sel.hi - sel.lo - 1u);
    sel.bits = b ? b : 1u;
    s.sel[kSlotCand] = sel;
  }
}

// Candidate counts before slot s of device j: candidates | sure << 32.
__device__ inline uint64_t slot_pre(const Ctx& c, uint32_t j, uint32_t s)
{
  if (s >= c.nslot) return c.st[j].cand | (c.st[j].sure << 32);
  return c.slot_off[(uint64_t)j * c.nslot + s];
}

// ---- 3. selection-interval keys per tile ---------------------------------------------------
// The keys of a tile's candidates below t_hi (the selection interval [t_lo,
// t_hi)) start its slot region; k_overflow writes those of an overflowed tile
// to the device's band list at the tile's band offset (candidates - sure keys
// before it). band_tiles walks them for tiles t0 .. t0 + kBT - 1 of
// device j, tile after tile, in index order within a tile, 64 at a time:
// visit(key, valid) takes one window, done(i, sure) closes tile t0 + i (sure:
// its keys >= t_hi). The first window of every tile is loaded at once, before
// the counts arrive (lane l then holds tile t0 + l's counts), longer runs four
// windows at once; all without conditions: tile indices are clamped, region
// positions wrap inside the region and band-list positions are clamped into
// the tile's run, so every load is in bounds; keys past a tile's count are
// ignored. Sources of the staged tiles' keys (kSrc): kBandRegions, their
// slot regions; kBandCopy, the same, also copying the keys to the band list
// at the tiles' band offsets, which completes the list (the overflowed tiles'
// keys are there already): the device's selection-interval keys, contiguous
// and in index order; kBandList, that completed list (every tile's first
// window then loads once its offset is known). kBT, the tiles per wave, is
// chosen per call (band_tiles_per_wave).
constexpr int kBandRegions = 0, kBandCopy = 1, kBandList = 2;

template <int kBT, int kSrc = kBandRegions, class Visit, class Done>
__device__ inline void band_tiles(const Ctx& c, uint32_t j, uint32_t t0, Visit visit, Done done)
{
  constexpr uint32_t kMask = kSlotWords - 1u;
  constexpr bool kCopy = kSrc == kBandCopy;
  const uint32_t l = lane_id();
  const uint32_t last = c.nslot - 1;
  const uint64_t row = (uint64_t)j * c.nslot;
  const GLOBAL uint32_t* reg = gptr(c.slot);
  uint32_t kv[kBT];
  if (kSrc != kBandList) {
#pragma unroll
    for (int i = 0; i < kBT; ++i) {
      const uint32_t ti = t0 + i < last ? t0 + i : last;
      kv[i] = reg[(row + ti) * kSlotWords + l];
    }
  }
  const uint32_t tl = t0 + l < last ? t0 + l : last;
  const uint32_t v = t0 + l < c.nslot ? c.slot_cnt[row + tl] : 0u;
  const uint32_t cand = v & 0x7FFFu, sure = v >> 16, nb = cand - sure;
  const uint32_t ovf = (v >> 15) & 1u;
  uint32_t kb = 0;                                      // the tile's keys: band-list position
  if (ovf || kSrc != kBandRegions) {
    const uint64_t pre = slot_pre(c, j, tl);
    kb = (uint32_t)pre - (uint32_t)(pre >> 32);
  }
  const uint32_t nt = c.nslot - t0 < (uint32_t)kBT ? c.nslot - t0 : (uint32_t)kBT;
  GLOBAL uint32_t* blist = gptr(c.band) + c.desc[j].cand_off;
  if (kSrc == kBandList) {
    // first windows: key l of tile i (loaded only where it exists)
#pragma unroll
    for (int i = 0; i < kBT; ++i)
      kv[i] = l < __builtin_amdgcn_readlane(nb, i) ? blist[__builtin_amdgcn_readlane(kb, i) + l] : 0u;
  }
  // windows e0 .. of a run of nbi keys, four at a time; key_at(e) is in bounds
  // for every e; key e also goes to dst[e] when dst is set
  auto run = [&](uint32_t e0, uint32_t nbi, auto key_at, GLOBAL uint32_t* dst) {
    for (uint32_t e = e0; e < nbi; e += 256) {
      uint32_t w4[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) w4[m] = key_at(e + m * 64 + l);
#pragma unroll
      for (int m = 0; m < 4; ++m)
        if (e + m * 64 < nbi) {
          const bool valid = e + m * 64 + l < nbi;
          if (dst && valid) dst[e + m * 64 + l] = w4[m];
          visit(w4[m], valid);
        }
    }
  };
#pragma unroll
  for (int i = 0; i < kBT; ++i) {
    if ((uint32_t)i >= nt) break;
    const uint32_t nbi = __builtin_amdgcn_readlane(nb, i);
    if (kSrc == kBandList) {
      visit(kv[i], l < nbi);
      const GLOBAL uint32_t* p = blist + __builtin_amdgcn_readlane(kb, i);
      if (nbi > 64u) run(64u, nbi, [&](uint32_t e) { return p[e < nbi ? e : nbi - 1u]; }, nullptr);
    } else if (!__builtin_amdgcn_readlane(ovf, i)) {
      GLOBAL uint32_t* dst = kCopy ? blist + __builtin_amdgcn_readlane(kb, i) : nullptr;
      if (kCopy && l < nbi) dst[l] = kv[i];
      visit(kv[i], l < nbi);
      const GLOBAL uint32_t* base = reg + (row + t0 + i) * kSlotWords;
      if (nbi > 64u) run(64u, nbi, [&](uint32_t e) { return base[e & kMask]; }, dst);
    } else if (nbi) {
      const GLOBAL uint32_t* p = blist + __builtin_amdgcn_readlane(kb, i);
      run(0u, nbi, [&](uint32_t e) { return p[e < nbi ? e : nbi - 1u]; }, nullptr);
    }
    done(i, __builtin_amdgcn_readlane(sure, i));
  }
}

// Overflowed tiles (a wave chunk of more than kWaveCap candidates, or more
// candidates and selection-interval keys than the slot region holds): re-scan
// the tile and write its candidates, in index order, at the tile's offset in
// the candidate list, and the keys of those below t_hi at its offset in the
// band list. The work items are (tile, chunk) pairs, chunk c being the 4096
// elements the main pass's wave c read; the main pass left each chunk's
// candidate and selection-key counts in the tile's (otherwise unused) slot
// region, so an item's offsets are known without the rest of the tile.
// Workgroup b of a device takes items b, b + blocks_per_dev, ...; its wave w
// takes 1024 elements of the chunk. Keys are compared as in the main pass:
// plain keys in interior tiles, rank keys (key + 1, pads 0) in edge tiles.
constexpr int kChunkRounds = kTileRounds / kWaves;    // rounds of one wave in one chunk

__global__ __launch_bounds__(kBlock) void k_overflow(Ctx c, uint32_t blocks_per_dev)
{
  __shared__ uint32_t s_n[kWaves], s_b[kWaves];
  const uint32_t jr = blockIdx.x / blocks_per_dev, b = blockIdx.x - jr * blocks_per_dev;
  const uint32_t j = c.j0 + jr;
  const DevState& st = c.st[j];
  if (st.fallback) return;
  const uint32_t items = st.ovf_n * kWaves;
  const DevDesc d = c.desc[j];
  const uint32_t l = lane_id(), w = threadIdx.x >> 6;
  const Row row{gptr(d.grad), d.shift, c.n};
  GLOBAL uint32_t* cidx = gptr(c.cand_idx + d.cand_off);
  GLOBAL float* cval = gptr(c.cand_val + d.cand_off);
  GLOBAL uint32_t* band = gptr(c.band + d.cand_off);
  for (uint32_t it = b; it < items; it += blocks_per_dev) {
    const uint32_t s = c.ovf_list[(uint64_t)j * c.nslot + it / kWaves], ch = it % kWaves;
    const uint64_t slot = (uint64_t)j * c.nslot + s;
    const GLOBAL uint32_t* ccnt = gptr(c.slot) + slot * kSlotWords;
    const uint64_t vbase = (uint64_t)s * kTile;
    const bool full = vbase >= row.shift && vbase + kTile <= row.shift + row.n;
    const uint32_t lo = full ? st.t_lo : st.t_lo + 1u, hi = full ? st.t_hi : st.t_hi + 1u;
    const uint64_t v0 = vbase + (uint64_t)ch * (kTileRounds * 256) + (uint64_t)w * (kChunkRounds * 256) + l * 4;
    f4 x[kChunkRounds];
#pragma unroll
    for (int r = 0; r < kChunkRounds; ++r) x[r] = load4(row, v0 + (uint64_t)r * 256, false);
    uint32_t cb = 0, bb0 = 0;       // candidates and selection keys of the chunks before
    for (uint32_t u = 0; u < ch; ++u) {
      cb += ccnt[u];
      bb0 += ccnt[kWaves + u];
    }
    auto key = [&](float v) { return full ? key_of(v) : rank_key(v); };
    uint32_t cnt = 0, bcnt = 0;
#pragma unroll
    for (int r = 0; r < kChunkRounds; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t kq = key(x[r][q]);
        cnt += (uint32_t)__builtin_popcountll(ballot(kq >= lo));
        bcnt += (uint32_t)__builtin_popcountll(ballot(kq >= lo && kq < hi));
      }
    if (l == 0) {
      s_n[w] = cnt;
      s_b[w] = bcnt;
    }
    __syncthreads();
    const uint64_t pre = slot_pre(c, j, s);
    uint64_t run = (uint32_t)pre + cb;
    uint64_t brun = (uint32_t)pre - (uint32_t)(pre >> 32) + bb0;
    for (uint32_t u = 0; u < w; ++u) {
      run += s_n[u];
      brun += s_b[u];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kChunkRounds; ++r) {
      bool f[4], fb[4];
      uint64_t bm[4], bbm[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t kq = key(x[r][q]);
        f[q] = kq >= lo;
        fb[q] = f[q] && kq < hi;
        bm[q] = ballot(f[q]);
        bbm[q] = ballot(fb[q]);
      }
      uint64_t pos = run + mbcnt(bm[0]) + mbcnt(bm[1]) + mbcnt(bm[2]) + mbcnt(bm[3]);
      uint64_t bpos = brun + mbcnt(bbm[0]) + mbcnt(bbm[1]) + mbcnt(bbm[2]) + mbcnt(bbm[3]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (f[q]) {
          if (pos < d.cap) {
            cidx[pos] = (uint32_t)(v0 + (uint64_t)r * 256 + q - row.shift);
            cval[pos] = x[r][q];
          }
          ++pos;
        }
        if (fb[q]) {
          if (bpos < d.cap) band[bpos] = key_of(x[r][q]);
          ++bpos;
        }
      }
      run += __builtin_popcountll(bm[0]) + __builtin_popcountll(bm[1]) + __builtin_popcountll(bm[2]) +
             __builtin_popcountll(bm[3]);
      brun += __builtin_popcountll(bbm[0]) + __builtin_popcountll(bbm[1]) + __builtin_popcountll(bbm[2]) +
              __builtin_popcountll(bbm[3]);
    }
  }
}

// ---- 4. histogram pass over selection-interval keys (fast devices) and full data (exact devices)
// Fast devices, first pass: workgroup b of device j takes tiles [b, b + 1) *
// kBT * kWaves, walking the tiles' keys and copying those of the
// staged tiles to the band list, which then holds all of the device's keys;
// later passes: workgroup b takes keys [b, b + 1) * kBandChunk of that list
// (and every per_dev-th chunk after it).
constexpr uint32_t kBandChunk = 16 * kBlock;
template <int kBT>
__global__ __launch_bounds__(kBlock) void k_hist_cf(Ctx c, uint32_t ncand_blocks, uint32_t pass)
{
  __shared__ uint32_t h[kBins];
  if (blockIdx.x < ncand_blocks) {
    const uint32_t per_dev = (c.nslot + kBT * kWaves - 1) / (kBT * kWaves);
    const uint32_t jr = blockIdx.x / per_dev, b = blockIdx.x - jr * per_dev;
    const uint32_t j = c.j0 + jr;
    const DevState& s = c.st[j];
    if (s.fallback) return;
    const Sel sel = s.sel[kSlotCand];
    if (!sel.active) return;
    const uint32_t nband = (uint32_t)(s.cand - s.sure);       // keys in [t_lo, t_hi): at most cap < 2^31
    if (pass > 0 && (uint64_t)b * kBandChunk >= nband) return;
    for (int i = threadIdx.x; i < kBins; i += kBlock) h[i] = 0u;
    __syncthreads();
    const SelView sv = view_of(sel, true);
    auto add = [&](uint32_t key, bool valid) {
      uint32_t dg;
      if (valid && sel_digit(sv, key, dg)) atomicAdd(&h[dg], 1u);
    };
    if (pass == 0) {
      const uint32_t t0 = (b * kWaves + (threadIdx.x >> 6)) * kBT;
      if (t0 < c.nslot) band_tiles<kBT, kBandCopy>(c, j, t0, add, [](uint32_t, uint32_t) {});
    } else {
      const GLOBAL uint32_t* blist = gptr(c.band) + c.desc[j].cand_off;
      for (uint64_t o = (uint64_t)b * kBandChunk; o < nband; o += (uint64_t)per_dev * kBandChunk) {
        uint32_t key[kBandChunk / kBlock];
#pragma unroll
        for (int r = 0; r < (int)(kBandChunk / kBlock); ++r) {
          const uint64_t e = o + (uint64_t)r * kBlock + threadIdx.x;
          key[r] = e < nband ? blist[e] : 0u;
        }
#pragma unroll
        for (int r = 0; r < (int)(kBandChunk / kBlock); ++r)
          add(key[r], o + (uint64_t)r * kBlock + threadIdx.x < nband);
      }
    }
    __syncthreads();
    flush_hist(h, c.hist + ((uint64_t)j * kSlots + kSlotCand) * kBins, kBins);
    return;
  }
  const uint32_t worker = blockIdx.x - ncand_blocks, G = gridDim.x - ncand_blocks;
  if (*c.fb_count == 0u) return;
  // Work items are the (device, block) pairs of the group, device-major, taken
  // grid-stride: every worker has a share of every exact-path device. A
  // worker's items of one device share its histogram, flushed when the device
  // changes (all conditions below are uniform over the workgroup).
  const uint64_t items = (uint64_t)c.jn * c.nfb;
  uint32_t cur = kNoDevice;
  SelView sv{};
  Row row{};
  for (uint64_t it = worker; it < items; it += G) {
    const uint32_t jr = (uint32_t)(it / c.nfb), blk = (uint32_t)(it - (uint64_t)jr * c.nfb);
    const uint32_t j = c.j0 + jr;
    if (j != cur) {
      if (cur != kNoDevice) {
        __syncthreads();
        flush_hist(h, c.hist + ((uint64_t)cur * kSlots + kSlotFull) * kBins, kBins);
        cur = kNoDevice;
      }
      const DevState& s = c.st[j];
      if (!s.fallback || !s.sel[kSlotFull].active) continue;
      __syncthreads();
      for (int i = threadIdx.x; i < kBins; i += kBlock) h[i] = 0u;
      __syncthreads();
      cur = j;
      sv = view_of(s.sel[kSlotFull], true);
      row = Row{gptr(c.desc[j].grad), c.desc[j].shift, c.n};
    }
    const uint64_t vbase = (uint64_t)blk * kCBlk;
#pragma unroll 4
    for (int r = 0; r < kCBlkRounds; ++r) {
      const uint64_t v = vbase + (uint64_t)r * kRound + threadIdx.x * 4;
      const f4 x = load4(row, v, true);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t dg;
        if (in_row(row, v + q) && sel_digit(sv, key_of(x[q]), dg)) atomicAdd(&h[dg], 1u);
      }
    }
  }
  if (cur != kNoDevice) {
    __syncthreads();
    flush_hist(h, c.hist + ((uint64_t)cur * kSlots + kSlotFull) * kBins, kBins);
  }
}

// ---- 5. ordered output of the fast path ----------------------------------------------------
// Output groups are kGatherSlots consecutive slots. Kept: key > thr, or
// key == thr while fewer than `need` equal keys came before (index order);
// a kept entry goes to (keys above thr before it) + min(equal keys before it, need).

// Per group: keys above the threshold | keys equal to it << 32. The threshold
// lies in [t_lo, t_hi): equal keys and the keys above it below t_hi are
// counted on the tiles' selection-interval keys, the keys >= t_hi come from
// the slot counts. One wave per kBT tiles (kBT / 2 groups).
template <int kBT>
__device__ inline void grp_count_body(const Ctx& c, uint32_t b)
{
  const uint32_t per_dev = (c.nslot + kBT * kWaves - 1) / (kBT * kWaves);
  const uint32_t jr = b / per_dev;
  const uint32_t j = c.j0 + jr;
  const uint32_t t0 = ((b - jr * per_dev) * kWaves + (threadIdx.x >> 6)) * kBT;
  const DevState& st = c.st[j];
  if (st.fallback || t0 >= c.nslot) return;
  static_assert(kGatherSlots == 2 && kBT % 2 == 0 && kBT <= 64, "groups are tile pairs; a lane holds a tile's counts");
  uint32_t thr;
  uint64_t need;
  threshold_of(st, thr, need);
  const uint32_t l = lane_id();
  uint32_t gt = 0, eq = 0;
  uint64_t mine = 0;
  // the first histogram pass completed the band list
  band_tiles<kBT, kBandList>(
      c, j, t0,
      [&](uint32_t key, bool valid) {
        gt += (uint32_t)__builtin_popcountll(ballot(valid && key > thr));
        eq += (uint32_t)__builtin_popcountll(ballot(valid && key == thr));
      },
      [&](uint32_t i, uint32_t sure) {
        gt += sure;
        if ((i & 1u) || t0 + i + 1 == c.nslot) {
          if (l == i / 2) mine = (uint64_t)gt | ((uint64_t)eq << 32);
          gt = eq = 0;
        }
      });
  const uint32_t g = t0 / 2 + l;
  if (l < (uint32_t)kBT / 2 && g < c.ngrp) c.grp_cnt[(uint64_t)j * c.ngrp + g] = mine;
}

// Exclusive prefix of nb packed counts, one workgroup.
__device__ inline void block_excl_scan_u64(const uint64_t* cnt, uint64_t* pre, uint32_t nb, uint64_t* s_w)
{
  const uint32_t tid = threadIdx.x;
  const uint32_t per = (nb + kBlock - 1) / kBlock;
  const uint32_t b0 = tid * per, b1 = (b0 + per < nb) ? b0 + per : nb;
  uint64_t sum = 0;
  for (uint32_t b = b0; b < b1; ++b) sum += cnt[b];
  const uint64_t incl = wave_incl_scan_u64(sum);
  if (lane_id() == 63) s_w[tid >> 6] = incl;
  __syncthreads();
  uint64_t base = 0;
  for (uint32_t i = 0; i < (tid >> 6); ++i) base += s_w[i];
  uint64_t run = base + incl - sum;
  for (uint32_t b = b0; b < b1; ++b) {
    pre[b] = run;
    run += cnt[b];
  }
}

__device__ inline void grp_scan_body(const Ctx& c, uint32_t jr)
{
  __shared__ uint64_t s_w[4];
  const uint32_t j = c.j0 + jr;
  if (c.st[j].fallback) return;
  block_excl_scan_u64(c.grp_cnt + (uint64_t)j * c.ngrp, c.grp_pre + (uint64_t)j * c.ngrp, c.ngrp, s_w);
}

// Output pass: one wave per kWriteGroups consecutive groups of kGatherSlots
// tiles (their counts and group offsets are loaded together): the tiles'
// candidates in index order, kept ones written to the device's outputs; the
// kept sum of squares of each group goes to epart[j][group]. A tile's values
// and offsets are loaded kWriteBatch windows at a time (positions clamped into
// the tile's candidates); an overflowed tile's entries come from the candidate
// list.
constexpr int kWriteBatch = 8;
constexpr uint32_t kWriteGroups = 1;
constexpr uint32_t kWriteTiles = kWriteGroups * kGatherSlots;
static_assert(kWriteTiles <= 64, "a wave holds its tiles' counts in lanes");

__device__ inline void write_fast_body(const Ctx& c, uint32_t b)
{
  constexpr uint32_t kPerBlock = kWriteGroups * kWaves;
  const uint32_t bpd = (c.ngrp + kPerBlock - 1) / kPerBlock;
  const uint32_t jr = b / bpd;
  const uint32_t j = c.j0 + jr;
  const uint32_t g0 = ((b - jr * bpd) * kWaves + (threadIdx.x >> 6)) * kWriteGroups;
  if (g0 >= c.ngrp) return;
  const uint32_t ng = c.ngrp - g0 < kWriteGroups ? c.ngrp - g0 : kWriteGroups;
  const uint32_t l = lane_id();
  const uint32_t s0 = g0 * kGatherSlots;
  // lane i < kWriteTiles: tile s0 + i's counts (and list offset when it overflowed);
  // lane q < ng: group g0 + q's kept-above | equal << 32 offsets. Loaded before
  // the device's state is known (in bounds for any device).
  const uint32_t sl = s0 + (l < kWriteTiles ? l : 0u);
  const bool live = l < kWriteTiles && sl < c.nslot;
  const uint32_t cnt = live ? c.slot_cnt[(uint64_t)j * c.nslot + sl] : 0u;
  const uint64_t gpre = c.grp_pre[(uint64_t)j * c.ngrp + g0 + (l < ng ? l : 0u)];
  const DevState& st = c.st[j];
  if (st.fallback) return;
  uint32_t thr;
  uint64_t need;
  threshold_of(st, thr, need);
  const DevDesc d = c.desc[j];
  GLOBAL uint32_t* oi = gptr(d.idx_out);
  GLOBAL float* ov = gptr(d.val_out);
  const uint32_t at = ((cnt >> 15) & 1u) ? (uint32_t)slot_pre(c, j, sl) : 0u;
  // 32-bit counts and positions: k < 2^32
  uint32_t run_g = 0, run_e = 0;
  const uint32_t need32 = (uint32_t)need, k32 = d.k;
  double e2 = 0.0;
  // Fused step: the aggregation range markers of the ranges starting in the
  // groups' index span [b0, b1): lb[r] = kept entries with idx < r * kARange,
  // i.e. the output position of the first candidate at or after the range
  // start (or the kept total after the groups). Ranges from rnext on are open.
  GLOBAL uint32_t* lbj = c.lb ? gptr(c.lb) + (uint64_t)j * c.nrange : nullptr;
  const uint64_t vg = (uint64_t)s0 * kTile;
  const uint64_t b0 = vg > d.shift ? vg - d.shift : 0;
  uint64_t b1 = vg + (uint64_t)ng * kGatherSlots * kTile - d.shift;
  if (b1 > c.n) b1 = c.n;
  uint32_t rnext = (uint32_t)((b0 + kARange - 1) / kARange);
  const uint32_t rend = (uint32_t)((b1 + kARange - 1) / kARange);
  auto visit = [&](uint32_t idx, uint32_t vb, bool valid) {
    const uint32_t key = vb & kKeyMask;
    const bool fg = valid && key > thr, fe = valid && key == thr;
    const uint64_t bg = ballot(fg), be = ballot(fe);
    const uint32_t gt_b = run_g + mbcnt(bg), eq_b = run_e + mbcnt(be);
    if (lbj) {
      const uint32_t ri = idx / (uint32_t)kARange;
      const uint32_t rp = __shfl_up(ri, 1, 64);
      const uint64_t vm = ballot(valid);
      if (valid) {
        const uint32_t p = gt_b + (eq_b < need32 ? eq_b : need32);
        for (uint32_t r = (l == 0 ? rnext : rp + 1u); r <= ri; ++r) lbj[r] = p;
      }
      if (vm) rnext = __builtin_amdgcn_readlane(ri, 63 - __builtin_clzll(vm)) + 1u;
    }
    if (fg || (fe && eq_b < need32)) {
      const uint32_t pos = gt_b + (eq_b < need32 ? eq_b : need32);
      const float v = __uint_as_float(vb);
      if (pos < k32) {
        oi[pos] = idx + c.idx_base;
        ov[pos] = v;
      }
      e2 = __builtin_fma((double)v, (double)v, e2);
    }
    run_g += (uint32_t)__builtin_popcountll(bg);
    run_e += (uint32_t)__builtin_popcountll(be);
  };
  // windows e0 .. of a tile's cn entries: ld(e, vb, idx) loads entry e (e < cn)
  auto walk = [&](uint32_t cn, auto ld) {
    for (uint32_t e0 = 0; e0 < cn; e0 += kWriteBatch * 64) {
      uint32_t vb[kWriteBatch], ix[kWriteBatch];
#pragma unroll
      for (int m = 0; m < kWriteBatch; ++m) {
        vb[m] = ix[m] = 0u;
        const uint32_t e = e0 + m * 64 + l;
        if (e0 + m * 64 < cn) ld(e < cn ? e : cn - 1u, vb[m], ix[m]);
      }
#pragma unroll
      for (int m = 0; m < kWriteBatch; ++m)
        if (e0 + m * 64 < cn) visit(ix[m], vb[m], e0 + m * 64 + l < cn);
    }
  };
  for (uint32_t q = 0; q < ng; ++q) {
    run_g = __builtin_amdgcn_readlane((uint32_t)gpre, q);
    run_e = __builtin_amdgcn_readlane((uint32_t)(gpre >> 32), q);
    for (uint32_t i = q * kGatherSlots; i < (q + 1) * kGatherSlots; ++i) {
      const uint32_t ci = __builtin_amdgcn_readlane(cnt, i);
      const uint32_t cn = ci & 0x7FFFu;
      if (cn == 0) continue;
      const uint32_t s = s0 + i;
      if (!((ci >> 15) & 1u)) {
        const GLOBAL uint32_t* reg = gptr(c.slot) + ((uint64_t)j * c.nslot + s) * kSlotWords;
        const GLOBAL uint16_t* r16 = reinterpret_cast<const GLOBAL uint16_t*>(reg);
        const GLOBAL uint32_t* vals = reg + (cn - (ci >> 16));     // after the selection keys
        const uint32_t ibase = (uint32_t)((uint64_t)s * kTile - d.shift);
        walk(cn, [&](uint32_t e, uint32_t& vb, uint32_t& ix) {
          vb = vals[e];
          ix = ibase + r16[slot_off16_at(e)];
        });
      } else {
        const uint64_t o = d.cand_off + __builtin_amdgcn_readlane(at, i);
        const GLOBAL uint32_t* cidx = gptr(c.cand_idx) + o;
        const GLOBAL uint32_t* cval = reinterpret_cast<const GLOBAL uint32_t*>(gptr(c.cand_val) + o);
        walk(cn, [&](uint32_t e, uint32_t& vb, uint32_t& ix) {
          vb = cval[e];
          ix = cidx[e];
        });
      }
    }
    const double es = wave_sum_f64(e2);
    if (l == 0) c.epart[(uint64_t)j * c.nslot + g0 + q] = es;
    e2 = 0.0;
  }
  if (lbj) {
    const uint32_t p = run_g + (run_e < need32 ? run_e : need32);
    for (uint32_t r = rnext + l; r < rend; r += 64) lbj[r] = p;
  }
}

// ---- 6. ordered compaction of the exact path ------------------------------------------------
// Blocks are kCBlk positions of a device's candidate list (fast path) or of its
// gradient's virtual row (exact path), in index order. Counting uses rank keys
// (key + 1, pads 0) against thr + 1, so pads are never above or equal to it.
// Per block: counts of keys above the threshold (gt) and equal to it (eq).
template <int R>
__device__ inline uint64_t block_gt_eq(const Row& row, uint64_t vbase, uint32_t thr, uint32_t* lds)
{
  const uint32_t w = threadIdx.x >> 6, l = lane_id();
  const uint32_t thr1 = thr + 1u;
  uint32_t gt = 0, eq = 0;
#pragma unroll 4
  for (int r = 0; r < R; ++r) {
    const f4 x = load4(row, vbase + elem_of<R>(w, r, l), false);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t key1 = rank_key(x[q]);
      gt += (key1 > thr1) ? 1u : 0u;
      eq += (key1 == thr1) ? 1u : 0u;
    }
  }
  uint32_t tg, te;
  wave_prefix_of_block(gt, lds, tg);
  wave_prefix_of_block(eq, lds, te);
  return (uint64_t)tg | ((uint64_t)te << 32);
}

__device__ inline void count_cf_body(const Ctx& c, uint32_t worker, uint32_t workers)
{
  __shared__ uint32_t lds[8];
  if (*c.fb_count == 0u) return;
  // (device, block) items of the group, grid-stride (see k_hist_cf)
  const uint64_t items = (uint64_t)c.jn * c.nfb;
  for (uint64_t it = worker; it < items; it += workers) {
    const uint32_t jr = (uint32_t)(it / c.nfb), blk = (uint32_t)(it - (uint64_t)jr * c.nfb);
    const uint32_t j = c.j0 + jr;
    const DevState& s = c.st[j];
    if (!s.fallback) continue;
    uint32_t thr;
    uint64_t need;
    threshold_of(s, thr, need);
    const Row row{gptr(c.desc[j].grad), c.desc[j].shift, c.n};
    const uint64_t r = block_gt_eq<kCBlkRounds>(row, (uint64_t)blk * kCBlk, thr, lds);
    if (threadIdx.x == 0) c.blk_cnt[(uint64_t)j * c.nbmax + blk] = r;
  }
}

// Exclusive prefix of the packed block counts of one exact-path device.
__device__ inline void scan_cf_body(const Ctx& c, uint32_t jr)
{
  __shared__ uint64_t s_w[4];
  const uint32_t j = c.j0 + jr;
  if (!c.st[j].fallback) return;
  block_excl_scan_u64(c.blk_cnt + (uint64_t)j * c.nbmax, c.blk_pre + (uint64_t)j * c.nbmax, c.nfb, s_w);
}

// Writes the kept entries of one block in index order.
//   kept: key > thr, or key == thr with fewer than `need` equal keys before it;
//   position: (keys > thr before it) + min(equal keys before it, need).
// An element's index is its virtual position minus the row's shift, plus
// `base` (the offset of a layer selected on its own).
__device__ inline uint32_t write_count(const f4& x, uint32_t thr1)
{
  uint32_t cnt = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t key1 = rank_key(x[q]);
    cnt += (key1 > thr1) ? 1u : 0u;
    cnt += (key1 == thr1) ? 0x10000u : 0u;
  }
  return cnt;
}

// One round of the ordered write: the wave's elements above the threshold, and
// equal ones while fewer than `need` came before, at their kept positions.
__device__ inline void write_round(const f4& x, uint64_t e, uint64_t vbase, const Row& row, uint32_t base,
                                   uint32_t thr1, uint64_t need, uint32_t k, GLOBAL uint32_t* out_idx, GLOBAL float* out_val,
                                   uint64_t& run_g, uint64_t& run_e, double& e2)
{
  bool fg[4], fe[4];
  uint64_t bg[4], be[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t key1 = rank_key(x[q]);
    fg[q] = key1 > thr1;
    fe[q] = key1 == thr1;
    bg[q] = ballot(fg[q]);
    be[q] = ballot(fe[q]);
  }
  if ((bg[0] | bg[1] | bg[2] | bg[3] | be[0] | be[1] | be[2] | be[3]) == 0ull) return;
  uint64_t gt_b = run_g + mbcnt(bg[0]) + mbcnt(bg[1]) + mbcnt(bg[2]) + mbcnt(bg[3]);
  uint64_t eq_b = run_e + mbcnt(be[0]) + mbcnt(be[1]) + mbcnt(be[2]) + mbcnt(be[3]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool keep = fg[q] || (fe[q] && eq_b < need);
    if (keep) {
      const uint64_t pos = gt_b + (eq_b < need ? eq_b : need);
      const float val = x[q];
      if (pos < k) {
        out_idx[pos] = (uint32_t)(vbase + e + q - row.shift) + base;
        out_val[pos] = val;
      }
      e2 = __builtin_fma((double)val, (double)val, e2);
    }
    gt_b += fg[q];
    eq_b += fe[q];
  }
  run_g += __builtin_popcountll(bg[0]) + __builtin_popcountll(bg[1]) + __builtin_popcountll(bg[2]) +
           __builtin_popcountll(bg[3]);
  run_e += __builtin_popcountll(be[0]) + __builtin_popcountll(be[1]) + __builtin_popcountll(be[2]) +
           __builtin_popcountll(be[3]);
}

// Writes the kept entries of one block in index order.
//   kept: key > thr, or key == thr with fewer than `need` equal keys before it;
//   position: (keys > thr before it) + min(equal keys before it, need).
// An element's index is its virtual position minus the row's shift, plus
// `base` (the offset of a layer selected on its own).
template <int R>
__device__ inline double block_write(const Row& row, uint64_t vbase, uint32_t base, uint32_t thr,
                                     uint64_t need, uint64_t pre, uint32_t k, GLOBAL uint32_t* out_idx, GLOBAL float* out_val,
                                     uint32_t* lds)
{
  const uint32_t w = threadIdx.x >> 6, l = lane_id();
  const uint32_t thr1 = thr + 1u;
  const bool full = vbase >= row.shift && vbase + R * kRound <= row.shift + row.n;
  f4 x[R];
  uint32_t cnt = 0;
  if (full) {
    const GLOBAL float* p = row.p + (vbase - row.shift);
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = ld4(p + elem_of<R>(w, r, l));
#pragma unroll
    for (int r = 0; r < R; ++r) cnt += write_count(x[r], thr1);
  } else {
    for (int r = 0; r < R; ++r) cnt += write_count(load4(row, vbase + elem_of<R>(w, r, l), false), thr1);
  }
  uint32_t tot;
  const uint32_t wex = wave_prefix_of_block(cnt, lds, tot);
  uint64_t run_g = (pre & 0xFFFFFFFFull) + (wex & 0xFFFFu);
  uint64_t run_e = (pre >> 32) + (wex >> 16);
  double e2 = 0.0;
  if (full) {
#pragma unroll
    for (int r = 0; r < R; ++r)
      write_round(x[r], elem_of<R>(w, r, l), vbase, row, base, thr1, need, k, out_idx, out_val, run_g, run_e, e2);
  } else {
    for (int r = 0; r < R; ++r) {
      const uint64_t e = elem_of<R>(w, r, l);
      write_round(load4(row, vbase + e, false), e, vbase, row, base, thr1, need, k, out_idx, out_val, run_g,
                  run_e, e2);
    }
  }
  return e2;
}

__device__ inline void write_cf_body(const Ctx& c, uint32_t worker, uint32_t workers)
{
  __shared__ uint32_t lds[8];
  __shared__ double s_e[4];
  if (*c.fb_count == 0u) return;
  // (device, block) items of the group, grid-stride (see k_hist_cf)
  const uint64_t items = (uint64_t)c.jn * c.nfb;
  for (uint64_t it = worker; it < items; it += workers) {
    const uint32_t jr = (uint32_t)(it / c.nfb), blk = (uint32_t)(it - (uint64_t)jr * c.nfb);
    const uint32_t j = c.j0 + jr;
    const DevState& s = c.st[j];
    if (!s.fallback) continue;
    uint32_t thr;
    uint64_t need;
    threshold_of(s, thr, need);
    const DevDesc d = c.desc[j];
    const Row row{gptr(d.grad), d.shift, c.n};
    const double e2 = block_write<kCBlkRounds>(row, (uint64_t)blk * kCBlk, c.idx_base, thr, need,
                                               c.blk_pre[(uint64_t)j * c.nbmax + blk], d.k, gptr(d.idx_out),
                                               gptr(d.val_out), lds);
    const double es = block_sum_f64(e2, s_e);
    if (threadIdx.x == 0) c.blk_e[(uint64_t)j * c.nbmax + blk] = es;
    __syncthreads();
  }
}

// ---- 7. energies of the adaptive rule and per-device decision --------------------------------
// §IV: send Top-k(g) when | ||g||^2 - ||Top-k(g)||^2 | / ||g||^2 <= delta.
__device__ inline void final_body(const Ctx& c, uint32_t jr)
{
  __shared__ double s_e[4];
  const uint32_t j = c.j0 + jr;
  DevState& s = c.st[j];
  const bool fast = !s.fallback;
  const uint32_t nb = fast ? c.ngrp : c.nfb;
  const double* ep = fast ? c.epart + (uint64_t)j * c.nslot : c.blk_e + (uint64_t)j * c.nbmax;
  const uint64_t* pre = fast ? c.grp_pre + (uint64_t)j * c.ngrp : c.blk_pre + (uint64_t)j * c.nbmax;
  const uint64_t* cnt = fast ? c.grp_cnt + (uint64_t)j * c.ngrp : c.blk_cnt + (uint64_t)j * c.nbmax;
  double acc = 0.0;
  for (uint32_t b = threadIdx.x; b < nb; b += kBlock) acc += ep[b];
  const double e_kept = block_sum_f64(acc, s_e);
  if (threadIdx.x != 0) return;
  uint32_t thr;
  uint64_t need;
  if (!threshold_of(s, thr, need)) s.err |= kErrNoThreshold;
  const uint64_t tot = pre[nb - 1] + cnt[nb - 1];
  s.thr = thr;
  s.c_gt = tot & 0xFFFFFFFFull;
  s.need = need;
  if (s.c_gt + need != c.desc[j].k || (c.inject_count_error && j == 0)) s.err |= kErrCount;
  if (c.err_acc && (s.err & kErrFatal)) atomicOr(c.err_acc + j, s.err & kErrFatal);
  s.e_kept = e_kept;
  // §IV: the rule compares the energies, optionally their moving averages
  s.sparse = adaptive_rule(s.e_all, e_kept, c.ewma ? c.ewma + 2 * (uint64_t)j : nullptr, c.ewma_beta, c.delta);
  if (c.counters) account(c.counters + 3 * (uint64_t)j, s.sparse, c.desc[j].k, c.n);
  if (c.energies_out) {
    c.energies_out[(uint64_t)c.e_stride * j] = s.e_all;
    c.energies_out[(uint64_t)c.e_stride * j + 1] = e_kept;
  }
  if (c.compressed_out) c.compressed_out[j] = (uint8_t)s.sparse;
}

// ---- merged launches ------------------------------------------------------------------------
// Each launch of the rest of the selection serves both paths: the fast-path
// blocks first, then the exact path's workers (which return at once when no
// device fell back). In the fused step the output pass of a fast device also
// writes its aggregation range markers; the decision launch's extra blocks
// build those of exact-path devices.
template <int kBT>
__global__ __launch_bounds__(kBlock) void k_count(Ctx c, uint32_t nfast)
{
  if (blockIdx.x < nfast) grp_count_body<kBT>(c, blockIdx.x);
  else count_cf_body(c, blockIdx.x - nfast, gridDim.x - nfast);
}

__global__ __launch_bounds__(kBlock) void k_offsets(Ctx c, uint32_t fast)
{
  if (fast && blockIdx.x < c.jn) grp_scan_body(c, blockIdx.x);
  else scan_cf_body(c, blockIdx.x - (fast ? c.jn : 0u));
}

__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(8, 8))) void k_write(Ctx c)
{
  write_fast_body(c, blockIdx.x);
}

// The exact path's output pass has a launch of its own: it needs about twice
// the registers of the fast one.
__global__ __launch_bounds__(kBlock) void k_write_cf(Ctx c)
{
  write_cf_body(c, blockIdx.x, gridDim.x);
}

__global__ __launch_bounds__(kBlock) void k_final(Ctx c, uint32_t lb_blocks)
{
  if (blockIdx.x < c.jn) {
    final_body(c, blockIdx.x);
    return;
  }
  if (*c.fb_count == 0u) return;
  const uint32_t b = blockIdx.x - c.jn;
  const uint32_t j = c.j0 + b / lb_blocks;
  if (!c.st[j].fallback) return;
  const DevDesc& d = c.desc[j];
  lb_ranges(d.idx_out, d.k, c.lb + (uint64_t)j * c.nrange, c.nrange, (b % lb_blocks) * kBlock + threadIdx.x,
            lb_blocks * kBlock);
}

// ---- host-side launchers ---------------------------------------------------------------------
// Everything after the main pass for devices [c.j0, c.j0 + c.jn), on stream s,
// in two halves: 0, the threshold (scans, path decision, overflowed tiles,
// radix passes, group counts and offsets), latency-bound and light on memory;
// 1, the output (ordered compaction with the range markers, energies and decision),
// which moves most of the bytes.
// Tiles per wave of the walks over the tiles' selection-interval keys (the
// first radix pass and the group counts): the most, up to 16, that still
// give 6000 waves over the devices of the launch, else 4. Few tiles per wave
// keep small launches wide; many keep large ones from flushing a histogram
// per few tiles (16 / 8 / 4: 3.83 / 3.84 / 3.89 ms per step at 32 x 143.7M,
// 0.737 / 0.707 / 0.692 at 16 x 25.6M, 0.276 / 0.263 / 0.256 at 8 x 11.2M).
// Beside another launch's main pass (a layer of the per-layer selection)
// always 16: fewer workgroups wait less for the slots that pass leaves.
static int band_tiles_per_wave(const Ctx& c, const SelectPlan& p)
{
  if (p.beside) return 16;
  const uint64_t tiles = (uint64_t)c.jn * c.nslot;
  if (tiles / 16 >= 6000) return 16;
  if (tiles / 8 >= 6000) return 8;
  return 4;
}

template <int kBT>
static void launch_band_passes(const Ctx& c, const SelectPlan& p, hipStream_t s)
{
  const uint32_t ncand = p.any_fast ? c.jn * ((c.nslot + kBT * kWaves - 1) / (kBT * kWaves)) : 0u;
  for (int pass = 0; pass < 3; ++pass) {
    k_hist_cf<kBT><<<ncand + p.full_workers, kBlock, 0, s>>>(c, ncand, (uint32_t)pass);
    k_find<<<c.jn, 64, 0, s>>>(c, kSlotCand, kSlotFull + 1, 0);
  }
  k_count<kBT><<<ncand + p.full_workers, kBlock, 0, s>>>(c, ncand);
}

static void launch_post(const Ctx& c, const SelectPlan& p, hipStream_t s, int half)
{
  if (half == 0) {
    if (p.beside) k_scan<kScanBlockSmall><<<c.jn, kScanBlockSmall, 0, s>>>(c);
    else k_scan<kScanBlockLarge><<<c.jn, kScanBlockLarge, 0, s>>>(c);
    if (p.any_fast) k_overflow<<<c.jn * kOverflowBlocks, kBlock, 0, s>>>(c, kOverflowBlocks);
    switch (band_tiles_per_wave(c, p)) {
      case 16: launch_band_passes<16>(c, p, s); break;
      case 8: launch_band_passes<8>(c, p, s); break;
      default: launch_band_passes<4>(c, p, s); break;
    }
    k_offsets<<<(p.any_fast ? 2 : 1) * c.jn, kBlock, 0, s>>>(c, p.any_fast);
    return;
  }
  if (p.any_fast) k_write<<<c.jn * ((c.ngrp + kWriteGroups * kWaves - 1) / (kWriteGroups * kWaves)), kBlock, 0, s>>>(c);
  k_write_cf<<<p.full_workers, kBlock, 0, s>>>(c);
  uint32_t lbb = 0;
  if (c.lb) {
    lbb = (c.nrange + kBlock - 1) / kBlock;
    if (lbb > 64) lbb = 64;
  }
  k_final<<<c.jn * (1 + lbb), kBlock, 0, s>>>(c, lbb);
}

// The whole selection. The devices are split into p.parts groups whose main
// passes run one after the other on s. A main pass is bound by HBM bandwidth,
// the threshold half of the rest of a group's selection by latency: that half
// of group i runs on s2 while the main pass of group i + 1 runs on s, and the
// output half of group i, which moves more bytes, only once that main pass is
// done (the last group's rest runs on s); s waits for s2 at the end.
// done[i] (events of s2's owner) mark the end of main pass i. Profiling events
// (ev, optional; as few as possible, each costs a few microseconds of queue
// time): 0 start, 1 bracket done, 3 + 2i the end of main pass i (main pass i
// starts at the end of the previous one; with profiling these also serve as
// done[i]), 2 + 2 * parts all done.
hipError_t launch_select(const Ctx& c0, const PrepArgs& a, const SelectPlan& p, hipStream_t s, hipStream_t s2,
                         hipEvent_t* done, hipEvent_t join, hipEvent_t* ev)
{
  Ctx c = c0;
  c.j0 = 0;
  c.jn = c.K;
  const uint64_t zero_words = (uint64_t)c.K * kSlots * kBins;
  uint32_t gprep = (uint32_t)((zero_words + kBlock * 8 - 1) / (kBlock * 8));
  gprep = gprep < 1 ? 1 : (gprep > 2048 ? 2048 : gprep);
  k_prep<<<gprep, kBlock, 0, s>>>(c, a);
  if (p.any_fast) {
    for (int pass = 0; pass < kBracketPasses; ++pass) {
      k_hist_sample<<<dim3(p.sample_blocks, c.K), kBlock, 0, s>>>(c);
      k_find<<<c.K, 64, 0, s>>>(c, kSlotSampleLo, kSlotSampleHi + 1, pass + 1 == kBracketPasses);
    }
  }
  if (ev) (void)hipEventRecord(ev[1], s);
  GradArgs ga;
  for (uint32_t j = 0; j < c.K; ++j) ga.grad[j] = a.grad[j];
  const uint32_t parts = p.parts;
  auto group = [&](uint32_t i) {
    Ctx ci = c;
    ci.j0 = c.K * i / parts;
    ci.jn = c.K * (i + 1) / parts - ci.j0;
    return ci;
  };
  for (uint32_t i = 0; i < parts; ++i) {
    const Ctx ci = group(i);
    k_main<<<ci.jn * c.tpd, kBlock, 0, s>>>(ci, ga);
    hipEvent_t de = ev ? ev[3 + 2 * i] : (parts > 1 ? done[i] : nullptr);
    if (de) {
      hipError_t e = hipEventRecord(de, s);
      if (e == hipSuccess && parts > 1) e = hipStreamWaitEvent(s2, de, 0);
      if (e != hipSuccess) return e;
    }
    if (i > 0) launch_post(group(i - 1), p, s2, 1);
    if (i + 1 < parts) {
      launch_post(ci, p, s2, 0);
    } else {
      launch_post(ci, p, s, 0);
      launch_post(ci, p, s, 1);
    }
  }
  if (parts > 1) {
    hipError_t e = hipEventRecord(join, s2);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, join, 0);
    if (e != hipSuccess) return e;
  }
  if (ev) (void)hipEventRecord(ev[2 + 2 * parts], s);
  return hipGetLastError();
}

// The selection of all devices in three parts, for callers that pipeline
// several selections on alternating workspaces (the long layers of a
// per-layer selection): preparation and bracket; the main pass; everything
// after it. The caller orders them and the workspace reuse with events.
hipError_t launch_bracket(const Ctx& c0, const PrepArgs& a, const SelectPlan& p, hipStream_t s)
{
  Ctx c = c0;
  c.j0 = 0;
  c.jn = c.K;
  const uint64_t zero_words = (uint64_t)c.K * kSlots * kBins;
  uint32_t gprep = (uint32_t)((zero_words + kBlock * 8 - 1) / (kBlock * 8));
  gprep = gprep < 1 ? 1 : (gprep > 2048 ? 2048 : gprep);
  k_prep<<<gprep, kBlock, 0, s>>>(c, a);
  if (p.any_fast) {
    for (int pass = 0; pass < kBracketPasses; ++pass) {
      k_hist_sample<<<dim3(p.sample_blocks, c.K), kBlock, 0, s>>>(c);
      k_find<<<c.K, 64, 0, s>>>(c, kSlotSampleLo, kSlotSampleHi + 1, pass + 1 == kBracketPasses);
    }
  }
  return hipGetLastError();
}

hipError_t launch_main(const Ctx& c0, const PrepArgs& a, hipStream_t s)
{
  Ctx c = c0;
  c.j0 = 0;
  c.jn = c.K;
  GradArgs ga;
  for (uint32_t j = 0; j < c.K; ++j) ga.grad[j] = a.grad[j];
  k_main<<<c.K * c.tpd, kBlock, 0, s>>>(c, ga);
  return hipGetLastError();
}

hipError_t launch_rest(const Ctx& c0, const SelectPlan& p, hipStream_t s)
{
  Ctx c = c0;
  c.j0 = 0;
  c.jn = c.K;
  launch_post(c, p, s, 0);
  launch_post(c, p, s, 1);
  return hipGetLastError();
}

}  // namespace scadles
