// scadles_internal.h -- device-side structures, constants and primitives of the
// ScaDLES hot-path kernels for gfx950 (CDNA4, wave64). Internal to libscadles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scadles {

// ---- launch geometry --------------------------------------------------------------------
constexpr int kBlock = 256;            // threads per workgroup (4 wave64)
constexpr int kWaves = kBlock / 64;
constexpr int kRound = kBlock * 4;     // elements per "round": one float4 per thread
constexpr int kTile = 16384;           // main select pass: elements per workgroup (64 KiB)
constexpr int kTileRounds = kTile / kRound;
constexpr int kCBlk = 8192;            // candidate blocks (hist/compaction over candidates)
constexpr int kCBlkRounds = kCBlk / kRound;
constexpr int kSBlk = 4096;            // sample elements per workgroup
constexpr int kSChunk = 256;           // contiguous sample chunk (1 KiB)
constexpr int kBins = 2048;            // radix digit: 11 bits
constexpr int kDigitBits = 11;
constexpr int kARange = 2048;          // aggregation: positions per wave (16 KiB of doubles in LDS)
constexpr int kABatch = 8;             // aggregation: devices whose entries are loaded together
constexpr int kMaxK = 64;              // SCADLES_MAX_DEVICES
constexpr int kSlots = 4;              // selection slots per device
constexpr int kSlotSampleLo = 0, kSlotSampleHi = 1, kSlotCand = 2, kSlotFull = 3;
constexpr uint32_t kKeyInf = 0x80000000u;   // above every 31-bit key
constexpr uint32_t kKeyMask = 0x7FFFFFFFu;
constexpr uint64_t kSat31 = 0x7FFFFFFFull;
constexpr int kFullWorkers = 1024;     // grid of the grid-stride exact-path kernels
constexpr int kWaveCap = 512;          // main pass: candidates one wave chunk (4096 elements) can stage
constexpr int kSlotWords = 1024;       // 32-bit words of one tile's slot region (4 KiB)
constexpr int kGatherSlots = 2;        // tiles per wave in the selection-list and output passes
constexpr int kOverflowBlocks = 128;   // workgroups per device re-scanning overflowed tiles

enum : uint32_t { kModeFast = 0, kModeExact = 1 };

// DevState::err bits. A bracket miss only sends the device to the exact path;
// the others mean its output is wrong and are reported in validation mode.
enum : uint32_t {
  kErrBracket = 2u,       // a sample selection of the bracket missed (recovered by the exact path)
  kErrSelect = 4u,        // a radix pass of the threshold selection missed
  kErrNoThreshold = 8u,   // the threshold selection did not finish
  kErrCount = 16u,        // keys above the threshold + ties kept != k
};
constexpr uint32_t kErrFatal = kErrSelect | kErrNoThreshold | kErrCount;

// ---- workspace structures ---------------------------------------------------------------
struct DevDesc {          // per device, written once per call by the prep kernel
  const float* grad;
  uint32_t* idx_out;
  float* val_out;
  uint64_t cand_off;      // first element of the device's candidate region
  uint32_t k;
  uint32_t cap;           // candidate capacity (0 in exact mode)
  uint32_t mode;
  uint32_t r_lo;          // sample ranks that bracket the k-th largest key
  uint32_t r_hi;          // 0: no upper bracket
  uint32_t shift;         // (grad address / 4) % 4: offset of element 0 in its 16-byte word
};

// State of one radix selection: the key of 1-based descending rank `rank` among
// the keys in [lo, hi) of some population, decided 11 bits at a time on the
// offset (key - lo), most significant first.
struct Sel {
  uint32_t active;        // a histogram pass is pending
  uint32_t found;         // finished: result holds the key
  uint32_t lo, hi;        // band [lo, hi)
  uint32_t bits;          // low bits of (key - lo) still undecided
  uint32_t prefix;        // decided high bits of (key - lo)
  uint32_t result;
  uint32_t pad;
  uint64_t rank;          // rank still sought among keys matching the prefix
  uint64_t above;         // band keys above the prefix range seen so far
};

struct DevState {
  Sel sel[kSlots];
  uint64_t cand, sure;    // main pass totals: keys >= t_lo, keys >= t_hi
  uint32_t t_lo, t_hi;    // bracket used by the main pass
  uint32_t fallback;      // 1: the exact full-data path produces this device's output
  uint32_t thr;           // final threshold key (k-th largest)
  uint32_t err;           // internal error bits, kErr*
  uint64_t c_gt, need;    // keys above thr; keys equal to thr that are kept
  double e_all, e_kept;
  uint32_t sparse;        // 1: the device sends Top-k (adaptive rule), 0: dense
  uint32_t ovf_n;         // entries in the device's ovf_list
};

// Kernel context: where everything lives in the workspace, plus call scalars.
struct Ctx {
  DevDesc* desc;
  DevState* st;
  uint32_t* hist;         // [K][kSlots][kBins]
  uint32_t* slot_cnt;     // [K][nslot] per tile: candidates | overflowed << 15 | sure << 16
  uint64_t* slot_off;     // [K][nslot] candidate | sure << 32 counts of the device's tiles before each tile
  uint32_t* slot;         // [K][nslot][kSlotWords] per tile: candidates' value bits, then the keys of those
                          // below t_hi; from the top down, the candidates' 16-bit offsets in the tile
  uint32_t* ovf_list;     // [K][nslot] tiles with a wave chunk of more than kWaveCap candidates
  double* epart;          // [K][nslot] sum of squares per tile, later kept sum of squares per write group
  uint32_t* cand_idx;     // candidate regions (entries of overflowed slots only)
  float* cand_val;
  uint32_t* band;         // band lists: keys below t_hi of overflowed tiles, per device at cand_off
  uint64_t* grp_cnt;      // [K][ngrp] kept-above | equal << 32 counts per write group of slots
  uint64_t* grp_pre;      // [K][ngrp] exclusive prefix of grp_cnt
  uint64_t* blk_cnt;      // [K][nbmax] packed (gt | eq << 32) per compaction block
  uint64_t* blk_pre;      // [K][nbmax] exclusive prefix of blk_cnt
  double* blk_e;          // [K][nbmax] kept sum of squares per compaction block
  double* energies_out;   // caller's (dev, 2K) or null
  uint8_t* compressed_out;// caller's (dev, K) or null
  uint64_t n;
  uint32_t K;
  uint32_t tpd;           // main tiles per device: ceil((n + 3) / kTile)
  uint32_t nslot;         // slots (main-pass tiles) per device: tpd
  uint32_t ngrp;          // write groups per device: ceil(nslot / kGatherSlots)
  uint32_t nfb;           // exact-path blocks per device: ceil((n + 3) / kCBlk)
  uint32_t nbmax;         // exact-path blocks allocated per device (nfb)
  uint32_t s_stride;      // sample chunk stride (elements)
  uint32_t s_n;           // sample elements per device
  uint32_t force_fallback;
  uint32_t inject_count_error;   // testing: device 0 reports kErrCount
  uint32_t j0, jn;        // devices [j0, j0 + jn) of this launch (the per-device kernels)
  uint32_t* fb_count;     // devices on the exact path (the exact-path kernels exit early at 0)
  uint32_t* lb;           // fused step: aggregation range markers (see AggCtx), else null
  uint32_t nrange;
  double* ewma;           // [K][2] moving averages of E_all, E_kept (adaptive rule), or null
  double ewma_beta;
  uint64_t* counters;     // [K][3] iterations compressed, iterations, floats sent; or null
  uint32_t idx_base;      // added to every output index (a layer's offset in the gradient)
  uint32_t e_stride;      // doubles between devices' energy pairs in energies_out (2: packed)
  uint32_t* err_acc;      // [K] fatal error bits of every selection of a call ORed together, or null
  double delta;
};

// Per-call parameters that only the prep kernel needs (passed by value).
struct PrepArgs {
  const float* grad[kMaxK];
  uint32_t* idx[kMaxK];
  float* val[kMaxK];
  uint32_t k[kMaxK];
  uint32_t cap[kMaxK];
  uint32_t mode[kMaxK];
  uint32_t r_lo[kMaxK];
  uint32_t r_hi[kMaxK];
};

// Gradient pointers of the main pass, passed as kernel arguments.
struct GradArgs {
  const float* grad[kMaxK];
};

// Aggregation context.
struct AggArgs {
  const uint32_t* idx[kMaxK];   // sparse sets (null: dense)
  const float* val[kMaxK];
  const float* dense[kMaxK];    // dense gradient used when the device is dense
  uint32_t k[kMaxK];
  float w[kMaxK];
};

struct AggCtx {
  const DevState* st;     // fused path: per-device sparse/dense decision; null otherwise
  uint32_t* lb;           // [K][nrange] entries of each device with idx below the range's start; the
                          // entries of range r are [lb[r], lb[r + 1]) (lb[nrange] taken as k)
  uint32_t* err;          // validation flag
  float* out;             // dense aggregate
  float* params;          // null: no SGD
  float* mbuf;            // not null: momentum SGD with weight decay (momentum buffer), else Eqn 4c
  float lr;
  float mom, wd;
  uint32_t K;
  uint32_t nrange;        // ceil(n / kARange): waves of the aggregation kernel
  uint32_t kmax;
  uint64_t n;
};

// Launch plan of the selection pipeline (host side).
constexpr uint32_t kMaxParts = 4;      // device groups whose main passes are pipelined
struct SelectPlan {
  uint32_t any_fast;          // some device takes the sampled single-read path
  uint32_t sample_blocks;     // sample workgroups per device
  uint32_t full_workers;      // grid-stride workgroups of the exact full-data path
  uint32_t parts;             // device groups, 1 .. kMaxParts
  uint32_t beside;            // the rest runs beside other selections' main passes (small workgroups)
};

// Launchers (select.hip, aggregate.hip). done[parts] and join are events of
// the caller's second stream s2; `ev`, when not null, receives the profiling
// events described at launch_select.
hipError_t launch_select(const Ctx& c, const PrepArgs& a, const SelectPlan& p, hipStream_t s, hipStream_t s2,
                         hipEvent_t* done, hipEvent_t join, hipEvent_t* ev);
// All devices in one group, in three parts on streams of the caller's choice:
// preparation and bracket, the main pass, the rest (see select.hip).
hipError_t launch_bracket(const Ctx& c, const PrepArgs& a, const SelectPlan& p, hipStream_t s);
hipError_t launch_main(const Ctx& c, const PrepArgs& a, hipStream_t s);
hipError_t launch_rest(const Ctx& c, const SelectPlan& p, hipStream_t s);
hipError_t launch_aggregate(const AggArgs& a, const AggCtx& c, uint32_t validate, bool marks_done, hipStream_t s);
hipError_t launch_marks(const AggArgs& a, const AggCtx& c, hipStream_t s);
hipError_t launch_marks_built(const AggArgs& a, const AggCtx& c, hipStream_t s);
hipError_t launch_sgd(float* p, const float* g, uint64_t n, float lr, hipStream_t s);
hipError_t launch_momentum_sgd(float* p, float* v, const float* g, uint64_t n, float lr, float mom, float wd,
                               hipStream_t s);

// Momentum SGD with weight decay on one element: every product of two floats is
// exact in double, each step rounds once in double, and the stored buffer is
// the value the parameter update uses.
__device__ inline void momentum_step(float& p, float& v, float g, double nlr, double mom, double wd)
{
  const double d = __builtin_fma(wd, (double)p, (double)g);
  v = (float)__builtin_fma(mom, (double)v, d);
  p = (float)__builtin_fma(nlr, (double)v, (double)p);
}

// ---- per-layer selection of short layers: one workgroup per (device, layer) row ------
// Layers of at most RowsCtx::row_max elements are selected by k_rows, one
// workgroup of kRowBlock threads per row, instead of running the multi-launch
// selection once per layer.
constexpr int kRowBlock = 1024;
constexpr int kRowCand = 14336;        // keys of the threshold bin held in LDS
constexpr int kPutWords = 240;         // table words per k_put launch (kernel-argument copy)

struct RowDesc {
  const float* grad;     // the layer's first element
  uint32_t* idx_out;     // the row's first output
  float* val_out;
  uint32_t n, k;
  uint32_t base;         // index of the layer's first element in the whole gradient
  uint32_t eslot;        // j * L + l: where the row's energies go
};

struct RowsPrep {
  const float* grad[kMaxK];
  uint32_t* idx[kMaxK];
  float* val[kMaxK];
  double ratio[kMaxK];
};

// Rows of more than the option "row_split" elements are split into parts of
// kRowPartLen elements, each read by its own workgroup (k_big_* kernels), so
// that one long row does not keep a single compute unit busy while the rest of
// the GPU idles. A part is kRowPartChunks chunks of kRowChunkLen elements; a
// chunk is what one wave reads at once.
constexpr uint32_t kRowChunkLen = 2048;
constexpr uint32_t kRowPartChunks = 8;
constexpr uint64_t kRowPartLen = (uint64_t)kRowChunkLen * kRowPartChunks;
constexpr uint32_t kRowPartWaves = 4;       // waves of a part workgroup
constexpr uint64_t kRowWaveLen = kRowPartLen / kRowPartWaves;   // elements of one wave in a part
constexpr uint64_t kRowSplitMin = 65536;   // smallest row that may be split
constexpr uint64_t kRowSplitMax = 1u << 24; // longest row that may be split
constexpr uint32_t kChunkWords = 4;         // words of a chunk's record

// Per split row: its bracket, whether some wave's candidates overflowed their
// region, and the outcome of its threshold selection.
struct BigRowState {
  uint32_t t_lo, t_hi;    // bracket of the sampled selection
  uint32_t ovf;           // nonzero: a wave had more candidates than its region holds
  uint32_t slow;          // 1: the select kernel wrote the row on its own (bracket missed or ovf)
  uint32_t thr;           // threshold key and the number of keys equal to it that are kept
  uint32_t need;
  uint32_t pad[2];
};

struct RowsCtx {
  const uint64_t* table;  // seg_off[0..L], then per layer its position among the short layers (or ~0),
                          // then part_pre[0..Lb], then cand_pre[0..Lb]
  RowDesc* rows;          // [Ls x K]: row q * K + j is device j's q-th short layer (longest first)
  double* row_e;          // [K x L x 2]: E_all, E_kept of device j's layer l
  uint32_t K, L, Ls;
  // Split rows: the first Lb short layers (the longest). Part p of device j's
  // row of split layer q is workgroup part_pre[q] * K + j * (part_pre[q + 1] -
  // part_pre[q]) + p of the part kernels; its chunks are kRowPartChunks
  // records of `chunk` from that number times kRowPartChunks on. The row's
  // candidates are staged from cand_pre[q] * K + j * (cand_pre[q + 1] -
  // cand_pre[q]) of `cand` on, in a region of equal size per wave of its parts.
  uint32_t Lb;
  uint32_t nparts;        // part workgroups of all split rows
  BigRowState* bst;       // [Lb x K]
  uint32_t* chunk;        // [nparts x kRowPartChunks x kChunkWords]: per chunk, keys >= t_hi, 0, where
                          // its candidates start in the row's region, their number; after the
                          // selection the first two are the kept entries above / equal to the
                          // threshold before the chunk
  uint64_t* cand;         // staged candidates: index | value bits << 32, in index order per chunk
  double* part_e;         // [2 x nparts x 4] E_all, then E_kept, partial sums per wave of each part
};

hipError_t launch_put_table(const uint64_t* src, uint64_t count, uint64_t* dst, hipStream_t s);

// Decision of the per-layer fused step.
struct DecideArgs {
  const double* e;          // [K x 2] whole-gradient energies
  DevState* st;             // .sparse receives the decision
  double* ewma;             // moving-average states or null
  double beta, delta;
  uint64_t* counters;       // accounting or null
  double* energies_out;     // copy of e, or null
  uint8_t* compressed_out;  // or null
  uint64_t n;
  uint32_t K;
  uint32_t k[kMaxK];        // entries kept per device
};
hipError_t launch_layers_decide(const DecideArgs& a, hipStream_t s);
hipError_t launch_rows(const RowsCtx& rc, const RowsPrep& rp, double* energies, hipStream_t s);
// energies = the short layers' energies (layer order) + add (the long layers', or null)
hipError_t launch_rows_energy(const RowsCtx& rc, double* energies, hipStream_t s);
hipError_t launch_zero_words(uint32_t* p, uint32_t n, hipStream_t s);

// k = clamp(floor(ratio * n), 1, n), the same double arithmetic on host and device.
__host__ __device__ inline uint64_t k_of(uint64_t n, double ratio)
{
  if (n == 0) return 0;
  const double f = __builtin_floor(ratio * (double)n);
  uint64_t k = (uint64_t)f;
  if (k < 1) k = 1;
  if (k > n) k = n;
  return k;
}

// The adaptive compression rule of §IV on a device's energies E_all, E_kept:
// with a moving-average state m (2 doubles; both 0 means no history, and the
// energies are taken as they are) the rule sees m <- beta m + (1 - beta) E.
// Returns 1 to send Top-k (relative energy loss at most delta), else 0.
__device__ inline uint32_t adaptive_rule(double ea, double ek, double* m, double beta, double delta)
{
  if (m) {
    if (m[0] == 0.0 && m[1] == 0.0) {
      m[0] = ea;
      m[1] = ek;
    } else {
      m[0] = beta * m[0] + (1.0 - beta) * ea;
      m[1] = beta * m[1] + (1.0 - beta) * ek;
    }
    ea = m[0];
    ek = m[1];
  }
  const double rho = (ea == 0.0) ? 0.0 : __builtin_fabs(ea - ek) / ea;
  return (rho <= delta) ? 1u : 0u;
}

// §V-G accounting of one iteration: [0] iterations that sent Top-k, [1]
// iterations, [2] floats sent (k when compressed, n otherwise).
__device__ inline void account(uint64_t* q, uint32_t sparse, uint64_t k, uint64_t n)
{
  q[0] += sparse;
  q[1] += 1u;
  q[2] += sparse ? k : n;
}

// ---- sizing shared by host and device -----------------------------------------------------
__host__ __device__ inline uint32_t bitlen32(uint32_t x) { return x ? 32u - (uint32_t)__builtin_clz(x) : 0u; }

__host__ __device__ inline uint32_t ceil_div_u64(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }

// ---- device primitives ------------------------------------------------------------------
__device__ inline uint32_t key_of(float x) { return __float_as_uint(x) & kKeyMask; }

__device__ inline uint32_t lane_id() { return threadIdx.x & 63; }

__device__ inline uint64_t ballot(bool p) { return __ballot(p); }

// Set bits of `mask` in lanes below the calling lane.
__device__ inline uint32_t mbcnt(uint64_t mask)
{
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ inline uint32_t wave_incl_scan(uint32_t v)
{
  const uint32_t l = lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t t = __shfl_up(v, d, 64);
    if (l >= (uint32_t)d) v += t;
  }
  return v;
}

__device__ inline uint64_t wave_sum_u64(uint64_t v)
{
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

__device__ inline double wave_sum_f64(double v)
{
  // Butterfly: every lane ends with the same value, summed in a fixed pattern.
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// Fixed-order block sum of one double per thread (deterministic).
__device__ inline double block_sum_f64(double v, double* lds4)
{
  v = wave_sum_f64(v);
  if (lane_id() == 0) lds4[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = ((lds4[0] + lds4[1]) + (lds4[2] + lds4[3]));
  __syncthreads();
  return r;
}

}  // namespace scadles
