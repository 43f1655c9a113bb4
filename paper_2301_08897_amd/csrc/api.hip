// api.hip -- the C ABI of libscadles (declared in include/scadles.h).
//
// Host side only: argument validation, the k rule, workspace layout, path
// choice per device, and the launch sequence. Every entry point validates
// before launching anything and never allocates device memory.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "scadles.h"
#include "scadles_internal.h"

using namespace scadles;

namespace scadles {

thread_local std::string g_err;

scadles_status fail(scadles_status st, const char* fmt, ...)
{
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

}  // namespace scadles

namespace {

std::atomic<int> g_validate{0}, g_force_exact{0}, g_force_fallback{0}, g_parts{1}, g_inject_count_error{0};
// per-layer selection: layers of at most this many elements go to the row kernels
std::atomic<int64_t> g_row_max{1 << 21};
std::atomic<int64_t> g_row_split{65536};
std::atomic<int64_t> g_layer_order{1};
// Per-layer selection: workspace regions of the long layers, used in turn; the
// brackets of the first kLayerRegions long layers are computed up front.
constexpr uint32_t kLayerRegions = 2;
// Per-layer selection: the short layers' rows on a third stream beside the
// long layers (true) or on the caller's stream before them (false).
constexpr bool kRowsBeside = true;

scadles_status hip_fail(hipError_t e, const char* where)
{
  return fail(SCADLES_EHIP, "%s: %s", where, hipGetErrorString(e));
}

// ---- stage profiling ------------------------------------------------------------------------
// Per call: 0 start, 1 bracket done, 2 + 2i / 3 + 2i around main-pass group i,
// 2 + 2P selection done, 3 + 2P call done (P = groups of that call).
constexpr int kStages = SCADLES_PROFILE_STAGES;
constexpr int kProfEv = 4 + 2 * (int)kMaxParts;
constexpr int kProfMax = 4096;
std::mutex g_prof_mu;
bool g_prof_on = false;
struct ProfRec {
  hipEvent_t ev[kProfEv];
  uint32_t parts;
};
std::vector<ProfRec> g_prof_pool;
size_t g_prof_used = 0;

// A record to fill, or null when profiling is off or full.
ProfRec* prof_slot()
{
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on || g_prof_used >= g_prof_pool.size()) return nullptr;
  return &g_prof_pool[g_prof_used++];
}

// ---- the second stream of the pipelined selection, per GPU ---------------------------------
struct StreamSet {
  bool ready = false;
  hipStream_t s2 = nullptr;
  hipEvent_t done[kMaxParts] = {};   // end of each main pass
  hipEvent_t join = nullptr;
  std::mutex launch_mu;      // one call's launch sequence at a time (the events are shared)
  // per-layer selection: the short layers' rows run on s3 beside the long layers
  hipStream_t s3 = nullptr;
  hipEvent_t fork = nullptr, rows_done = nullptr;
  // long layers: end of a layer's main pass; end of the bracket of the layer
  // using each of the two workspace regions; end of all the layers' rests
  hipEvent_t layer_main = nullptr, bracket_done[kLayerRegions] = {}, rests_done = nullptr;
  std::mutex rows_mu;
};
constexpr int kMaxGpus = 64;
StreamSet g_streams[kMaxGpus];
std::mutex g_streams_mu;

// The calling thread's current GPU's set, created on first use (default priority).
StreamSet* stream_set()
{
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxGpus) return nullptr;
  std::lock_guard<std::mutex> lk(g_streams_mu);
  StreamSet& ss = g_streams[dev];
  if (!ss.ready) {
    if (hipStreamCreateWithFlags(&ss.s2, hipStreamNonBlocking) != hipSuccess) return nullptr;
    for (auto& e : ss.done)
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipStreamCreateWithFlags(&ss.s3, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&ss.rows_done, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&ss.layer_main, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&ss.rests_done, hipEventDisableTiming) != hipSuccess) return nullptr;
    for (auto& e : ss.bracket_done)
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
    ss.ready = true;
  }
  return &ss;
}

// ---- static scratch of the allocation-free selection --------------------------------------
// scadles_topk_select_noalloc keeps its workspace here instead of in a caller
// buffer: one array per GPU, created when the code object loads on that GPU
// and held until the process ends. In host code `scratch` names a host-side
// stand-in, not device memory: only the address from hipGetSymbolAddress,
// taken once per device with that device current, is passed to kernels.
constexpr size_t kScratchBytes = SCADLES_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void* g_scratch_ptr[kMaxGpus] = {};
std::mutex g_scratch_mu;

// The current GPU's scratch address, looked up on the first call on that GPU.
hipError_t scratch_address(void** out)
{
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxGpus) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// ---- layout ---------------------------------------------------------------------------------
constexpr uint64_t kFastMinN = 65536;
constexpr uint64_t kCapAlign = 64;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
  uint32_t K = 0, tpd = 0, nslot = 0, ngrp = 0, nfb = 0, nbmax = 0, nrange = 0, s_stride = 0, s_n = 0;
  uint64_t n = 0;
  uint32_t k[kMaxK], cap[kMaxK], mode[kMaxK], r_lo[kMaxK], r_hi[kMaxK];
  uint32_t any_fast = 0;
  size_t o_desc, o_st, o_hist, o_scnt, o_soff, o_olist, o_slot, o_epart, o_cidx, o_cval, o_band, o_gcnt, o_gpre, o_bcnt, o_bpre, o_be, o_fb, o_lb,
      o_aerr;
  size_t total = 0;
};

uint64_t k_rule(uint64_t n, double ratio)
{
  if (n == 0 || n > 0xFFFFFFFFull) return 0;
  if (!(ratio > 0.0) || !(ratio <= 1.0)) return 0;
  const double f = std::floor(ratio * (double)n);
  uint64_t k = (uint64_t)f;
  if (k < 1) k = 1;
  if (k > n) k = n;
  return k;
}

// Sample: one chunk of kSChunk elements every `stride` elements.
void sample_geometry(uint64_t n, uint32_t& stride, uint32_t& s_n)
{
  // at most one chunk per 65536 elements, at least 1024 chunks while n allows:
  // a smaller sample widens the bracket and overflows the tiles' regions
  uint64_t st = 65536;
  if (n / st < 1024) {
    st = (n / 1024) / kSChunk * kSChunk;
    if (st < (uint64_t)kSChunk) st = kSChunk;
  }
  const uint64_t chunks = (n + st - 1) / st;
  uint64_t total = 0;
  for (uint64_t c = 0; c < chunks; ++c) {
    const uint64_t start = c * st;
    total += (n - start < (uint64_t)kSChunk) ? n - start : (uint64_t)kSChunk;
  }
  stride = (uint32_t)st;
  s_n = (uint32_t)total;
}

bool make_layout(uint32_t K, uint64_t n, const double* ratios, bool force_exact, bool with_select, Layout& L)
{
  L.K = K;
  L.n = n;
  // Tiles cover the 16-byte-aligned virtual row [0, n + shift), shift <= 3.
  L.tpd = ceil_div_u64(n + 3, kTile);
  L.nslot = L.tpd;
  L.ngrp = ceil_div_u64(L.nslot, kGatherSlots);
  L.nrange = ceil_div_u64(n, kARange);
  sample_geometry(n, L.s_stride, L.s_n);
  uint64_t sum_cap = 0;
  L.any_fast = 0;
  for (uint32_t j = 0; j < K; ++j) {
    const uint64_t k = with_select ? k_rule(n, ratios[j]) : 0;
    if (with_select && k == 0) return false;
    L.k[j] = (uint32_t)k;
    L.cap[j] = 0;
    L.mode[j] = kModeExact;
    L.r_lo[j] = L.r_hi[j] = 0;
    if (!with_select) continue;
    uint64_t slack = n / 8;
    if (slack > (1ull << 20)) slack = 1ull << 20;
    uint64_t cap = 2 * k + slack;
    cap = (cap + kCapAlign - 1) / kCapAlign * kCapAlign;
    const bool fast = !force_exact && n >= kFastMinN && 2 * cap <= n && cap < (1ull << 31);
    if (fast) {
      L.mode[j] = kModeFast;
      L.cap[j] = (uint32_t)cap;
      const double kf = (double)k * (double)L.s_n / (double)n;
      const double sd = std::sqrt(kf);
      double rlo = std::ceil(kf + 6.0 * sd + 8.0);
      if (rlo > (double)L.s_n) rlo = (double)L.s_n;
      if (rlo < 1.0) rlo = 1.0;
      double rhi = std::floor(kf - 6.0 * sd - 8.0);
      if (rhi < 1.0) rhi = 0.0;
      L.r_lo[j] = (uint32_t)rlo;
      L.r_hi[j] = (uint32_t)rhi;
      L.any_fast = 1;
      sum_cap += cap;
    }
  }
  L.nfb = ceil_div_u64(n + 3, kCBlk);
  L.nbmax = L.nfb;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  if (with_select) {
    L.o_desc = take(sizeof(DevDesc) * K);
    L.o_st = take(sizeof(DevState) * K);
    L.o_hist = take(sizeof(uint32_t) * (size_t)K * kSlots * kBins);
    // Slots are needed only by fast-path devices; sized for all K for simplicity.
    const size_t nslots = L.any_fast ? (size_t)K * L.nslot : 0;
    L.o_scnt = take(sizeof(uint32_t) * (size_t)K * L.nslot);
    L.o_soff = take(sizeof(uint64_t) * (size_t)K * L.nslot);
    L.o_olist = take(sizeof(uint32_t) * (size_t)K * L.nslot);
    L.o_slot = take(sizeof(uint32_t) * nslots * kSlotWords);
    L.o_epart = take(sizeof(double) * (size_t)K * L.nslot);
    L.o_cidx = take(sizeof(uint32_t) * sum_cap);
    L.o_cval = take(sizeof(float) * sum_cap);
    L.o_band = take(sizeof(uint32_t) * sum_cap);
    L.o_gcnt = take(sizeof(uint64_t) * (size_t)K * L.ngrp);
    L.o_gpre = take(sizeof(uint64_t) * (size_t)K * L.ngrp);
    L.o_bcnt = take(sizeof(uint64_t) * (size_t)K * L.nbmax);
    L.o_bpre = take(sizeof(uint64_t) * (size_t)K * L.nbmax);
    L.o_be = take(sizeof(double) * (size_t)K * L.nbmax);
    L.o_fb = take(sizeof(uint32_t));
  }
  L.o_lb = take(sizeof(uint32_t) * (size_t)K * L.nrange);
  L.o_aerr = take(256);
  L.total = o;
  return true;
}

Ctx make_ctx(const Layout& L, void* ws)
{
  char* b = static_cast<char*>(ws);
  Ctx c;
  memset(&c, 0, sizeof(c));
  c.desc = reinterpret_cast<DevDesc*>(b + L.o_desc);
  c.st = reinterpret_cast<DevState*>(b + L.o_st);
  c.hist = reinterpret_cast<uint32_t*>(b + L.o_hist);
  c.slot_cnt = reinterpret_cast<uint32_t*>(b + L.o_scnt);
  c.slot_off = reinterpret_cast<uint64_t*>(b + L.o_soff);
  c.ovf_list = reinterpret_cast<uint32_t*>(b + L.o_olist);
  c.slot = reinterpret_cast<uint32_t*>(b + L.o_slot);
  c.epart = reinterpret_cast<double*>(b + L.o_epart);
  c.cand_idx = reinterpret_cast<uint32_t*>(b + L.o_cidx);
  c.cand_val = reinterpret_cast<float*>(b + L.o_cval);
  c.band = reinterpret_cast<uint32_t*>(b + L.o_band);
  c.grp_cnt = reinterpret_cast<uint64_t*>(b + L.o_gcnt);
  c.grp_pre = reinterpret_cast<uint64_t*>(b + L.o_gpre);
  c.blk_cnt = reinterpret_cast<uint64_t*>(b + L.o_bcnt);
  c.blk_pre = reinterpret_cast<uint64_t*>(b + L.o_bpre);
  c.blk_e = reinterpret_cast<double*>(b + L.o_be);
  c.fb_count = reinterpret_cast<uint32_t*>(b + L.o_fb);
  c.n = L.n;
  c.K = L.K;
  c.tpd = L.tpd;
  c.nslot = L.nslot;
  c.ngrp = L.ngrp;
  c.nfb = L.nfb;
  c.nbmax = L.nbmax;
  c.s_stride = L.s_stride;
  c.s_n = L.s_n;
  return c;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Whether two float arrays of n elements share memory.
bool overlap(const float* a, const float* b, uint64_t n)
{
  const char* x = reinterpret_cast<const char*>(a);
  const char* y = reinterpret_cast<const char*>(b);
  return x < y + n * sizeof(float) && y < x + n * sizeof(float);
}

scadles_status check_ws(void* ws, size_t ws_bytes, size_t need)
{
  if (!ws) return fail(SCADLES_EWORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (!aligned(ws, 256)) return fail(SCADLES_EWORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(SCADLES_EWORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return SCADLES_OK;
}

scadles_status check_n(uint64_t n)
{
  if (n == 0 || n > 0xFFFFFFFFull) return fail(SCADLES_EINVAL, "n = %llu is outside [1, 2^32 - 1]", (unsigned long long)n);
  return SCADLES_OK;
}

scadles_status check_weights(const float* w, uint32_t K)
{
  if (!w) return fail(SCADLES_EINVAL, "weights is NULL");
  double sum = 0.0;
  for (uint32_t j = 0; j < K; ++j) {
    if (!std::isfinite(w[j]) || w[j] < 0.0f) return fail(SCADLES_EINVAL, "weight %u is negative or not finite", j);
    sum += (double)w[j];
  }
  if (std::fabs(sum - 1.0) > (double)K * std::ldexp(1.0, -23))
    return fail(SCADLES_EINVAL, "weights sum to %.17g, not 1 (Eqn 4a)", sum);
  return SCADLES_OK;
}

// Number of pipelined device groups for a call (option "parts", at most K).
uint32_t parts_for(const Layout& L)
{
  int p = g_parts.load();
  if (p < 1) p = 1;
  if (p > (int)kMaxParts) p = (int)kMaxParts;
  if ((uint32_t)p > L.K) p = (int)L.K;
  return (uint32_t)p;
}

// Kernel context and launch plan of one selection call.
void select_setup(const Layout& L, void* ws, double delta, double* energies, uint8_t* compressed, uint32_t* lb,
                  const scadles_step_options* opt, uint32_t idx_base, uint32_t e_stride, Ctx& c, SelectPlan& p)
{
  c = make_ctx(L, ws);
  c.delta = delta;
  c.energies_out = energies;
  c.compressed_out = compressed;
  c.force_fallback = g_force_fallback.load() ? 1u : 0u;
  c.inject_count_error = g_inject_count_error.load() ? 1u : 0u;
  p.any_fast = L.any_fast;
  p.sample_blocks = ceil_div_u64(L.s_n, kSBlk);
  const uint64_t tiles = (uint64_t)L.K * L.tpd;
  p.full_workers = (uint32_t)(tiles < (uint64_t)kFullWorkers ? tiles : (uint64_t)kFullWorkers);
  p.parts = parts_for(L);
  p.beside = 0;
  c.lb = lb;
  c.nrange = L.nrange;
  c.idx_base = idx_base;
  c.e_stride = e_stride;
  if (opt) {
    c.ewma = opt->ewma;
    c.ewma_beta = opt->ewma_beta;
    c.counters = opt->counters;
  }
}

scadles_status run_select(const Layout& L, const PrepArgs& a, void* ws, double delta, double* energies,
                          uint8_t* compressed, hipStream_t s, ProfRec* pr, uint32_t* lb = nullptr,
                          const scadles_step_options* opt = nullptr)
{
  Ctx c;
  SelectPlan p;
  select_setup(L, ws, delta, energies, compressed, lb, opt, 0, 2u, c, p);
  if (pr) pr->parts = p.parts;
  StreamSet* ss = p.parts > 1 ? stream_set() : nullptr;
  if (p.parts > 1 && !ss) return fail(SCADLES_EHIP, "could not create the pipeline stream");
  hipError_t e;
  if (ss) {
    std::lock_guard<std::mutex> lk(ss->launch_mu);
    e = launch_select(c, a, p, s, ss->s2, ss->done, ss->join, pr ? pr->ev : nullptr);
  } else {
    e = launch_select(c, a, p, s, nullptr, nullptr, nullptr, pr ? pr->ev : nullptr);
  }
  if (e != hipSuccess) return hip_fail(e, "select launch");
  return SCADLES_OK;
}

// Validation mode: waits for the call's work on s and reports a device whose
// selection state carries an error bit other than a recovered bracket miss
// (its output would be wrong).
scadles_status check_states(const Layout& L, void* ws, hipStream_t s)
{
  DevState st[kMaxK];
  hipError_t e = hipMemcpyAsync(st, static_cast<char*>(ws) + L.o_st, sizeof(DevState) * L.K, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "selection state readback");
  for (uint32_t j = 0; j < L.K; ++j)
    if (st[j].err & kErrFatal)
      return fail(SCADLES_EINTERNAL, "device %u: the selection's internal check failed (error bits 0x%x)", j,
                  st[j].err);
  return SCADLES_OK;
}

}  // namespace

// ---- ABI ----------------------------------------------------------------------------------------
extern "C" {

uint64_t scadles_topk_k(uint64_t n, double ratio) { return k_rule(n, ratio); }

size_t scadles_workspace_bytes(uint32_t K, uint64_t n, const double* ratios)
{
  if (K == 0 || K > kMaxK || !ratios || n == 0 || n > 0xFFFFFFFFull) return 0;
  Layout L;
  if (!make_layout(K, n, ratios, g_force_exact.load() != 0, true, L)) return 0;
  // The fast/exact choice may change with the force_exact option; size for the larger.
  Layout Lf;
  make_layout(K, n, ratios, false, true, Lf);
  return L.total > Lf.total ? L.total : Lf.total;
}

size_t scadles_aggregate_workspace_bytes(uint32_t K, uint64_t n)
{
  if (K == 0 || K > kMaxK || n == 0 || n > 0xFFFFFFFFull) return 0;
  Layout L;
  make_layout(K, n, nullptr, false, false, L);
  return L.total;
}

// Argument checks and layout of a one-gradient selection.
static scadles_status topk_args(const float* grad, uint64_t n, double ratio, uint32_t* idx, float* val,
                                double* energies, Layout& L)
{
  if (scadles_status st = check_n(n)) return st;
  if (!grad || !idx || !val) return fail(SCADLES_EINVAL, "grad, idx and val must not be NULL");
  if (!aligned(grad, 4)) return fail(SCADLES_EINVAL, "grad must be 4-byte aligned");
  if (!aligned(idx, 4) || !aligned(val, 4)) return fail(SCADLES_EINVAL, "idx and val must be 4-byte aligned");
  if (energies && !aligned(energies, 8)) return fail(SCADLES_EINVAL, "energies must be 8-byte aligned");
  if (k_rule(n, ratio) == 0) return fail(SCADLES_EINVAL, "ratio %g is not in (0, 1]", ratio);
  make_layout(1, n, &ratio, g_force_exact.load() != 0, true, L);
  return SCADLES_OK;
}

// The selection of one gradient into a checked workspace (one device: one
// group, so no library stream is created and nothing is allocated).
static scadles_status topk_run(const float* grad, const Layout& L, uint32_t* idx, float* val, double* energies,
                               void* ws, hipStream_t s)
{
  PrepArgs a;
  memset(&a, 0, sizeof(a));
  a.grad[0] = grad;
  a.idx[0] = idx;
  a.val[0] = val;
  a.k[0] = L.k[0];
  a.cap[0] = L.cap[0];
  a.mode[0] = L.mode[0];
  a.r_lo[0] = L.r_lo[0];
  a.r_hi[0] = L.r_hi[0];
  ProfRec* pr = prof_slot();
  if (pr) (void)hipEventRecord(pr->ev[0], s);
  scadles_status st = run_select(L, a, ws, INFINITY, energies, nullptr, s, pr);
  if (pr) (void)hipEventRecord(pr->ev[3 + 2 * pr->parts], s);
  if (st == SCADLES_OK && g_validate.load()) st = check_states(L, ws, s);
  return st;
}

scadles_status scadles_topk_select(const float* grad, uint64_t n, double ratio, uint32_t* idx, float* val,
                                   double* energies, void* ws, size_t ws_bytes, void* stream)
{
  Layout L;
  if (scadles_status st = topk_args(grad, n, ratio, idx, val, energies, L)) return st;
  if (scadles_status st = check_ws(ws, ws_bytes, L.total)) return st;
  return topk_run(grad, L, idx, val, energies, ws, static_cast<hipStream_t>(stream));
}

scadles_status scadles_topk_select_noalloc(const float* grad, uint64_t n, double ratio, uint32_t* idx, float* val,
                                           double* energies, void* stream)
{
  Layout L;
  if (scadles_status st = topk_args(grad, n, ratio, idx, val, energies, L)) return st;
  if (L.total > kScratchBytes)
    return fail(SCADLES_EWORKSPACE,
                "n = %llu at ratio %g needs %zu bytes of scratch; the library's static scratch holds %zu "
                "(use scadles_topk_select with a workspace)",
                (unsigned long long)n, ratio, L.total, kScratchBytes);
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return hip_fail(e, "scratch address");
  return topk_run(grad, L, idx, val, energies, ws, static_cast<hipStream_t>(stream));
}

// Layers of a per-layer selection: checks seg_off (0 = off[0] < ... < off[L]
// <= 2^32 - 1) and returns the kept entries of one device.
// At most 2^24 layers: keeps every (device, layer) index within 32 bits.
constexpr uint32_t kMaxLayers = 1u << 24;

static scadles_status check_layers(const uint64_t* seg_off, uint32_t L)
{
  if (!seg_off || L == 0) return fail(SCADLES_EINVAL, "seg_off must not be NULL and L >= 1");
  if (L > kMaxLayers) return fail(SCADLES_EINVAL, "L = %u exceeds 2^24 layers", L);
  if (seg_off[0] != 0) return fail(SCADLES_EINVAL, "seg_off[0] must be 0");
  for (uint32_t l = 0; l < L; ++l)
    if (!(seg_off[l] < seg_off[l + 1])) return fail(SCADLES_EINVAL, "layer %u is empty or out of order", l);
  if (seg_off[L] > 0xFFFFFFFFull) return fail(SCADLES_EINVAL, "n = %llu exceeds 2^32 - 1", (unsigned long long)seg_off[L]);
  return SCADLES_OK;
}

uint64_t scadles_layers_k(const uint64_t* seg_off, uint32_t L, double ratio)
{
  if (!seg_off || L == 0 || L > kMaxLayers || seg_off[0] != 0) return 0;
  uint64_t k = 0;
  for (uint32_t l = 0; l < L; ++l) {
    if (!(seg_off[l] < seg_off[l + 1]) || seg_off[L] > 0xFFFFFFFFull) return 0;
    const uint64_t kl = k_rule(seg_off[l + 1] - seg_off[l], ratio);
    if (kl == 0) return 0;
    k += kl;
  }
  return k;
}

// Workspace of a per-layer selection: the selection region (the largest
// layer's, for layers selected by the multi-launch path) and after it the
// row region (layer table, row descriptors, per-row energies).
struct LayersWs {
  size_t sel = 0, table = 0, rows = 0, row_e = 0, bst = 0, chunk = 0, cand = 0, part_e = 0, err = 0, total = 0;
};

// Parts of a split row of n elements (the virtual row [0, n + shift), shift <= 3).
static uint64_t row_parts_of(uint64_t n) { return ceil_div_u64(n + 3, kRowPartLen); }

// Capacity of one wave's candidate region in the split rows of a layer of n
// elements: twice the wave's share of 2 k_max + 4096 (k_max the largest k of
// the devices) plus 64, in multiples of 64; 0 when that exceeds half a
// wave's elements (high ratios) or n exceeds kRowSplitMax: such rows are not
// split. Up to kRowSplitMax it falls as n grows, so the split rows are the
// longest ones.
static uint64_t row_wave_cap(uint64_t n, const double* ratios, uint32_t K)
{
  if (n > kRowSplitMax) return 0;
  uint64_t kmax = 0;
  for (uint32_t j = 0; j < K; ++j) kmax = std::max<uint64_t>(kmax, k_rule(n, ratios[j]));
  const uint64_t share = (2 * (2 * kmax + 4096) * kRowWaveLen + n - 1) / n + 64;
  return share <= kRowWaveLen / 2 ? (share + 63) / 64 * 64 : 0;
}

// Entries of a split row's candidate list (0: the row is not split).
static uint64_t row_cand_list(uint64_t n, const double* ratios, uint32_t K)
{
  return row_parts_of(n) * kRowPartWaves * row_wave_cap(n, ratios, K);
}

static LayersWs layers_ws(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios)
{
  LayersWs w;
  size_t most = 0;
  for (uint32_t l = 0; l < L; ++l) {
    const size_t b = scadles_workspace_bytes(K, seg_off[l + 1] - seg_off[l], ratios);
    if (b == 0) return LayersWs{};
    if (b > most) most = b;
  }
  // two selection regions: consecutive long layers alternate between them
  // split rows: room for every layer that could be split under any option
  uint64_t nbig = 0, parts = 0, cands = 0;
  for (uint32_t l = 0; l < L; ++l) {
    const uint64_t nl = seg_off[l + 1] - seg_off[l];
    if (nl > kRowSplitMin && row_cand_list(nl, ratios, K) > 0) {
      ++nbig;
      parts += row_parts_of(nl);
      cands += row_cand_list(nl, ratios, K);
    }
  }
  parts *= K;
  cands *= K;
  w.sel = align256(most);
  w.table = kLayerRegions * w.sel;
  w.rows = align256(w.table + sizeof(uint64_t) * (4ull * L + 3));
  w.row_e = align256(w.rows + sizeof(RowDesc) * (size_t)K * L);
  w.bst = align256(w.row_e + sizeof(double) * 2ull * K * L);
  w.chunk = align256(w.bst + sizeof(BigRowState) * (size_t)(nbig * K));
  w.cand = align256(w.chunk + sizeof(uint32_t) * (size_t)kChunkWords * kRowPartChunks * parts);
  w.part_e = align256(w.cand + sizeof(uint64_t) * cands);
  w.err = align256(w.part_e + sizeof(double) * 2ull * kRowPartWaves * parts);
  w.total = align256(w.err + sizeof(uint32_t) * K);
  return w;
}

size_t scadles_layers_workspace_bytes(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios)
{
  if (K == 0 || K > kMaxK || !ratios || scadles_layers_k(seg_off, L, 0.5) == 0) return 0;
  for (uint32_t j = 0; j < K; ++j)
    if (scadles_layers_k(seg_off, L, ratios[j]) == 0) return 0;
  return layers_ws(K, seg_off, L, ratios).total;
}

// The per-layer selection into idx / val with the whole-gradient energies
// (arguments validated by the caller; lw laid out in ws).
static scadles_status run_layers(const float* const* grads, uint32_t K, const uint64_t* seg_off, uint32_t L,
                                 const double* ratios, uint32_t* const* idx, float* const* val, double* energies,
                                 void* ws, const LayersWs& lw, hipStream_t s)
{
  uint8_t* base = static_cast<uint8_t*>(ws);

  // Short layers (at most row_max elements), longest first, go to the row
  // kernels: one workgroup per (layer, device) row, all in one launch.
  const uint64_t row_max = (uint64_t)g_row_max.load();
  std::vector<uint32_t> shorts;
  for (uint32_t l = 0; l < L; ++l)
    if (seg_off[l + 1] - seg_off[l] <= row_max) shorts.push_back(l);
  std::stable_sort(shorts.begin(), shorts.end(), [&](uint32_t a, uint32_t b) {
    return seg_off[a + 1] - seg_off[a] > seg_off[b + 1] - seg_off[b];
  });
  // The longest of them, those of more than row_split elements, are split into
  // parts, each read by a workgroup of its own.
  const uint64_t split = std::max<uint64_t>((uint64_t)g_row_split.load(), kRowSplitMin);
  // (rows above kRowSplitMax are not split; they come first in the order, so
  // the split rows are moved to the front of the row list)
  std::stable_partition(shorts.begin(), shorts.end(), [&](uint32_t l) {
    const uint64_t nl = seg_off[l + 1] - seg_off[l];
    return nl > split && row_cand_list(nl, ratios, K) > 0;
  });
  uint32_t Lb = 0;
  while (Lb < shorts.size()) {
    const uint64_t nl = seg_off[shorts[Lb] + 1] - seg_off[shorts[Lb]];
    if (nl <= split || row_cand_list(nl, ratios, K) == 0) break;
    ++Lb;
  }
  std::vector<uint64_t> table(2ull * L + 1, ~0ull);
  for (uint32_t l = 0; l <= L; ++l) table[l] = seg_off[l];
  for (size_t q = 0; q < shorts.size(); ++q) table[L + 1 + shorts[q]] = q;
  uint64_t part_pre = 0;
  for (uint32_t q = 0; q < Lb; ++q) {
    table.push_back(part_pre);
    part_pre += row_parts_of(seg_off[shorts[q] + 1] - seg_off[shorts[q]]);
  }
  table.push_back(part_pre);
  uint64_t cand_pre = 0;
  for (uint32_t q = 0; q < Lb; ++q) {
    table.push_back(cand_pre);
    cand_pre += row_cand_list(seg_off[shorts[q] + 1] - seg_off[shorts[q]], ratios, K);
  }
  table.push_back(cand_pre);
  RowsCtx rc;
  rc.table = reinterpret_cast<const uint64_t*>(base + lw.table);
  rc.rows = reinterpret_cast<RowDesc*>(base + lw.rows);
  rc.row_e = reinterpret_cast<double*>(base + lw.row_e);
  rc.K = K;
  rc.L = L;
  rc.Ls = (uint32_t)shorts.size();
  rc.Lb = Lb;
  rc.nparts = (uint32_t)(part_pre * K);
  rc.bst = reinterpret_cast<BigRowState*>(base + lw.bst);
  rc.chunk = reinterpret_cast<uint32_t*>(base + lw.chunk);
  rc.cand = reinterpret_cast<uint64_t*>(base + lw.cand);
  rc.part_e = reinterpret_cast<double*>(base + lw.part_e);
  RowsPrep rp;
  memset(&rp, 0, sizeof(rp));
  for (uint32_t j = 0; j < K; ++j) {
    rp.grad[j] = grads[j];
    rp.idx[j] = idx[j];
    rp.val[j] = val[j];
    rp.ratio[j] = ratios[j];
  }
  const bool any_long = rc.Ls < L;
  // Consecutive long layers pipeline over two workspace regions: each one's
  // main pass runs on s, everything after it on the library's second stream
  // s2, and the bracket of the next layer goes to s2 ahead of that rest (right
  // after the rest of the layer before, the last user of its region), so it
  // runs during the main pass. The first layer's bracket runs on s, and only
  // then do the rows of the short layers start on the third stream beside
  // them: their workgroups fill whole compute units and would hold the small
  // bracket kernels back. Every layer's energies go to a slot of their own,
  // summed in layer order once s has waited for everything, so the order in
  // which the long layers run does not change them.
  StreamSet* ss = any_long ? stream_set() : nullptr;
  if (any_long && !ss) return fail(SCADLES_EHIP, "could not create the layer pipeline streams");
  std::unique_lock<std::mutex> lk;
  if (ss) lk = std::unique_lock<std::mutex>(ss->rows_mu);
  const bool both = ss && rc.Ls > 0;               // long and short layers
  const bool rows_beside = both && kRowsBeside;
  // validation mode: the long layers' fatal error bits, ORed per device
  uint32_t* err_acc = ss && g_validate.load() ? reinterpret_cast<uint32_t*>(base + lw.err) : nullptr;

  // Long layers: the multi-launch selection of each, its indices offset by the
  // layer's start, its energies in the layer's own slot.
  struct LongLayer {
    Ctx c;
    SelectPlan p;
    PrepArgs a;
  };
  // the long layers in index order (layer[i]) with where their entries start
  // in each device's output (at[i * K + j]), then the order they run in
  std::vector<uint32_t> layer;
  std::vector<uint64_t> at;
  {
    uint64_t run[kMaxK] = {};
    for (uint32_t l = 0; l < L; ++l) {
      const uint64_t nl = seg_off[l + 1] - seg_off[l];
      if (nl > row_max) {
        layer.push_back(l);
        at.insert(at.end(), run, run + K);
      }
      for (uint32_t j = 0; j < K; ++j) run[j] += k_rule(nl, ratios[j]);
    }
  }
  std::vector<uint32_t> order(layer.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (uint32_t)i;
  const int64_t lorder = g_layer_order.load();
  if (lorder == 1 || lorder == 2)
    std::stable_sort(order.begin(), order.end(), [&](uint32_t x, uint32_t y) {
      const uint64_t nx = seg_off[layer[x] + 1] - seg_off[layer[x]], ny = seg_off[layer[y] + 1] - seg_off[layer[y]];
      return lorder == 1 ? nx < ny : nx > ny;
    });
  std::vector<LongLayer> longs(order.size());
  for (size_t q = 0; q < order.size(); ++q) {
    const uint32_t i = order[q], l = layer[i];
    const uint64_t off = seg_off[l], nl = seg_off[l + 1] - off;
    Layout Ll;
    make_layout(K, nl, ratios, g_force_exact.load() != 0, true, Ll);
    LongLayer& ll = longs[q];
    PrepArgs& a = ll.a;
    memset(&a, 0, sizeof(a));
    for (uint32_t j = 0; j < K; ++j) {
      a.grad[j] = grads[j] + off;
      a.idx[j] = idx[j] + at[(size_t)i * K + j];
      a.val[j] = val[j] + at[(size_t)i * K + j];
      a.k[j] = Ll.k[j];
      a.cap[j] = Ll.cap[j];
      a.mode[j] = Ll.mode[j];
      a.r_lo[j] = Ll.r_lo[j];
      a.r_hi[j] = Ll.r_hi[j];
    }
    // the layer's energies go to its own slot of the per-layer energies
    select_setup(Ll, base + (q % kLayerRegions) * lw.sel, INFINITY, energies ? rc.row_e + 2ull * l : nullptr,
                 nullptr, nullptr, nullptr, (uint32_t)off, 2u * L, ll.c, ll.p);
    ll.p.parts = 1;
    ll.p.beside = 1;
    ll.c.err_acc = err_acc;
  }

  hipError_t e = hipSuccess;
  if (err_acc) {
    e = launch_zero_words(err_acc, K, s);
    if (e != hipSuccess) return hip_fail(e, "error word clear");
  }
  if (ss) {
    // the library's streams start after the caller's earlier work on s (which may write the gradients)
    e = hipEventRecord(ss->fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(ss->s2, ss->fork, 0);
    if (e != hipSuccess) return hip_fail(e, "stream fork");
  }
  if (!longs.empty()) {
    e = launch_bracket(longs[0].c, longs[0].a, longs[0].p, s);
    if (e != hipSuccess) return hip_fail(e, "layer bracket");
  }
  hipStream_t sr = rows_beside ? ss->s3 : s;
  if (rows_beside) {
    e = hipEventRecord(ss->fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(sr, ss->fork, 0);
    if (e != hipSuccess) return hip_fail(e, "row stream fork");
  }
  e = launch_put_table(table.data(), table.size(), reinterpret_cast<uint64_t*>(base + lw.table), sr);
  if (e != hipSuccess) return hip_fail(e, "layer table");
  e = launch_rows(rc, rp, any_long ? nullptr : energies, sr);
  if (e != hipSuccess) return hip_fail(e, "row selection");
  if (rows_beside) {
    e = hipEventRecord(ss->rows_done, sr);
    if (e != hipSuccess) return hip_fail(e, "row stream join");
  }
  // the brackets of long layers 1 .. kLayerRegions - 1 on s2 up front; layer
  // li + kLayerRegions - 1's bracket after layer li - 1's rest (its region's
  // last user), ahead of layer li's rest
  for (size_t li = 1; li < longs.size() && li < kLayerRegions; ++li) {
    e = launch_bracket(longs[li].c, longs[li].a, longs[li].p, ss->s2);
    if (e == hipSuccess) e = hipEventRecord(ss->bracket_done[li % kLayerRegions], ss->s2);
    if (e != hipSuccess) return hip_fail(e, "layer bracket");
  }
  for (size_t li = 0; li < longs.size(); ++li) {
    const LongLayer& ll = longs[li];
    if (li > 0) {
      e = hipStreamWaitEvent(s, ss->bracket_done[li % kLayerRegions], 0);
      if (e != hipSuccess) return hip_fail(e, "layer pipeline");
    }
    e = launch_main(ll.c, ll.a, s);
    if (e == hipSuccess) e = hipEventRecord(ss->layer_main, s);
    const size_t nx = li + kLayerRegions - 1;
    if (e == hipSuccess && li > 0 && nx < longs.size()) {
      e = launch_bracket(longs[nx].c, longs[nx].a, longs[nx].p, ss->s2);
      if (e == hipSuccess) e = hipEventRecord(ss->bracket_done[nx % kLayerRegions], ss->s2);
    }
    if (e == hipSuccess) e = hipStreamWaitEvent(ss->s2, ss->layer_main, 0);
    if (e == hipSuccess) e = launch_rest(ll.c, ll.p, ss->s2);
    if (e != hipSuccess) return hip_fail(e, "layer pipeline");
  }
  if (!longs.empty()) {
    // s2 runs the layers' rests in order: its last one's end is all of them
    e = hipEventRecord(ss->rests_done, ss->s2);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, ss->rests_done, 0);
    if (e != hipSuccess) return hip_fail(e, "layer pipeline join");
  }
  if (rows_beside) {
    e = hipStreamWaitEvent(s, ss->rows_done, 0);
    if (e != hipSuccess) return hip_fail(e, "row stream join");
  }
  if (any_long && energies) {
    e = launch_rows_energy(rc, energies, s);
    if (e != hipSuccess) return hip_fail(e, "layer energies");
  }
  if (err_acc) {
    uint32_t err[kMaxK];
    e = hipMemcpyAsync(err, err_acc, sizeof(uint32_t) * K, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "selection state readback");
    for (uint32_t j = 0; j < K; ++j)
      if (err[j])
        return fail(SCADLES_EINTERNAL, "device %u: a long layer's internal check failed (error bits 0x%x)", j, err[j]);
  }
  return SCADLES_OK;
}

scadles_status scadles_topk_select_layers(const float* const* grads, uint32_t K, const uint64_t* seg_off, uint32_t L,
                                          const double* ratios, uint32_t* const* idx, float* const* val,
                                          double* energies, void* ws, size_t ws_bytes, void* stream)
{
  if (K == 0 || K > kMaxK) return fail(SCADLES_EINVAL, "K = %u is outside [1, %d]", K, kMaxK);
  if (scadles_status st = check_layers(seg_off, L)) return st;
  if (!grads || !ratios || !idx || !val) return fail(SCADLES_EINVAL, "NULL argument");
  if (energies && !aligned(energies, 8)) return fail(SCADLES_EINVAL, "energies must be 8-byte aligned");
  for (uint32_t j = 0; j < K; ++j) {
    if (!grads[j] || !idx[j] || !val[j]) return fail(SCADLES_EINVAL, "device %u has a NULL pointer", j);
    if (!aligned(grads[j], 4)) return fail(SCADLES_EINVAL, "grads[%u] must be 4-byte aligned", j);
    if (!aligned(idx[j], 4) || !aligned(val[j], 4)) return fail(SCADLES_EINVAL, "device %u outputs misaligned", j);
    if (scadles_layers_k(seg_off, L, ratios[j]) == 0)
      return fail(SCADLES_EINVAL, "ratio %g of device %u is not in (0, 1]", ratios[j], j);
  }
  const LayersWs lw = layers_ws(K, seg_off, L, ratios);
  if (scadles_status st = check_ws(ws, ws_bytes, lw.total)) return st;
  return run_layers(grads, K, seg_off, L, ratios, idx, val, energies, ws, lw, static_cast<hipStream_t>(stream));
}

// Workspace of the per-layer fused step: the per-layer selection's, then the
// energies, decisions, aggregation range markers and validation flag.
struct StepLayersWs {
  LayersWs lw;
  size_t e = 0, st = 0, lb = 0, err = 0, total = 0;
  uint32_t nrange = 0;
};

static StepLayersWs step_layers_ws(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios)
{
  StepLayersWs w;
  w.lw = layers_ws(K, seg_off, L, ratios);
  if (!w.lw.total) return StepLayersWs{};
  w.nrange = ceil_div_u64(seg_off[L], kARange);
  w.e = w.lw.total;
  w.st = align256(w.e + sizeof(double) * 2 * K);
  w.lb = align256(w.st + sizeof(DevState) * K);
  w.err = align256(w.lb + sizeof(uint32_t) * (size_t)K * w.nrange);
  w.total = align256(w.err + sizeof(uint32_t));
  return w;
}

size_t scadles_step_layers_workspace_bytes(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios)
{
  if (scadles_layers_workspace_bytes(K, seg_off, L, ratios) == 0) return 0;
  return step_layers_ws(K, seg_off, L, ratios).total;
}

scadles_status scadles_step_fused_layers(const float* const* grads, uint32_t K, const uint64_t* seg_off, uint32_t L,
                                         const double* ratios, double delta, const float* weights,
                                         uint32_t* const* idx, float* const* val, float* dense, double* energies,
                                         uint8_t* compressed, float* params, float lr,
                                         const scadles_step_options* options, void* ws, size_t ws_bytes,
                                         void* stream)
{
  if (K == 0 || K > kMaxK) return fail(SCADLES_EINVAL, "K = %u is outside [1, %d]", K, kMaxK);
  if (scadles_status st = check_layers(seg_off, L)) return st;
  const uint64_t n = seg_off[L];
  scadles_step_options opt;
  memset(&opt, 0, sizeof(opt));
  if (options) opt = *options;
  if (!grads || !ratios || !idx || !val || !dense) return fail(SCADLES_EINVAL, "NULL argument");
  if (std::isnan(delta) || delta < 0.0) return fail(SCADLES_EINVAL, "delta must be >= 0 (or +INFINITY)");
  if (!aligned(dense, 16)) return fail(SCADLES_EINVAL, "dense must be 16-byte aligned");
  if (params && !aligned(params, 16)) return fail(SCADLES_EINVAL, "params must be 16-byte aligned");
  if (params && !std::isfinite(lr)) return fail(SCADLES_EINVAL, "lr is not finite");
  if (opt.momentum_buf) {
    if (!params) return fail(SCADLES_EINVAL, "the momentum update needs params");
    if (!aligned(opt.momentum_buf, 16)) return fail(SCADLES_EINVAL, "momentum_buf must be 16-byte aligned");
    if (!std::isfinite(opt.momentum) || !std::isfinite(opt.weight_decay))
      return fail(SCADLES_EINVAL, "momentum and weight_decay must be finite");
    if (overlap(opt.momentum_buf, params, n) || overlap(opt.momentum_buf, dense, n))
      return fail(SCADLES_EINVAL, "momentum_buf overlaps params or dense");
  }
  if (opt.ewma) {
    if (!aligned(opt.ewma, 8)) return fail(SCADLES_EINVAL, "ewma must be 8-byte aligned");
    if (!(opt.ewma_beta >= 0.0 && opt.ewma_beta < 1.0)) return fail(SCADLES_EINVAL, "ewma_beta must be in [0, 1)");
  }
  if (opt.counters && !aligned(opt.counters, 8)) return fail(SCADLES_EINVAL, "counters must be 8-byte aligned");
  if (energies && !aligned(energies, 8)) return fail(SCADLES_EINVAL, "energies must be 8-byte aligned");
  if (scadles_status st = check_weights(weights, K)) return st;
  uint64_t kk[kMaxK];
  for (uint32_t j = 0; j < K; ++j) {
    if (!grads[j] || !idx[j] || !val[j]) return fail(SCADLES_EINVAL, "device %u has a NULL pointer", j);
    if (!aligned(grads[j], 4)) return fail(SCADLES_EINVAL, "grads[%u] must be 4-byte aligned", j);
    if (!aligned(idx[j], 4) || !aligned(val[j], 4)) return fail(SCADLES_EINVAL, "device %u outputs misaligned", j);
    kk[j] = scadles_layers_k(seg_off, L, ratios[j]);
    if (kk[j] == 0) return fail(SCADLES_EINVAL, "ratio %g of device %u is not in (0, 1]", ratios[j], j);
  }
  const StepLayersWs w = step_layers_ws(K, seg_off, L, ratios);
  if (scadles_status st = check_ws(ws, ws_bytes, w.total)) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* b = static_cast<char*>(ws);
  double* e_ws = reinterpret_cast<double*>(b + w.e);
  if (scadles_status st = run_layers(grads, K, seg_off, L, ratios, idx, val, e_ws, ws, w.lw, s)) return st;
  DecideArgs da;
  memset(&da, 0, sizeof(da));
  da.e = e_ws;
  da.st = reinterpret_cast<DevState*>(b + w.st);
  da.ewma = opt.ewma;
  da.beta = opt.ewma_beta;
  da.delta = delta;
  da.counters = opt.counters;
  da.energies_out = energies;
  da.compressed_out = compressed;
  da.n = n;
  da.K = K;
  AggArgs g;
  memset(&g, 0, sizeof(g));
  uint64_t kmax = 0;
  for (uint32_t j = 0; j < K; ++j) {
    da.k[j] = (uint32_t)kk[j];
    g.idx[j] = idx[j];
    g.val[j] = val[j];
    g.dense[j] = grads[j];
    g.k[j] = (uint32_t)kk[j];
    g.w[j] = weights[j];
    if (kk[j] > kmax) kmax = kk[j];
  }
  hipError_t e = launch_layers_decide(da, s);
  if (e != hipSuccess) return hip_fail(e, "decision launch");
  AggCtx c;
  memset(&c, 0, sizeof(c));
  c.st = da.st;
  c.lb = reinterpret_cast<uint32_t*>(b + w.lb);
  c.err = reinterpret_cast<uint32_t*>(b + w.err);
  c.out = dense;
  c.params = params;
  c.mbuf = opt.momentum_buf;
  c.lr = lr;
  c.mom = opt.momentum;
  c.wd = opt.weight_decay;
  c.K = K;
  c.nrange = w.nrange;
  c.kmax = (uint32_t)kmax;
  c.n = n;
  e = launch_marks_built(g, c, s);
  if (e != hipSuccess) return hip_fail(e, "marker launch");
  e = launch_aggregate(g, c, 0, true, s);
  if (e != hipSuccess) return hip_fail(e, "aggregate launch");
  return SCADLES_OK;
}

scadles_status scadles_weighted_aggregate(const scadles_sparse* sets, const float* weights, uint32_t K, uint64_t n,
                                          float* dense, void* ws, size_t ws_bytes, void* stream)
{
  if (K == 0 || K > kMaxK) return fail(SCADLES_EINVAL, "K = %u is outside [1, %d]", K, kMaxK);
  if (scadles_status st = check_n(n)) return st;
  if (!sets || !dense) return fail(SCADLES_EINVAL, "sets and dense must not be NULL");
  if (!aligned(dense, 16)) return fail(SCADLES_EINVAL, "dense must be 16-byte aligned");
  if (scadles_status st = check_weights(weights, K)) return st;
  // Empty sets contribute nothing and are dropped; the others keep their order.
  AggArgs a;
  memset(&a, 0, sizeof(a));
  uint64_t kmax = 0;
  uint32_t Kc = 0;
  for (uint32_t j = 0; j < K; ++j) {
    const scadles_sparse& S = sets[j];
    if (S.k == 0) continue;
    if (!S.val) return fail(SCADLES_EINVAL, "set %u has a NULL val", j);
    if (!S.idx) {
      if (S.k != n) return fail(SCADLES_EINVAL, "dense set %u must have k == n", j);
      if (!aligned(S.val, 4)) return fail(SCADLES_EINVAL, "dense set %u must be 4-byte aligned", j);
      a.dense[Kc] = S.val;
    } else {
      if (S.k > n) return fail(SCADLES_EINVAL, "set %u has k = %llu > n", j, (unsigned long long)S.k);
      if (!aligned(S.idx, 4) || !aligned(S.val, 4)) return fail(SCADLES_EINVAL, "set %u is misaligned", j);
      if (S.k > kmax) kmax = S.k;
    }
    a.idx[Kc] = S.idx;
    a.val[Kc] = S.val;
    a.k[Kc] = (uint32_t)S.k;
    a.w[Kc] = weights[j];
    ++Kc;
  }
  Layout L;
  make_layout(K, n, nullptr, false, false, L);
  if (scadles_status st = check_ws(ws, ws_bytes, L.total)) return st;
  char* b = static_cast<char*>(ws);
  AggCtx c;
  memset(&c, 0, sizeof(c));
  c.st = nullptr;
  c.lb = reinterpret_cast<uint32_t*>(b + L.o_lb);
  c.err = reinterpret_cast<uint32_t*>(b + L.o_aerr);
  c.out = dense;
  c.K = Kc;
  c.nrange = L.nrange;
  c.kmax = (uint32_t)kmax;
  c.n = n;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t validate = g_validate.load() ? 1u : 0u;
  hipError_t e = launch_aggregate(a, c, validate, false, s);
  if (e != hipSuccess) return hip_fail(e, "aggregate launch");
  if (validate) {
    uint32_t flag = 0;
    e = hipMemcpyAsync(&flag, c.err, sizeof(flag), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "aggregate validation");
    if (flag) return fail(SCADLES_EUNSORTED, "a sparse set's idx is not strictly ascending or reaches n");
  }
  return SCADLES_OK;
}

scadles_status scadles_apply_momentum_sgd(float* params, float* momentum_buf, const float* grad, uint64_t n,
                                          float lr, float momentum, float weight_decay, void* stream)
{
  if (scadles_status st = check_n(n)) return st;
  if (!params || !momentum_buf || !grad) return fail(SCADLES_EINVAL, "params, momentum_buf and grad must not be NULL");
  if (!aligned(params, 16) || !aligned(momentum_buf, 16) || !aligned(grad, 16))
    return fail(SCADLES_EINVAL, "params, momentum_buf and grad must be 16-byte aligned");
  if (!std::isfinite(lr) || !std::isfinite(momentum) || !std::isfinite(weight_decay))
    return fail(SCADLES_EINVAL, "lr, momentum and weight_decay must be finite");
  if (overlap(params, grad, n) || overlap(momentum_buf, grad, n) || overlap(params, momentum_buf, n))
    return fail(SCADLES_EINVAL, "params, momentum_buf and grad must not overlap");
  hipError_t e = launch_momentum_sgd(params, momentum_buf, grad, n, lr, momentum, weight_decay,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "momentum sgd launch");
  return SCADLES_OK;
}

scadles_status scadles_apply_sgd(float* params, const float* grad, uint64_t n, float lr, void* stream)
{
  if (scadles_status st = check_n(n)) return st;
  if (!params || !grad) return fail(SCADLES_EINVAL, "params and grad must not be NULL");
  if (!aligned(params, 16) || !aligned(grad, 16)) return fail(SCADLES_EINVAL, "params and grad must be 16-byte aligned");
  if (!std::isfinite(lr)) return fail(SCADLES_EINVAL, "lr is not finite");
  const char* pb = reinterpret_cast<const char*>(params);
  const char* gb = reinterpret_cast<const char*>(grad);
  if (pb < gb + n * sizeof(float) && gb < pb + n * sizeof(float))
    return fail(SCADLES_EINVAL, "params and grad overlap");
  hipError_t e = launch_sgd(params, grad, n, lr, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgd launch");
  return SCADLES_OK;
}

// Both fused entry points (opt all zero: scadles_step_fused).
static scadles_status step_fused_impl(const float* const* grads, uint32_t K, uint64_t n, const double* ratios,
                                      double delta, const float* weights, uint32_t* const* idx, float* const* val,
                                      float* dense, double* energies, uint8_t* compressed, float* params,
                                      float lr, const scadles_step_options& opt, void* ws, size_t ws_bytes,
                                      void* stream)
{
  float* mbuf = opt.momentum_buf;
  const float mom = opt.momentum, wd = opt.weight_decay;
  if (K == 0 || K > kMaxK) return fail(SCADLES_EINVAL, "K = %u is outside [1, %d]", K, kMaxK);
  if (scadles_status st = check_n(n)) return st;
  if (!grads || !ratios || !idx || !val || !dense) return fail(SCADLES_EINVAL, "NULL argument");
  if (std::isnan(delta) || delta < 0.0) return fail(SCADLES_EINVAL, "delta must be >= 0 (or +INFINITY)");
  if (!aligned(dense, 16)) return fail(SCADLES_EINVAL, "dense must be 16-byte aligned");
  if (params && !aligned(params, 16)) return fail(SCADLES_EINVAL, "params must be 16-byte aligned");
  if (params && !std::isfinite(lr)) return fail(SCADLES_EINVAL, "lr is not finite");
  if (mbuf) {
    if (!params) return fail(SCADLES_EINVAL, "the momentum update needs params");
    if (!aligned(mbuf, 16)) return fail(SCADLES_EINVAL, "momentum_buf must be 16-byte aligned");
    if (!std::isfinite(mom) || !std::isfinite(wd)) return fail(SCADLES_EINVAL, "momentum and weight_decay must be finite");
    if (overlap(mbuf, params, n) || overlap(mbuf, dense, n))
      return fail(SCADLES_EINVAL, "momentum_buf overlaps params or dense");
  }
  if (opt.ewma) {
    if (!aligned(opt.ewma, 8)) return fail(SCADLES_EINVAL, "ewma must be 8-byte aligned");
    if (!(opt.ewma_beta >= 0.0 && opt.ewma_beta < 1.0)) return fail(SCADLES_EINVAL, "ewma_beta must be in [0, 1)");
  }
  if (opt.counters && !aligned(opt.counters, 8)) return fail(SCADLES_EINVAL, "counters must be 8-byte aligned");
  if (energies && !aligned(energies, 8)) return fail(SCADLES_EINVAL, "energies must be 8-byte aligned");
  if (scadles_status st = check_weights(weights, K)) return st;
  for (uint32_t j = 0; j < K; ++j) {
    if (!grads[j] || !idx[j] || !val[j]) return fail(SCADLES_EINVAL, "device %u has a NULL pointer", j);
    if (!aligned(grads[j], 4)) return fail(SCADLES_EINVAL, "grads[%u] must be 4-byte aligned", j);
    if (!aligned(idx[j], 4) || !aligned(val[j], 4)) return fail(SCADLES_EINVAL, "device %u outputs misaligned", j);
    if (k_rule(n, ratios[j]) == 0) return fail(SCADLES_EINVAL, "ratio %g of device %u is not in (0, 1]", ratios[j], j);
  }
  Layout L;
  make_layout(K, n, ratios, g_force_exact.load() != 0, true, L);
  if (scadles_status st = check_ws(ws, ws_bytes, L.total)) return st;
  PrepArgs a;
  memset(&a, 0, sizeof(a));
  AggArgs g;
  memset(&g, 0, sizeof(g));
  uint64_t kmax = 0;
  for (uint32_t j = 0; j < K; ++j) {
    a.grad[j] = grads[j];
    a.idx[j] = idx[j];
    a.val[j] = val[j];
    a.k[j] = L.k[j];
    a.cap[j] = L.cap[j];
    a.mode[j] = L.mode[j];
    a.r_lo[j] = L.r_lo[j];
    a.r_hi[j] = L.r_hi[j];
    g.idx[j] = idx[j];
    g.val[j] = val[j];
    g.dense[j] = grads[j];
    g.k[j] = L.k[j];
    g.w[j] = weights[j];
    if (L.k[j] > kmax) kmax = L.k[j];
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  ProfRec* pr = prof_slot();
  char* b = static_cast<char*>(ws);
  AggCtx c;
  memset(&c, 0, sizeof(c));
  c.st = reinterpret_cast<const DevState*>(b + L.o_st);
  c.lb = reinterpret_cast<uint32_t*>(b + L.o_lb);
  c.err = reinterpret_cast<uint32_t*>(b + L.o_aerr);
  c.out = dense;
  c.params = params;
  c.mbuf = mbuf;
  c.lr = lr;
  c.mom = mom;
  c.wd = wd;
  c.K = K;
  c.nrange = L.nrange;
  c.kmax = (uint32_t)kmax;
  c.n = n;
  // each device group's range markers are built right after its selection
  if (pr) (void)hipEventRecord(pr->ev[0], s);
  if (scadles_status st = run_select(L, a, ws, delta, energies, compressed, s, pr, c.lb, &opt)) return st;
  hipError_t e = launch_aggregate(g, c, 0, true, s);
  if (pr) (void)hipEventRecord(pr->ev[3 + 2 * pr->parts], s);
  if (e != hipSuccess) return hip_fail(e, "aggregate launch");
  if (g_validate.load()) return check_states(L, ws, s);
  return SCADLES_OK;
}

scadles_status scadles_step_fused(const float* const* grads, uint32_t K, uint64_t n, const double* ratios,
                                  double delta, const float* weights, uint32_t* const* idx, float* const* val,
                                  float* dense, double* energies, uint8_t* compressed, float* params, float lr,
                                  void* ws, size_t ws_bytes, void* stream)
{
  scadles_step_options none;
  memset(&none, 0, sizeof(none));
  return step_fused_impl(grads, K, n, ratios, delta, weights, idx, val, dense, energies, compressed, params, lr,
                         none, ws, ws_bytes, stream);
}

scadles_status scadles_step_fused_ex(const float* const* grads, uint32_t K, uint64_t n, const double* ratios,
                                     double delta, const float* weights, uint32_t* const* idx, float* const* val,
                                     float* dense, double* energies, uint8_t* compressed, float* params, float lr,
                                     const scadles_step_options* options, void* ws, size_t ws_bytes, void* stream)
{
  if (!options) return fail(SCADLES_EINVAL, "options must not be NULL");
  return step_fused_impl(grads, K, n, ratios, delta, weights, idx, val, dense, energies, compressed, params, lr,
                         *options, ws, ws_bytes, stream);
}

scadles_status scadles_stream_weights(const double* rates, uint32_t K, double b_min, double b_max, double base_batch,
                                      float* weights, double* gamma)
{
  if (!rates || !weights || K == 0) return fail(SCADLES_EINVAL, "rates and weights must not be NULL, K >= 1");
  if (std::isnan(b_min) || std::isnan(b_max) || !(b_min <= b_max))
    return fail(SCADLES_EINVAL, "need b_min <= b_max");
  double total = 0.0;
  std::vector<double> b(K);
  for (uint32_t j = 0; j < K; ++j) {
    double s = rates[j];
    if (!std::isfinite(s) || s < 0.0) return fail(SCADLES_EINVAL, "rate %u is negative or not finite", j);
    if (s < b_min) s = b_min;
    if (s > b_max) s = b_max;
    b[j] = s;
    total += s;
  }
  if (!(total > 0.0) || !std::isfinite(total)) return fail(SCADLES_EINVAL, "the bounded rates sum to %g", total);
  if (gamma && !(base_batch > 0.0)) return fail(SCADLES_EINVAL, "base_batch must be > 0");
  for (uint32_t j = 0; j < K; ++j) weights[j] = (float)(b[j] / total);
  if (gamma) *gamma = total / base_batch;
  return SCADLES_OK;
}

const char* scadles_last_error(void) { return g_err.c_str(); }

scadles_status scadles_set_option(const char* name, int64_t value)
{
  if (!name) return fail(SCADLES_EINVAL, "option name is NULL");
  if (!strcmp(name, "validate")) g_validate = value ? 1 : 0;
  else if (!strcmp(name, "force_exact")) g_force_exact = value ? 1 : 0;
  else if (!strcmp(name, "force_fallback")) g_force_fallback = value ? 1 : 0;
  else if (!strcmp(name, "inject_count_error")) g_inject_count_error = value ? 1 : 0;
  else if (!strcmp(name, "row_max")) {
    if (value < 0 || value > 0xFFFFFFFFll) return fail(SCADLES_EINVAL, "row_max must be in [0, 2^32 - 1]");
    g_row_max = value;
  }
  else if (!strcmp(name, "row_split")) {
    if (value < 0 || value > 0xFFFFFFFFll) return fail(SCADLES_EINVAL, "row_split must be in [0, 2^32 - 1]");
    g_row_split = value;
  }
  else if (!strcmp(name, "layer_order")) {
    if (value < 0 || value > 2) return fail(SCADLES_EINVAL, "layer_order must be 0, 1 or 2");
    g_layer_order = value;
  }
  else if (!strcmp(name, "parts")) {
    if (value < 1 || value > (int64_t)kMaxParts) return fail(SCADLES_EINVAL, "parts must be in [1, %u]", kMaxParts);
    g_parts = (int)value;
  }
  else return fail(SCADLES_EINVAL, "unknown option '%s'", name);
  return SCADLES_OK;
}

scadles_status scadles_profile_enable(int on)
{
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on && g_prof_pool.empty()) {
    g_prof_pool.resize(kProfMax);
    for (auto& r : g_prof_pool)
      for (auto& e : r.ev)
        if (hipEventCreate(&e) != hipSuccess) {
          g_prof_pool.clear();
          return fail(SCADLES_EHIP, "hipEventCreate failed");
        }
  }
  g_prof_on = on != 0;
  g_prof_used = 0;
  return SCADLES_OK;
}

scadles_status scadles_profile_read(double* stage_ms, uint32_t* calls)
{
  if (!stage_ms || !calls) return fail(SCADLES_EINVAL, "NULL argument");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (int i = 0; i < kStages; ++i) stage_ms[i] = 0.0;
  auto span = [](hipEvent_t a, hipEvent_t b) {
    float ms = 0.f;
    return hipEventElapsedTime(&ms, a, b) == hipSuccess ? (double)ms : 0.0;
  };
  for (size_t r = 0; r < g_prof_used; ++r) {
    const ProfRec& pr = g_prof_pool[r];
    const uint32_t P = pr.parts;
    if (hipEventSynchronize(pr.ev[3 + 2 * P]) != hipSuccess) return fail(SCADLES_EHIP, "hipEventSynchronize failed");
    stage_ms[0] += span(pr.ev[0], pr.ev[1]);
    for (uint32_t i = 0; i < P; ++i) stage_ms[1] += span(pr.ev[i == 0 ? 1 : 1 + 2 * i], pr.ev[3 + 2 * i]);
    stage_ms[2] += span(pr.ev[3 + 2 * (P - 1)], pr.ev[2 + 2 * P]);
    stage_ms[3] += span(pr.ev[2 + 2 * P], pr.ev[3 + 2 * P]);
    stage_ms[4] += span(pr.ev[0], pr.ev[3 + 2 * P]);
  }
  *calls = (uint32_t)g_prof_used;
  g_prof_used = 0;
  return SCADLES_OK;
}

}  // extern "C"
