// stream.hip -- the streaming buffers of the devices and what each iteration
// takes from them: batch sizes, Eqn 4a weights and the learning-rate scale
// (§II-C Eqns 2-3, §IV). Host only: nothing here touches GPU state.
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "scadles.h"

namespace scadles {
scadles_status fail(scadles_status st, const char* fmt, ...);
}
using scadles::fail;

namespace {

constexpr uint64_t kUsPerSecond = 1000000;
constexpr uint64_t kMaxRate = 0xFFFFFFFFull;

// Samples a continuous stream of `rate` samples/s has delivered after `us`
// microseconds: floor(rate * us / 10^6), as rate * whole seconds plus the
// part of the last second (exact; rate < 2^32 keeps both products in range).
inline uint64_t delivered(uint64_t rate, uint64_t us)
{
  return rate * (us / kUsPerSecond) + rate * (us % kUsPerSecond) / kUsPerSecond;
}

inline uint64_t batch_of(uint64_t rate, uint64_t b_min, uint64_t b_max)
{
  return rate < b_min ? b_min : (rate > b_max ? b_max : rate);
}

scadles_status check_common(uint32_t K, uint64_t b_min, uint64_t b_max, int policy)
{
  if (K == 0) return fail(SCADLES_EINVAL, "K must be >= 1");
  if (b_min > b_max) return fail(SCADLES_EINVAL, "need b_min <= b_max");
  if (policy != SCADLES_PERSISTENCE && policy != SCADLES_TRUNCATION)
    return fail(SCADLES_EINVAL, "unknown buffer policy %d", policy);
  return SCADLES_OK;
}

// Takes the batch from the buffer; returns it.
inline uint64_t take_batch(scadles_stream& s, uint64_t b_min, uint64_t b_max)
{
  const uint64_t b = batch_of(s.rate, b_min, b_max);
  const uint64_t used = b < s.queued ? b : s.queued;
  s.queued -= used;
  s.trained += used;
  return used;
}

// Adds the arrivals of an iteration of `us` microseconds under the policy.
inline void arrive(scadles_stream& s, uint64_t us, int policy)
{
  const uint64_t a = delivered(s.rate, s.elapsed_us + us) - delivered(s.rate, s.elapsed_us);
  s.elapsed_us += us;
  if (policy == SCADLES_PERSISTENCE) {
    s.queued += a;
    return;
  }
  const uint64_t keep = a < s.rate ? a : s.rate;  // the newest samples, at most one second's worth
  s.dropped += s.queued + (a - keep);
  s.queued = keep;
}

}  // namespace

extern "C" {

scadles_status scadles_stream_init(uint32_t K, const uint64_t* rate, scadles_stream* st)
{
  if (K == 0 || !rate || !st) return fail(SCADLES_EINVAL, "rate and st must not be NULL, K >= 1");
  for (uint32_t j = 0; j < K; ++j)
    if (rate[j] > kMaxRate) return fail(SCADLES_EINVAL, "rate %u exceeds 2^32 - 1", j);
  for (uint32_t j = 0; j < K; ++j) st[j] = scadles_stream{rate[j], 0, rate[j], 0, 0};
  return SCADLES_OK;
}

scadles_status scadles_stream_iteration(uint32_t K, scadles_stream* st, const uint64_t* iter_us, uint64_t b_min,
                                        uint64_t b_max, int policy, double base_batch, uint64_t* batch,
                                        float* weights, double* gamma)
{
  if (scadles_status e = check_common(K, b_min, b_max, policy)) return e;
  if (!st || !iter_us) return fail(SCADLES_EINVAL, "st and iter_us must not be NULL");
  if (gamma && !(base_batch > 0.0 && std::isfinite(base_batch)))
    return fail(SCADLES_EINVAL, "base_batch must be finite and > 0");
  for (uint32_t j = 0; j < K; ++j) {
    if (st[j].rate > kMaxRate) return fail(SCADLES_EINVAL, "st[%u] has a rate above 2^32 - 1", j);
    if (iter_us[j] > kMaxRate) return fail(SCADLES_EINVAL, "iter_us[%u] exceeds 2^32 - 1", j);
    if (st[j].elapsed_us > std::numeric_limits<uint64_t>::max() - iter_us[j])
      return fail(SCADLES_EINVAL, "st[%u]: stream time overflows", j);
  }
  std::vector<uint64_t> used(K);
  double total = 0.0;
  for (uint32_t j = 0; j < K; ++j) {
    used[j] = take_batch(st[j], b_min, b_max);
    total += (double)used[j];
  }
  if (batch)
    for (uint32_t j = 0; j < K; ++j) batch[j] = used[j];
  if (weights || gamma) {
    if (total > 0.0) {
      std::vector<double> r(used.begin(), used.end());
      const double inf = std::numeric_limits<double>::infinity();
      float* w = weights;
      std::vector<float> scratch;
      if (!w) {
        scratch.resize(K);
        w = scratch.data();
      }
      // the same rule as for rates, on the batches actually trained on
      if (scadles_status e = scadles_stream_weights(r.data(), K, 0.0, inf, gamma ? base_batch : 1.0, w, gamma))
        return e;
    } else {
      if (weights)
        for (uint32_t j = 0; j < K; ++j) weights[j] = 0.0f;
      if (gamma) *gamma = 0.0;
    }
  }
  for (uint32_t j = 0; j < K; ++j) arrive(st[j], iter_us[j], policy);
  return SCADLES_OK;
}

scadles_status scadles_stream_simulate(uint32_t K, const uint64_t* rate, const uint64_t* iter_us, uint64_t b_min,
                                       uint64_t b_max, int policy, uint64_t T, uint64_t* queued, uint64_t* batch,
                                       uint64_t* dropped)
{
  if (scadles_status e = check_common(K, b_min, b_max, policy)) return e;
  if (!rate || !iter_us) return fail(SCADLES_EINVAL, "rate and iter_us must not be NULL");
  for (uint32_t j = 0; j < K; ++j)
    if (iter_us[j] > kMaxRate) return fail(SCADLES_EINVAL, "iter_us[%u] exceeds 2^32 - 1", j);
  std::vector<scadles_stream> st(K);
  if (scadles_status e = scadles_stream_init(K, rate, st.data())) return e;
  if (T > 0 && (queued || batch)) {
    const uint64_t rows = (queued ? T + 1 : T);
    if (rows > std::numeric_limits<uint64_t>::max() / K / sizeof(uint64_t))
      return fail(SCADLES_EINVAL, "T x K outputs overflow the address space");
  }
  if (queued)
    for (uint32_t j = 0; j < K; ++j) queued[j] = st[j].queued;
  for (uint64_t t = 0; t < T; ++t) {
    for (uint32_t j = 0; j < K; ++j) {
      const uint64_t used = take_batch(st[j], b_min, b_max);
      if (batch) batch[t * K + j] = used;
      arrive(st[j], iter_us[j], policy);
      if (queued) queued[(t + 1) * K + j] = st[j].queued;
    }
  }
  if (dropped)
    for (uint32_t j = 0; j < K; ++j) dropped[j] = st[j].dropped;
  return SCADLES_OK;
}

}  // extern "C"
