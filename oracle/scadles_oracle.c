/*
 * scadles_oracle.c -- the CPU oracle of the ScaDLES hot path.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library. The product path
 * (paper_2301_08897_amd) never calls it, and the two share no code.
 *
 * Everything here is the plain definition of what the hot path computes,
 * written for a reader to check against the paper by eye: a full sort for
 * Top-k, serial sums in double in index / device order, no blocking, no
 * fusion, no reordering. Slow on purpose.
 *
 * Paper: Tyagi & Swany, "ScaDLES: Scalable Deep Learning over Streaming data
 * at the Edge", arXiv 2301.08897.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Number of entries kept at compression ratio `ratio` (§V-G: a CR of 0.1 keeps
 * a tenth of the tensor; Top-k "top k%" in §IV). Reading: k = floor(ratio*n)
 * evaluated in double, at least 1 and at most n. 0 flags invalid input.     */
uint64_t oracle_topk_k(uint64_t n, double ratio)
{
  if (n == 0 || n > 0xFFFFFFFFull) return 0;
  if (!(ratio > 0.0) || !(ratio <= 1.0)) return 0; /* also rejects NaN */
  double f = floor(ratio * (double)n);
  uint64_t k = (uint64_t)f;
  if (k < 1) k = 1;
  if (k > n) k = n;
  return k;
}

typedef struct {
  float mag; /* |g_i| */
  uint32_t i;
} mag_index;

/* Order of Top-k: larger magnitude first; equal magnitudes by lower index.
 * fabsf makes -0 and +0 equal. This is a strict total order on the pairs.  */
static int by_magnitude_then_index(const void* pa, const void* pb)
{
  const mag_index* a = (const mag_index*)pa;
  const mag_index* b = (const mag_index*)pb;
  if (a->mag > b->mag) return -1;
  if (a->mag < b->mag) return 1;
  if (a->i < b->i) return -1;
  if (a->i > b->i) return 1;
  return 0;
}

/* Top-k sparsification (§III-C, §IV "High communication cost"): the k entries
 * of largest magnitude, ties to the lower index, returned in ascending index
 * order with their signed values. Also the two energies of the adaptive rule
 * of §IV: e_all = sum g_i^2 over all i, e_kept = the same sum over the kept
 * entries, each summed in double in ascending index order.
 * Returns 0 on success, -1 on bad arguments or allocation failure.         */
int oracle_topk(const float* g, uint64_t n, uint64_t k, uint32_t* idx_out, float* val_out,
                double* e_all, double* e_kept)
{
  if (!g || n == 0 || n > 0xFFFFFFFFull || k < 1 || k > n) return -1;
  mag_index* order = (mag_index*)malloc(n * sizeof(mag_index));
  unsigned char* kept = (unsigned char*)calloc(n, 1);
  if (!order || !kept) {
    free(order);
    free(kept);
    return -1;
  }
  for (uint64_t i = 0; i < n; ++i) {
    order[i].mag = fabsf(g[i]);
    order[i].i = (uint32_t)i;
  }
  qsort(order, n, sizeof(mag_index), by_magnitude_then_index);
  for (uint64_t r = 0; r < k; ++r) kept[order[r].i] = 1;
  free(order);

  uint64_t out = 0;
  double all = 0.0, kep = 0.0;
  for (uint64_t i = 0; i < n; ++i) {
    double x = (double)g[i];
    all += x * x;
    if (kept[i]) {
      kep += x * x;
      if (idx_out) idx_out[out] = (uint32_t)i;
      if (val_out) val_out[out] = g[i];
      ++out;
    }
  }
  free(kept);
  if (e_all) *e_all = all;
  if (e_kept) *e_kept = kep;
  return out == k ? 0 : -1;
}

/* Per-layer Top-k: the reading of the Top-k of §IV in which every layer of the
 * model keeps its own top fraction. The gradient is cut into L layers, layer l
 * being positions [seg_off[l], seg_off[l+1]); each layer keeps its
 * oracle_topk_k(layer size, ratio) entries of largest magnitude (ties to the
 * lower index) among its own entries only. The kept set is the union over the
 * layers, written in ascending index order; e_all and e_kept are the energies
 * of the whole gradient, summed in ascending index order as in oracle_topk.
 * *k_out receives the total kept. Returns 0, or -1 on bad arguments.        */
int oracle_topk_layers(const float* g, const uint64_t* seg_off, uint32_t L, double ratio,
                       uint32_t* idx_out, float* val_out, double* e_all, double* e_kept, uint64_t* k_out)
{
  if (!g || !seg_off || L == 0 || seg_off[0] != 0 || seg_off[L] > 0xFFFFFFFFull) return -1;
  uint64_t at = 0;
  for (uint32_t l = 0; l < L; ++l) {
    if (seg_off[l + 1] <= seg_off[l]) return -1;
    uint64_t n_l = seg_off[l + 1] - seg_off[l];
    uint64_t k_l = oracle_topk_k(n_l, ratio);
    if (k_l == 0) return -1;
    /* the layer on its own: positions relative to its start */
    if (oracle_topk(g + seg_off[l], n_l, k_l, idx_out ? idx_out + at : NULL, val_out ? val_out + at : NULL,
                    NULL, NULL) != 0)
      return -1;
    if (idx_out)
      for (uint64_t r = 0; r < k_l; ++r) idx_out[at + r] += (uint32_t)seg_off[l];
    at += k_l;
  }
  if (k_out) *k_out = at;
  double all = 0.0, kep = 0.0;
  for (uint64_t i = 0; i < seg_off[L]; ++i) all += (double)g[i] * (double)g[i];
  if (val_out)
    for (uint64_t r = 0; r < at; ++r) kep += (double)val_out[r] * (double)val_out[r];
  if (e_all) *e_all = all;
  if (e_kept) *e_kept = kep;
  return 0;
}

/* The adaptive compression rule of §IV: send Top-k(g) when
 * | ||g||^2 - ||Top-k(g)||^2 | / ||g||^2 <= delta, else send g. A zero
 * gradient loses nothing (ratio 0). Returns 1 for "send Top-k", 0 for
 * "send g"; *loss receives the ratio.                                       */
int oracle_compress_decision(double e_all, double e_kept, double delta, double* loss)
{
  double rho = (e_all == 0.0) ? 0.0 : fabs(e_all - e_kept) / e_all;
  if (loss) *loss = rho;
  return rho <= delta ? 1 : 0;
}

/* Adaptive compression with the moving average of §IV (the energies of the
 * compressed and uncompressed gradients tracked as an exponentially weighted
 * moving average) and the accounting of §V-G (CNC ratio, floats sent). The
 * paper gives no smoothing factor, so beta is a parameter; beta = 0 is the
 * instantaneous rule. state[0..1] are one device's smoothed E_all and E_kept;
 * both zero means no history, and that iteration takes its energies as they
 * are. Otherwise each is replaced by beta * state + (1 - beta) * E, evaluated
 * in double. The rule of §IV is then applied to the smoothed pair.
 * counters (or NULL): [0] iterations that sent Top-k, [1] iterations, [2]
 * floats sent (k when compressed, n otherwise: the update's values, which is
 * what §V-G counts). Returns 1 to send Top-k, 0 to send the dense gradient.  */
int oracle_adaptive_step(double* state, uint64_t* counters, double e_all, double e_kept, double beta,
                         double delta, uint64_t k, uint64_t n)
{
  if (state[0] == 0.0 && state[1] == 0.0) {
    state[0] = e_all;
    state[1] = e_kept;
  } else {
    state[0] = beta * state[0] + (1.0 - beta) * e_all;
    state[1] = beta * state[1] + (1.0 - beta) * e_kept;
  }
  const int send = oracle_compress_decision(state[0], state[1], delta, NULL);
  if (counters) {
    counters[0] += (uint64_t)send;
    counters[1] += 1;
    counters[2] += send ? k : n;
  }
  return send;
}

/* Weighted aggregation, Eqn 4b: out[i] = sum_{j=0..K-1} w_j * v_j(i), where
 * v_j(i) is device j's value at i if i is one of its k_j kept positions and 0
 * otherwise. idx[j] == NULL marks a device that sent its dense gradient
 * (k[j] must then be n and val[j] holds n values). Accumulated in double in
 * device order, rounded to float once at the end.
 * Returns 0, or -1 on bad arguments.                                        */
int oracle_aggregate(uint32_t K, uint64_t n, const uint32_t* const* idx, const float* const* val,
                     const uint64_t* k, const float* w, float* out)
{
  if (K == 0 || n == 0 || !val || !k || !w || !out) return -1;
  double* acc = (double*)calloc(n, sizeof(double));
  if (!acc) return -1;
  for (uint32_t j = 0; j < K; ++j) {
    double wj = (double)w[j];
    if (idx == NULL || idx[j] == NULL) {
      if (k[j] != n) {
        free(acc);
        return -1;
      }
      for (uint64_t i = 0; i < n; ++i) acc[i] += wj * (double)val[j][i];
    } else {
      for (uint64_t t = 0; t < k[j]; ++t) {
        uint32_t i = idx[j][t];
        if (i >= n) {
          free(acc);
          return -1;
        }
        acc[i] += wj * (double)val[j][t];
      }
    }
  }
  for (uint64_t i = 0; i < n; ++i) out[i] = (float)acc[i];
  free(acc);
  return 0;
}

/* SGD update, Eqn 4c: w <- w - eta_scaled * g~, in double, rounded to float. */
void oracle_sgd(float* p, const float* g, uint64_t n, float lr)
{
  for (uint64_t i = 0; i < n; ++i) p[i] = (float)((double)p[i] - (double)lr * (double)g[i]);
}

/* Momentum SGD with weight decay after the aggregation: the optimizer of the
 * paper's evaluation (§V, training setup: momentum 0.9 with weight decay
 * 1e-4 for ResNet152 and 5e-4 for VGG19) applied to the aggregate of Eqn 4b
 * in place of the plain step of Eqn 4c. The usual formulation without
 * dampening or Nesterov: d = g + wd * w; v <- mu * v + d; w <- w - eta * v.
 * Every step is evaluated in double and every stored value rounded to float
 * once: v is stored as float and that float is the one the parameter update
 * uses. A zero v gives v = d on the first step; mu = wd = 0 is Eqn 4c.      */
void oracle_momentum_sgd(float* p, float* v, const float* g, uint64_t n, float lr, float mu, float wd)
{
  for (uint64_t i = 0; i < n; ++i) {
    const double d = (double)g[i] + (double)wd * (double)p[i];
    v[i] = (float)((double)mu * (double)v[i] + d);
    p[i] = (float)((double)p[i] - (double)lr * (double)v[i]);
  }
}

/* Weights and learning-rate scale from streaming rates (§IV "Heterogeneous
 * streams"): batch b_j = S_j bounded to [b_min, b_max]; Eqn 4a
 * r_j = b_j / sum b (so sum r = 1); linear scaling gamma = sum b / B.
 * Returns 0, or -1 on bad input (negative or non-finite rate, empty sum).  */
int oracle_stream_weights(const double* rates, uint32_t K, double b_min, double b_max,
                          double base_batch, float* w, double* gamma)
{
  if (!rates || K == 0 || !w || !(b_min <= b_max)) return -1;
  double* b = (double*)malloc(K * sizeof(double));
  if (!b) return -1;
  double total = 0.0;
  for (uint32_t j = 0; j < K; ++j) {
    double s = rates[j];
    if (!isfinite(s) || s < 0.0) {
      free(b);
      return -1;
    }
    if (s < b_min) s = b_min;
    if (s > b_max) s = b_max;
    b[j] = s;
    total += s;
  }
  if (!(total > 0.0) || !isfinite(total)) {
    free(b);
    return -1;
  }
  for (uint32_t j = 0; j < K; ++j) w[j] = (float)(b[j] / total);
  if (gamma) {
    if (!(base_batch > 0.0)) {
      free(b);
      return -1;
    }
    *gamma = total / base_batch;
  }
  free(b);
  return 0;
}

/* Streaming buffers of K devices over T training iterations (§II-C, Eqn 2;
 * §IV "Limited memory and storage": the persistence and truncation policies;
 * §IV "Heterogeneous streams": the batch rule b = S bounded to [b_min, b_max]).
 * Device j streams rate[j] samples per second; one iteration lasts iter_us[j]
 * microseconds. Iteration 0 starts with one second of arrivals in the buffer
 * (rate[j] samples; Eqn 2 at T = 0). Every iteration, in this order:
 *   1. the device trains on min(b_j, queued) samples, the oldest ones;
 *   2. the samples that arrived during the iteration are added: the count of
 *      arrivals up to the end of iteration T is floor(rate * iter_us * T / 10^6)
 *      (a continuous stream), the difference of two such counts per iteration;
 *   3. persistence keeps every sample; truncation discards the residual of
 *      step 1 and keeps at most rate[j] of the new arrivals (the newest ones).
 * queued[(T'+1) x K]: buffer occupancy before iteration T' (row 0) and after
 * the last one (row T); batch[T x K]: samples trained on; dropped[K]: samples
 * discarded by truncation over the run. Any output may be NULL.
 * policy 0 = persistence, 1 = truncation. Returns 0, or -1 on bad input.  */
int oracle_stream_run(uint32_t K, const uint64_t* rate, const uint64_t* iter_us, uint64_t b_min, uint64_t b_max,
                      int policy, uint64_t T, uint64_t* queued, uint64_t* batch, uint64_t* dropped)
{
  if (K == 0 || !rate || !iter_us || b_min > b_max || (policy != 0 && policy != 1)) return -1;
  for (uint32_t j = 0; j < K; ++j) {
    if (rate[j] > 0xFFFFFFFFull || iter_us[j] > 0xFFFFFFFFull) return -1;
    uint64_t b = rate[j];
    if (b < b_min) b = b_min;
    if (b > b_max) b = b_max;
    uint64_t q = rate[j];
    uint64_t lost = 0;
    if (queued) queued[j] = q;
    for (uint64_t t = 0; t < T; ++t) {
      uint64_t used = b < q ? b : q;
      q -= used;
      if (batch) batch[t * K + j] = used;
      /* arrivals during iteration t, from the cumulative count of a continuous stream */
      unsigned __int128 before = (unsigned __int128)rate[j] * iter_us[j] * t / 1000000u;
      unsigned __int128 after = (unsigned __int128)rate[j] * iter_us[j] * (t + 1) / 1000000u;
      uint64_t arrived = (uint64_t)(after - before);
      if (policy == 0) {
        q += arrived;
      } else {
        lost += q;
        q = arrived < rate[j] ? arrived : rate[j];
        lost += arrived - q;
      }
      if (queued) queued[(t + 1) * K + j] = q;
    }
    if (dropped) dropped[j] = lost;
  }
  return 0;
}
