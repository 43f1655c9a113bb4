/*
 * scadles.h -- C ABI of the ScaDLES data-parallel hot path on MI355X (gfx950).
 *
 * The hot path of one training step of ScaDLES (Tyagi & Swany, "ScaDLES:
 * Scalable Deep Learning over Streaming data at the Edge", arXiv 2301.08897):
 * K simulated edge devices each hold a flat fp32 gradient of n elements in the
 * HBM of one GPU. For every device the library
 *   1. keeps the Top-k entries by magnitude (Top-k sparsification, §III-C and
 *      §IV "High communication cost"), ties broken towards the lower index,
 *      with k = clamp(floor(ratio * n), 1, n) (compression ratio CR, §V-G);
 *   2. measures the energies ||g||^2 and ||Top-k(g)||^2 that drive the
 *      adaptive compression rule of §IV (send Top-k(g) when the relative
 *      energy loss is at most delta, else send g);
 * then
 *   3. aggregates all devices' (sparse or dense) gradients weighted by each
 *      device's streaming rate, g~ = sum_j r_j g_j (Eqn 4b, weights of Eqn 4a);
 *   4. applies the SGD update w <- w - eta_scaled * g~ (Eqn 4c).
 *
 * Conventions for every entry point:
 *   - Pointers marked (dev) are device pointers owned by the caller; the
 *     library never frees or retains them. Pointers marked (host) are host
 *     memory read during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Every device-side effect is asynchronous on that stream; outputs are
 *     valid once the stream has been synchronised.
 *   - No entry point allocates device memory. Scratch space is the
 *     caller-provided workspace `ws` of `ws_bytes` bytes (dev, 256-byte
 *     aligned), sized by the matching *_workspace_bytes() query. A workspace
 *     must not be shared by calls that may run concurrently.
 *   - All arguments are validated on the host before anything is launched; an
 *     invalid call returns a non-zero scadles_status, launches nothing, and
 *     scadles_last_error() describes the problem.
 *   - Gradients must be finite (NaN/Inf give unspecified results, never a
 *     memory fault). Magnitude ranking uses the 31-bit key bits(g) & 0x7FFFFFFF,
 *     so -0 and +0 rank equal and denormals are ranked exactly (no flushing).
 *   - Results are deterministic: re-running a call on the same inputs gives
 *     bit-identical outputs.
 */
#ifndef SCADLES_H
#define SCADLES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SCADLES_OK = 0,
  SCADLES_EINVAL = 1,      /* invalid argument (NULL pointer, size, ratio, weight ...) */
  SCADLES_EWORKSPACE = 2,  /* workspace NULL, misaligned or smaller than required     */
  SCADLES_EHIP = 3,        /* the HIP runtime reported an error while launching        */
  SCADLES_EUNSORTED = 4,   /* validation mode only: a sparse set's idx is not strictly
                              ascending or holds an entry >= n                          */
  SCADLES_EINTERNAL = 5    /* validation mode only: an internal consistency check of a
                              selection failed (a radix pass missed, the threshold was
                              not found, or the kept count is not k)                   */
} scadles_status;

/* Largest number of devices one call accepts. */
#define SCADLES_MAX_DEVICES 64

/* One device's contribution to the weighted aggregation (Eqn 4b).
 * Sparse: idx (dev, k entries, strictly ascending, each < n) and val (dev, k
 * entries) hold the kept gradient entries; every other position is zero.
 * Dense: idx == NULL and k == n; val (dev, n entries) is the full gradient.
 * Empty: k == 0 (idx and val are ignored and may be NULL); contributes nothing.
 * idx and val must be 4-byte aligned.                                        */
typedef struct {
  const uint32_t* idx;
  const float* val;
  uint64_t k;
} scadles_sparse;

/* Number of entries Top-k keeps for a vector of n elements at compression
 * ratio `ratio` (§V-G: CR 0.1 keeps a tenth of the entries):
 * k = clamp(floor(ratio * n), 1, n), computed in IEEE double.
 * Returns 0 when n == 0, n > 2^32 - 1 or ratio is not in (0, 1].            */
uint64_t scadles_topk_k(uint64_t n, double ratio);

/* Workspace bytes needed by scadles_step_fused for K devices of n elements at
 * the given per-device compression ratios (host[K]); scadles_topk_select uses
 * K = 1. Returns 0 for arguments the calls would reject.                    */
size_t scadles_workspace_bytes(uint32_t K, uint64_t n, const double* ratios);

/* Workspace bytes needed by scadles_weighted_aggregate for K sets over n
 * positions. Returns 0 for arguments the call would reject.                 */
size_t scadles_aggregate_workspace_bytes(uint32_t K, uint64_t n);

/* Top-k sparsification of one gradient (§IV "High communication cost";
 * Top-k as in §III-C), with the energies of the adaptive rule.
 *   grad      (dev, n floats, 4-byte aligned) the gradient; not modified.
 *   n         1 <= n <= 2^32 - 1.
 *   ratio     compression ratio in (0, 1]; k = scadles_topk_k(n, ratio).
 *   idx, val  (dev, k entries each) receive the kept positions in strictly
 *             ascending order and their signed values (bit copies of grad).
 *             The kept set holds the k largest |grad|; among equal magnitudes
 *             the lower index is kept.
 *   energies  (dev, 2 doubles) or NULL: receives sum grad^2 and the sum over
 *             the kept entries, both accumulated in double.
 * Returns SCADLES_EINVAL for a NULL or misaligned pointer, n out of range or
 * a ratio outside (0, 1]; SCADLES_EWORKSPACE for an undersized workspace.   */
scadles_status scadles_topk_select(const float* grad, uint64_t n, double ratio,
                                   uint32_t* idx, float* val, double* energies,
                                   void* ws, size_t ws_bytes, void* stream);

/* scadles_topk_select without a workspace argument and without allocating,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation). The
 * workspace is a static array of SCADLES_NOALLOC_SCRATCH_BYTES bytes that the
 * library holds on every GPU it runs on until the process ends; its address is
 * looked up once per GPU, on the first call there. The call allocates nothing
 * and launches the same kernels as scadles_topk_select, with the same
 * results, and clears the parts of the scratch that must start at zero.
 * Every call on one GPU shares that GPU's scratch: calls that may overlap on
 * one GPU (several host threads, or streams that do not order them) race and
 * give unspecified results; order them on one stream. Arguments and errors as
 * for scadles_topk_select; in addition SCADLES_EWORKSPACE when the selection
 * needs more scratch than the maximum (scadles_workspace_bytes(1, n, &ratio) >
 * SCADLES_NOALLOC_SCRATCH_BYTES; e.g. a gradient of 143,667,240 elements fits
 * at ratio 0.01 but not at 0.1). The first call on a GPU may return
 * SCADLES_EHIP if the scratch address cannot be looked up.               */
#define SCADLES_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
scadles_status scadles_topk_select_noalloc(const float* grad, uint64_t n, double ratio,
                                           uint32_t* idx, float* val, double* energies,
                                           void* stream);

/* Per-layer Top-k: the per-layer reading of the Top-k sparsification of §IV
 * (each layer of the model keeps its own top fraction) for K devices whose
 * flat gradients share one layer layout. Layer l is positions
 * [seg_off[l], seg_off[l+1]) of every gradient and keeps k_l =
 * scadles_topk_k(seg_off[l+1] - seg_off[l], ratio_j) entries of device j,
 * chosen as scadles_topk_select chooses them within the layer. Device j's
 * kept set is the union over its layers, written in ascending index order
 * (layer after layer, indices relative to the whole gradient) to idx[j] /
 * val[j]: scadles_layers_k(seg_off, L, ratio_j) entries.
 *   grads     (host[K] of dev pointers, seg_off[L] floats each, 4-byte aligned).
 *   seg_off   (host[L+1]) 0 = seg_off[0] < seg_off[1] < ... < seg_off[L] <= 2^32 - 1;
 *             1 <= L <= 2^24.
 *   ratios    (host[K]) in (0, 1].
 *   idx, val  (host[K] of dev pointers, 4-byte aligned).
 *   energies  (dev, 2K doubles) or NULL: E_all and E_kept of each whole gradient.
 *   ws        scadles_layers_workspace_bytes(K, seg_off, L, ratios) bytes.
 * Layers of at most "row_max" elements (scadles_set_option) are selected as
 * (device, layer) rows, all at once: one workgroup per row, or, for rows of
 * more than "row_split" elements, one workgroup per 16384-element part of the
 * row in each of its passes. Longer layers are selected by the selection of
 * scadles_topk_select, one layer after the other, overlapped with each other
 * on a second and third stream the library creates per GPU (default
 * priority; those streams start after the caller's earlier work on `stream`,
 * and the caller's stream waits for them before the call's work ends on it).
 * Results do not depend on these splits. Feed the sets to
 * scadles_weighted_aggregate for Eqn 4b, or use scadles_step_fused_layers.
 * Same error convention as above.                                           */
uint64_t scadles_layers_k(const uint64_t* seg_off, uint32_t L, double ratio);
size_t scadles_layers_workspace_bytes(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios);
scadles_status scadles_topk_select_layers(const float* const* grads, uint32_t K, const uint64_t* seg_off,
                                          uint32_t L, const double* ratios, uint32_t* const* idx,
                                          float* const* val, double* energies, void* ws, size_t ws_bytes,
                                          void* stream);

/* Weighted aggregation of K devices' contributions (Eqn 4b):
 *   dense[i] = sum over j = 0..K-1, in that order, of w_j * v_j(i)
 * where v_j(i) is device j's value at i (zero when i is not in a sparse set).
 * The sum is accumulated in double with one fused multiply-add per term and
 * rounded to float once, so the result does not depend on the launch shape.
 *   sets     (host[K]) the contributions, see scadles_sparse.
 *   weights  (host[K]) r_j of Eqn 4a: finite, >= 0, summing to 1 within
 *            K * 2^-23.
 *   dense    (dev, n floats, 16-byte aligned) overwritten; +0 where no device
 *            contributes.
 * Returns SCADLES_EINVAL for bad arguments; with the "validate" option set it
 * also synchronises `stream` and returns SCADLES_EUNSORTED if a set's idx is
 * not strictly ascending or reaches n. Without it such input gives
 * unspecified values (never an out-of-bounds access).                       */
scadles_status scadles_weighted_aggregate(const scadles_sparse* sets, const float* weights,
                                          uint32_t K, uint64_t n, float* dense,
                                          void* ws, size_t ws_bytes, void* stream);

/* SGD update (Eqn 4c): params[i] <- params[i] - lr * grad[i], evaluated as
 * one fused multiply-add in double and rounded to float once.
 *   params (dev, n floats) updated in place; grad (dev, n floats), may not
 *   alias params. Both 16-byte aligned. lr finite.                          */
scadles_status scadles_apply_sgd(float* params, const float* grad, uint64_t n, float lr,
                                 void* stream);

/* Momentum SGD with weight decay: the optimizer of the paper's evaluation
 * (§V training setup: momentum 0.9, weight decay 1e-4 for ResNet152 and
 * 5e-4 for VGG19), applied in place of the plain step of Eqn 4c. Per
 * element, without dampening or Nesterov:
 *   d         = grad[i] + weight_decay * params[i]
 *   buf[i]    = momentum * buf[i] + d
 *   params[i] = params[i] - lr * buf[i]     (with the buf[i] just stored)
 * Each line is evaluated in double as one fused multiply-add (every product
 * of two floats is exact in double) and rounded to float once. A zero-filled
 * buf gives buf = d on the first step; momentum = weight_decay = 0 is Eqn 4c.
 *   params, momentum_buf (dev, n floats) updated in place; grad (dev, n
 *   floats). All 16-byte aligned, no two overlapping. lr, momentum and
 *   weight_decay finite.                                                    */
scadles_status scadles_apply_momentum_sgd(float* params, float* momentum_buf, const float* grad, uint64_t n,
                                          float lr, float momentum, float weight_decay, void* stream);

/* One whole hot-path step for K devices in one call (the training step of
 * §IV): Top-k + energies for every device, the adaptive decision, weighted
 * aggregation and, optionally, the SGD update.
 *   grads      (host[K] of dev pointers, n floats each, 4-byte aligned).
 *   ratios     (host[K]) per-device compression ratio in (0, 1].
 *   delta      compression threshold of §IV: device j sends Top-k(g_j) when
 *              |E_all - E_kept| / E_all <= delta (E_all == 0 counts as 0) and
 *              its dense gradient otherwise. +INFINITY always compresses.
 *   weights    (host[K]) as for scadles_weighted_aggregate.
 *   idx, val   (host[K] of dev pointers) per-device outputs of k_j entries,
 *              exactly as scadles_topk_select writes them (always written,
 *              whatever the decision).
 *   dense      (dev, n floats, 16-byte aligned) receives g~ of Eqn 4b.
 *   energies   (dev, 2K doubles) or NULL: E_all and E_kept per device.
 *   compressed (dev, K bytes) or NULL: 1 if the device sent Top-k, else 0.
 *   params     (dev, n floats, 16-byte aligned) or NULL: when non-NULL the
 *              SGD update of Eqn 4c with learning rate lr is applied to it
 *              using the float g~ written to dense.
 * K <= SCADLES_MAX_DEVICES. Same error convention as above.                 */
scadles_status scadles_step_fused(const float* const* grads, uint32_t K, uint64_t n,
                                  const double* ratios, double delta, const float* weights,
                                  uint32_t* const* idx, float* const* val, float* dense,
                                  double* energies, uint8_t* compressed,
                                  float* params, float lr,
                                  void* ws, size_t ws_bytes, void* stream);

/* Options of scadles_step_fused_ex; an all-zero struct gives exactly
 * scadles_step_fused.
 *   momentum_buf  (dev, n floats, 16-byte aligned, not overlapping params or
 *                 dense) or NULL. When set, the update after the aggregation
 *                 is the momentum SGD of scadles_apply_momentum_sgd with
 *                 `momentum` and `weight_decay` (finite) in place of Eqn 4c,
 *                 computed from the float g~ written to dense; params is
 *                 then required.
 *   ewma          (dev, 2K doubles, 8-byte aligned) or NULL. When set, the
 *                 adaptive rule of §IV is applied to moving averages of each
 *                 device's energies kept here (the paper tracks them as an
 *                 exponentially weighted moving average but prints no
 *                 factor): ewma[2j], ewma[2j+1] <- ewma_beta * ewma + (1 -
 *                 ewma_beta) * (E_all, E_kept), in double; a device whose
 *                 pair is (0, 0) has no history and takes its energies as they
 *                 are. Zero-fill before the first step. ewma_beta in [0, 1);
 *                 0 is the instantaneous rule.
 *   counters      (dev, 3K uint64, 8-byte aligned) or NULL. When set, each
 *                 call adds per device j: counters[3j] += 1 if it sent Top-k,
 *                 counters[3j+1] += 1, counters[3j+2] += k_j if it sent
 *                 Top-k else n (floats sent; values only, as §V-G counts
 *                 them). The CNC ratio of §V-G is counters[3j] /
 *                 counters[3j+1].                                           */
typedef struct scadles_step_options {
  float* momentum_buf;
  float momentum;
  float weight_decay;
  double* ewma;
  double ewma_beta;
  uint64_t* counters;
} scadles_step_options;

/* scadles_step_fused with the options above (momentum SGD, moving-average
 * adaptive rule, CNC and floats-sent accounting). options must not be NULL.
 * Other arguments and errors as for scadles_step_fused.                    */
scadles_status scadles_step_fused_ex(const float* const* grads, uint32_t K, uint64_t n,
                                     const double* ratios, double delta, const float* weights,
                                     uint32_t* const* idx, float* const* val, float* dense,
                                     double* energies, uint8_t* compressed, float* params, float lr,
                                     const scadles_step_options* options, void* ws, size_t ws_bytes,
                                     void* stream);

/* The fused step with the per-layer Top-k: scadles_topk_select_layers for
 * every device, the adaptive rule of §IV on each device's whole-gradient
 * energies (with the moving average and accounting of `options`, which may
 * be NULL), then Eqn 4b over the layered sets (or the dense gradients of
 * devices that send g) and the update (Eqn 4c, or momentum SGD when
 * options->momentum_buf is set), as scadles_step_fused_ex does for the
 * whole-vector Top-k. idx[j] / val[j] hold scadles_layers_k(seg_off, L,
 * ratios[j]) entries; dense, params and the options as for
 * scadles_step_fused_ex; ws is scadles_step_layers_workspace_bytes(...) bytes.
 * Same error convention as above.                                           */
size_t scadles_step_layers_workspace_bytes(uint32_t K, const uint64_t* seg_off, uint32_t L, const double* ratios);
scadles_status scadles_step_fused_layers(const float* const* grads, uint32_t K, const uint64_t* seg_off, uint32_t L,
                                         const double* ratios, double delta, const float* weights,
                                         uint32_t* const* idx, float* const* val, float* dense, double* energies,
                                         uint8_t* compressed, float* params, float lr,
                                         const scadles_step_options* options, void* ws, size_t ws_bytes,
                                         void* stream);

/* Aggregation weights and learning-rate scale from streaming rates
 * (§IV "Heterogeneous streams", Eqn 4a and the linear scaling rule):
 *   b_j = clamp(S_j, b_min, b_max)   (batch bounded to [b_min, b_max]),
 *   r_j = b_j / sum_i b_i            (computed in double, stored as float),
 *   gamma = sum_i b_i / base_batch   (eta_scaled = gamma * eta).
 *   rates   (host[K]) S_j, finite and >= 0, not all zero after clamping.
 *   b_min <= b_max; pass 0 and +INFINITY for no bounds.
 *   weights (host[K]) receives r_j. gamma (host) may be NULL; if not,
 *   base_batch must be > 0.
 * Host-only; touches no GPU state.                                          */
scadles_status scadles_stream_weights(const double* rates, uint32_t K, double b_min,
                                      double b_max, double base_batch, float* weights,
                                      double* gamma);

/* ---- streaming buffers, batch sizes, weights and learning-rate scale --------
 * The step before the aggregation (§II-C, Eqns 2 and 3; §IV "Heterogeneous
 * streams" and "Limited memory and storage"): device j receives a continuous
 * stream of S_j samples per second into its buffer and trains one iteration
 * of t_j seconds on a batch of b_j = clamp(S_j, b_min, b_max) samples, or on
 * all it holds when that is fewer. After an iteration the samples that
 * arrived meanwhile join the buffer. Stream persistence keeps every sample;
 * stream truncation discards the residual the iteration left and keeps at
 * most S_j of the new arrivals (the newest), so its buffer stays O(S_j)
 * while persistence grows as (t_j S_j - b_j) T + S_j after T iterations
 * (Eqn 2). A continuous stream has delivered floor(S_j * us / 10^6) samples
 * after `us` microseconds; a buffer starts with one second of it (S_j).
 * Host-only: none of these calls touches GPU state.                         */
#define SCADLES_PERSISTENCE 0
#define SCADLES_TRUNCATION 1

/* One device's stream buffer. */
typedef struct scadles_stream {
  uint64_t rate;        /* S_j, samples per second, < 2^32                      */
  uint64_t elapsed_us;  /* stream time covered by the iterations so far         */
  uint64_t queued;      /* samples in the buffer                                */
  uint64_t trained;     /* samples trained on so far                            */
  uint64_t dropped;     /* samples discarded by truncation so far               */
} scadles_stream;

/* Sets st[j] to a fresh buffer of stream rate rate[j] (queued = rate[j]).
 *   rate (host[K]) < 2^32; st (host[K]).                                    */
scadles_status scadles_stream_init(uint32_t K, const uint64_t* rate, scadles_stream* st);

/* One training iteration of K devices: every device takes its batch from its
 * buffer (batch[j] = min(clamp(S_j, b_min, b_max), queued)), the weights and
 * learning-rate scale of that iteration follow from the batches as in
 * scadles_stream_weights (r_j = batch_j / sum batch, Eqn 4a; gamma = sum
 * batch / base_batch), then the arrivals of iter_us[j] microseconds join the
 * buffer under `policy`.
 *   st       (host[K], in/out) from scadles_stream_init.
 *   iter_us  (host[K]) this iteration's duration per device, < 2^32.
 *   b_min <= b_max (UINT64_MAX: no upper bound). policy: SCADLES_PERSISTENCE
 *   or SCADLES_TRUNCATION. base_batch > 0 when gamma is not NULL.
 *   batch (host[K]) or NULL; weights (host[K]) or NULL; gamma or NULL.
 * When no device holds a sample, weights are all 0 and gamma is 0 (there is
 * nothing to aggregate). Errors leave st unchanged.                        */
scadles_status scadles_stream_iteration(uint32_t K, scadles_stream* st, const uint64_t* iter_us, uint64_t b_min,
                                        uint64_t b_max, int policy, double base_batch, uint64_t* batch,
                                        float* weights, double* gamma);

/* T iterations of constant duration iter_us[j] from fresh buffers.
 *   queued (host[(T+1) x K]) or NULL: row t = buffer before iteration t, row T
 *   after the last; batch (host[T x K]) or NULL; dropped (host[K]) or NULL.   */
scadles_status scadles_stream_simulate(uint32_t K, const uint64_t* rate, const uint64_t* iter_us, uint64_t b_min,
                                       uint64_t b_max, int policy, uint64_t T, uint64_t* queued, uint64_t* batch,
                                       uint64_t* dropped);

/* Message for the last non-OK status returned on the calling thread.        */
const char* scadles_last_error(void);

/* Process-wide options, for testing and diagnosis:
 *   "validate"       1: scadles_weighted_aggregate checks its sets, and
 *                       scadles_topk_select(_noalloc), scadles_step_fused and
 *                       scadles_step_fused_ex read every device's selection
 *                       state back after the call and return
 *                       SCADLES_EINTERNAL if its internal checks failed;
 *                       scadles_topk_select_layers and
 *                       scadles_step_fused_layers do the same for their
 *                       layers of more than "row_max" elements (all of these
 *                       then synchronise `stream`).
 *   "inject_count_error" 1 (testing): the multi-launch selection (of the
 *                       whole vector, and of a per-layer selection's long
 *                       layers) reports a failed count check for device 0
 *                       (its outputs are unaffected), to exercise the
 *                       validation above.
 *   "force_exact"    1: Top-k skips the sampled single-read path and always
 *                       runs the exact multi-pass radix select.
 *   "force_fallback" 1: the sampled path runs but its result is discarded as
 *                       if the bracket had missed, exercising the fallback.
 *   "parts"          1..4 (default 1): device groups whose selections are
 *                       pipelined in scadles_step_fused (group i's main pass
 *                       overlaps the end of group i-1's selection, which runs
 *                       on a second stream the library creates per GPU, at the
 *                       default priority). Results do not depend on it.
 *   "row_max"        0..2^32-1 (default 2^21): in the per-layer selection,
 *                       layers of at most this many elements are selected as
 *                       (device, layer) rows; longer ones by the multi-launch
 *                       selection, consecutive ones pipelined on the library's
 *                       second stream and the rows on a third. Results do
 *                       not depend on it.
 *   "row_split"      0..2^32-1 (default 65536, the least that takes effect):
 *                       rows of more than this many elements (and at most
 *                       2^24) are read by one workgroup per 16384-element part
 *                       (their candidates staged, so each row is read once)
 *                       instead of one workgroup per row, unless their ratio
 *                       is so high that a part's candidates could exceed half
 *                       its elements. Results do not depend on it.
 *   "layer_order"    0..2 (default 1): the order in which the per-layer
 *                       selection runs its layers of more than "row_max"
 *                       elements: 0 index order, 1 ascending length (the
 *                       longest last, so the end of every earlier layer's
 *                       selection overlaps a long main pass), 2 descending
 *                       length. Every layer writes its own part of the
 *                       outputs and of the energy sums, so results do not
 *                       depend on it.
 * Returns SCADLES_EINVAL for an unknown name or a value out of range.       */
scadles_status scadles_set_option(const char* name, int64_t value);

/* Stage timing. While enabled, every scadles_topk_select / scadles_step_fused
 * call records HIP events on its stream at the boundaries of its stages.
 * scadles_profile_read synchronises those events, writes the summed
 * milliseconds of each stage to stage_ms (host[SCADLES_PROFILE_STAGES]) and
 * the number of calls recorded to *calls, and clears the record.
 * Stages: 0 bracket (sampling), 1 main select pass (one read of every
 * gradient; the sum over the device groups), 2 the rest of the selection
 * after the last main pass (exact threshold, ordered compaction, energies;
 * earlier groups' share overlaps the main passes), 3 weighted aggregation
 * (+SGD; empty for scadles_topk_select), 4 the whole call.                  */
#define SCADLES_PROFILE_STAGES 5
scadles_status scadles_profile_enable(int on);
scadles_status scadles_profile_read(double* stage_ms, uint32_t* calls);

#ifdef __cplusplus
}
#endif

#endif /* SCADLES_H */
