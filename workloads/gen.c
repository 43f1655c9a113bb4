/*
 * gen.c -- seeded synthetic gradients for the ScaDLES hot-path workloads.
 *
 * Shared by the tests, the benchmark and the oracle side; holds none of the
 * method's arithmetic (no ranking, selection, weighting or update), only
 * random numbers:
 *   - Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and
 *     Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11). Output
 *     depends only on (key, counter), so any thread split gives the same bytes.
 *   - Uniforms in (0, 1) with 53 random bits from two 32-bit words.
 *   - Normals by the Box-Muller transform (1958), in double.
 *   - Laplace by the inverse CDF, scale b = sd / sqrt(2).
 * Values are rounded to float with the C cast (round to nearest even).
 */
#include <math.h>
#include <stdint.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

typedef struct {
  uint32_t v[4];
} u32x4;

static inline u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1)
{
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * c.v[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * c.v[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    u32x4 o;
    o.v[0] = hi1 ^ c.v[1] ^ k0;
    o.v[1] = lo1;
    o.v[2] = hi0 ^ c.v[3] ^ k1;
    o.v[3] = lo0;
    c = o;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
  return c;
}

/* Exposed for the known-answer test of the generator. */
void gen_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
  u32x4 c = {{ctr[0], ctr[1], ctr[2], ctr[3]}};
  u32x4 r = philox4x32_10(c, key[0], key[1]);
  for (int i = 0; i < 4; ++i) out[i] = r.v[i];
}

/* (0, 1) from 53 bits: ((a << 21) | (b >> 11)) + 0.5, times 2^-53. */
static inline double u01(uint32_t a, uint32_t b)
{
  uint64_t x = ((uint64_t)a << 21) | (uint64_t)(b >> 11);
  return ((double)x + 0.5) * 0x1.0p-53;
}

static inline u32x4 draw(uint64_t seed, uint32_t tag, uint64_t m, uint32_t device, uint32_t iter)
{
  u32x4 c = {{(uint32_t)m, (uint32_t)(m >> 32), device, iter}};
  return philox4x32_10(c, (uint32_t)seed ^ (uint32_t)(seed >> 32), tag);
}

/* Uniform stream for host-side draws: out[t] for t in [offset, offset+count). */
void gen_uniforms(double* out, uint64_t count, uint64_t seed, uint32_t tag, uint32_t stream,
                  uint64_t offset)
{
  for (uint64_t t = 0; t < count; ++t) {
    uint64_t m = offset + t;
    u32x4 r = draw(seed, tag, m, stream, 0xFFFFFFFFu);
    out[t] = u01(r.v[0], r.v[1]);
  }
}

static inline uint32_t segment_of(uint64_t i, const uint64_t* seg_end, uint32_t nseg)
{
  uint32_t lo = 0, hi = nseg - 1;
  while (lo < hi) {
    uint32_t mid = (lo + hi) / 2;
    if (i < seg_end[mid]) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

/* Fill out[0..n) for (device, iter): element pair (2m, 2m+1) uses the draw
 * with counter (m, device, iter). dist 0: N(0, s_l^2); dist 1: Laplace with
 * standard deviation s_l; s_l is the scale of the segment holding the element
 * (segment l covers [seg_end[l-1], seg_end[l]), seg_end[nseg-1] == n).      */
void gen_fill(float* out, uint64_t n, uint64_t seed, uint32_t tag, uint32_t device, uint32_t iter,
              const uint64_t* seg_end, const double* seg_scale, uint32_t nseg, int dist,
              int nthreads)
{
  const uint64_t pairs = (n + 1) / 2;
  const double two_pi = 6.283185307179586476925286766559;
  const double inv_sqrt2 = 0.70710678118654752440084436210485;
  if (nthreads <= 0) nthreads = 1;
#pragma omp parallel for schedule(static, 65536) num_threads(nthreads)
  for (int64_t mi = 0; mi < (int64_t)pairs; ++mi) {
    uint64_t m = (uint64_t)mi;
    u32x4 r = draw(seed, tag, m, device, iter);
    double x0, x1;
    if (dist == 0) {
      double a = u01(r.v[0], r.v[1]);
      double b = u01(r.v[2], r.v[3]);
      double rad = sqrt(-2.0 * log(a));
      x0 = rad * cos(two_pi * b);
      x1 = rad * sin(two_pi * b);
    } else {
      double a = u01(r.v[0], r.v[1]) - 0.5;
      double b = u01(r.v[2], r.v[3]) - 0.5;
      x0 = -(a < 0 ? -1.0 : 1.0) * log(1.0 - 2.0 * fabs(a)) * inv_sqrt2;
      x1 = -(b < 0 ? -1.0 : 1.0) * log(1.0 - 2.0 * fabs(b)) * inv_sqrt2;
    }
    uint64_t i0 = 2 * m, i1 = 2 * m + 1;
    out[i0] = (float)(x0 * seg_scale[segment_of(i0, seg_end, nseg)]);
    if (i1 < n) out[i1] = (float)(x1 * seg_scale[segment_of(i1, seg_end, nseg)]);
  }
}

/* Per-element marks from one uniform u_i (counter (i, device, iter)):
 *   phase 0: u_i <  p_zero            -> g_i = +0 or -0 (sign from a spare bit)
 *   phase 1: p_zero <= u_i < p_zero + p_tie -> g_i = +mag or -mag
 * Running phase 0, then phase 1 with the same (seed, tag) marks disjoint sets. */
void gen_mark(float* g, uint64_t n, uint64_t seed, uint32_t tag, uint32_t device, uint32_t iter,
              int phase, double p_zero, double p_tie, float mag, int nthreads)
{
  if (nthreads <= 0) nthreads = 1;
#pragma omp parallel for schedule(static, 65536) num_threads(nthreads)
  for (int64_t ii = 0; ii < (int64_t)n; ++ii) {
    uint64_t i = (uint64_t)ii;
    u32x4 r = draw(seed, tag, i, device, iter);
    double u = u01(r.v[0], r.v[1]);
    int neg = (int)(r.v[2] & 1u);
    if (phase == 0) {
      if (u < p_zero) g[i] = neg ? -0.0f : 0.0f;
    } else {
      if (u >= p_zero && u < p_zero + p_tie) g[i] = neg ? -mag : mag;
    }
  }
}
