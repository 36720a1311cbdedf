/*
 * Seeded synthetic inputs for the sparse embedding layer (host side).
 *
 * This module holds no arithmetic of the embedding layer itself: it only
 * draws tables, bag lengths, ids and upstream gradients.  Both the HIP
 * library's tests/benchmark and the CPU oracle take their inputs from here.
 *
 * Every draw is counter based: value = splitmix64 chain over (seed, stream
 * tag, counter), so any element can be regenerated on its own, in any order,
 * on the host or (for table initial values) on the device, with identical
 * bits.  splitmix64 is the finaliser published by Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014.
 *
 * Distributions:
 *  - table initial values: U(-0.01, 0.01) on a 2^-23 * 0.01 grid, from the
 *    top 24 bits of the hash (exactly reproducible in fp32);
 *  - bounded Zipf(s) on ranks 1..n by rejection-inversion (Hormann and
 *    Derflinger, "Rejection-inversion to generate variates from monotone
 *    discrete distributions", ACM TOMACS 6(3), 1996), then a seeded affine
 *    bijection rank -> row so hot ids are scattered over the table;
 *  - Poisson(lambda) by inversion of its CDF;
 *  - N(0,1) by the Box-Muller transform.
 */
#include <stdint.h>
#include <math.h>
#include <string.h>

#define GOLDEN 0x9e3779b97f4a7c15ULL

static inline uint64_t sm64(uint64_t x) {
  uint64_t z = x + GOLDEN;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

/* Stream key for (seed, tag, a, b): tag names the quantity, a/b are small
 * coordinates such as the step and the table. */
uint64_t synth_stream(uint64_t seed, uint64_t tag, uint64_t a, uint64_t b) {
  return sm64(sm64(sm64(seed ^ (tag << 48)) ^ a) ^ (b * GOLDEN));
}

uint64_t synth_hash(uint64_t stream, uint64_t counter) { return sm64(stream ^ sm64(counter)); }

/* uniform double in [0, 1) with 53 random bits */
static inline double u01(uint64_t h) { return (double)(h >> 11) * (1.0 / 9007199254740992.0); }

/* ---------------------------------------------------------------- weights */

/* The weight grid: w = (int)(top24 - 2^23) * WSCALE, WSCALE = fl32(0.01 / 2^23).
 * One exact int->float conversion and one fp32 multiply: bit-identical on
 * any IEEE implementation. */
#define WSTEP ((float)(0.01 / 8388608.0))

static inline float weight_value(uint64_t stream, uint64_t r, uint64_t D, uint64_t d) {
  uint64_t h = synth_hash(stream, r * D + d);
  int32_t q = (int32_t)(h >> 40) - 8388608;
  return (float)q * WSTEP;
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

/* rows [r0, r0 + n) of the global (all tables stacked) weight matrix */
void synth_weights_f32(uint64_t seed, uint64_t r0, uint64_t n, int32_t D, float* out) {
  uint64_t st = synth_stream(seed, 4, 0, 0);
  for (uint64_t i = 0; i < n; ++i)
    for (int32_t d = 0; d < D; ++d) out[i * D + d] = weight_value(st, r0 + i, (uint64_t)D, (uint64_t)d);
}

void synth_weights_bf16(uint64_t seed, uint64_t r0, uint64_t n, int32_t D, uint16_t* out) {
  uint64_t st = synth_stream(seed, 4, 0, 0);
  for (uint64_t i = 0; i < n; ++i)
    for (int32_t d = 0; d < D; ++d)
      out[i * D + d] = f32_to_bf16_rne(weight_value(st, r0 + i, (uint64_t)D, (uint64_t)d));
}

/* the initial values of an arbitrary list of global rows */
void synth_weight_rows_f32(uint64_t seed, const uint32_t* rows, int64_t n, int32_t D, float* out) {
  uint64_t st = synth_stream(seed, 4, 0, 0);
  for (int64_t i = 0; i < n; ++i)
    for (int32_t d = 0; d < D; ++d) out[i * D + d] = weight_value(st, rows[i], (uint64_t)D, (uint64_t)d);
}

void synth_weight_rows_bf16(uint64_t seed, const uint32_t* rows, int64_t n, int32_t D, uint16_t* out) {
  uint64_t st = synth_stream(seed, 4, 0, 0);
  for (int64_t i = 0; i < n; ++i)
    for (int32_t d = 0; d < D; ++d)
      out[i * D + d] = f32_to_bf16_rne(weight_value(st, rows[i], (uint64_t)D, (uint64_t)d));
}

/* ------------------------------------------------------------ table sizes */

/* rows_t = round(exp(U(ln lo, ln hi))) for t < T */
void synth_loguniform_rows(uint64_t seed, int32_t T, double lo, double hi, int64_t* rows) {
  uint64_t st = synth_stream(seed, 5, 0, 0);
  for (int32_t t = 0; t < T; ++t) {
    double u = u01(synth_hash(st, (uint64_t)t));
    rows[t] = (int64_t)llround(exp(log(lo) + u * (log(hi) - log(lo))));
  }
}

/* ----------------------------------------------------------- bounded Zipf */

typedef struct {
  double s, n;
  double hx1, hn, sq; /* H(1.5)-h(1), H(n+0.5), squeeze constant */
} zipf_t;

/* log1p(x)/x and expm1(x)/x, continuous at 0 */
static double ln1p_over(double x) { return fabs(x) > 1e-8 ? log1p(x) / x : 1.0 - x * (0.5 - x / 3.0); }
static double em1_over(double x) { return fabs(x) > 1e-8 ? expm1(x) / x : 1.0 + x * (0.5 + x / 6.0); }

/* h(x) = x^-s; H(x) = integral of h = (x^(1-s) - 1)/(1-s) (log x at s = 1) */
static double zh(const zipf_t* z, double x) { return exp(-z->s * log(x)); }
static double zH(const zipf_t* z, double x) {
  double lx = log(x);
  return em1_over((1.0 - z->s) * lx) * lx;
}
static double zHinv(const zipf_t* z, double y) {
  double t = y * (1.0 - z->s);
  if (t < -1.0) t = -1.0; /* guards rounding at the left end of the support */
  return exp(ln1p_over(t) * y);
}

static void zipf_init(zipf_t* z, double s, int64_t n) {
  z->s = s;
  z->n = (double)n;
  z->hx1 = zH(z, 1.5) - 1.0;
  z->hn = zH(z, (double)n + 0.5);
  z->sq = 2.0 - zHinv(z, zH(z, 2.5) - zh(z, 2.0));
}

/* one rank in 1..n; uniforms come from (stream, counter, attempt) */
static int64_t zipf_draw(const zipf_t* z, uint64_t stream, uint64_t counter) {
  for (uint64_t a = 0;; ++a) {
    double u = z->hn + u01(synth_hash(stream ^ sm64(a + 1), counter)) * (z->hx1 - z->hn);
    double x = zHinv(z, u);
    int64_t k = (int64_t)(x + 0.5);
    if (k < 1) k = 1;
    if ((double)k > z->n) k = (int64_t)z->n;
    if ((double)k - x <= z->sq || u >= zH(z, (double)k + 0.5) - zh(z, (double)k)) return k;
  }
}

static uint64_t gcd64(uint64_t a, uint64_t b) {
  while (b) {
    uint64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

/* affine bijection on [0, n): row = (a*(k-1) + c) mod n, gcd(a, n) = 1 */
void synth_scramble_params(uint64_t seed, int32_t table, int64_t n, uint64_t* a, uint64_t* c) {
  uint64_t st = synth_stream(seed, 6, (uint64_t)table, 0);
  if (n <= 1) {
    *a = 1;
    *c = 0;
    return;
  }
  uint64_t aa = synth_hash(st, 0) % (uint64_t)n;
  if (aa == 0) aa = 1;
  while (gcd64(aa, (uint64_t)n) != 1) {
    aa += 1;
    if (aa >= (uint64_t)n) aa = 1;
  }
  *a = aa;
  *c = synth_hash(st, 1) % (uint64_t)n;
}

/* ------------------------------------------------------------- bag lengths */

/* kind 0: uniform 1..lmax; kind 1: clamp(Poisson(lambda), 1, lmax); kind 2: one-hot.
 * Writes lengths of bags [0, nbags) of one table for one step. */
void synth_bag_lengths(uint64_t seed, int64_t step, int32_t table, int32_t kind, int32_t lmax, double lambda,
                       int64_t nbags, int32_t* len) {
  uint64_t st = synth_stream(seed, 1, (uint64_t)step, (uint64_t)table);
  if (kind == 2) {
    for (int64_t b = 0; b < nbags; ++b) len[b] = 1;
    return;
  }
  if (kind == 0) {
    for (int64_t b = 0; b < nbags; ++b) {
      uint64_t h = synth_hash(st, (uint64_t)b) >> 32;
      len[b] = 1 + (int32_t)((h * (uint64_t)lmax) >> 32);
    }
    return;
  }
  /* Poisson by CDF inversion: smallest x with u < F(x) */
  for (int64_t b = 0; b < nbags; ++b) {
    double u = u01(synth_hash(st, (uint64_t)b));
    double p = exp(-lambda), cdf = p;
    int32_t x = 0;
    while (u >= cdf && x < 100000) {
      ++x;
      p *= lambda / (double)x;
      cdf += p;
    }
    if (x < 1) x = 1;
    if (x > lmax) x = lmax;
    len[b] = x;
  }
}

/* ------------------------------------------------------------------- ids */

/* ids for positions [0, n) of one table in one step.  dist 0: uniform over
 * [0, rows); dist 1: bounded Zipf(s) over ranks then the table's scramble. */
void synth_ids(uint64_t seed, int64_t step, int32_t table, int32_t dist, double s, int64_t rows, int64_t n,
               int32_t* ids) {
  uint64_t st = synth_stream(seed, 2, (uint64_t)step, (uint64_t)table);
  if (dist == 0) {
    for (int64_t j = 0; j < n; ++j) {
      uint64_t h = synth_hash(st, (uint64_t)j) >> 32;
      ids[j] = (int32_t)((h * (uint64_t)rows) >> 32);
    }
    return;
  }
  zipf_t z;
  zipf_init(&z, s, rows);
  uint64_t a, c;
  synth_scramble_params(seed, table, rows, &a, &c);
  for (int64_t j = 0; j < n; ++j) {
    uint64_t k = (uint64_t)zipf_draw(&z, st, (uint64_t)j) - 1;
    unsigned __int128 v = (unsigned __int128)a * k + c;
    ids[j] = (int32_t)(uint64_t)(v % (uint64_t)rows);
  }
}

/* rank -> row of the scramble (used by tests to locate hot rows) */
int64_t synth_rank_to_row(uint64_t seed, int32_t table, int64_t rows, int64_t rank1) {
  uint64_t a, c;
  synth_scramble_params(seed, table, rows, &a, &c);
  unsigned __int128 v = (unsigned __int128)a * (uint64_t)(rank1 - 1) + c;
  return (int64_t)(uint64_t)(v % (uint64_t)rows);
}

/* ------------------------------------------------------ upstream gradients */

/* N(0,1) fp32 for elements [e0, e0 + n) of the step's [M][D] gradient */
void synth_normal_f32(uint64_t seed, int64_t step, int64_t e0, int64_t n, float* out) {
  uint64_t st = synth_stream(seed, 3, (uint64_t)step, 0);
  const double two_pi = 6.283185307179586476925286766559;
  for (int64_t i = 0; i < n; ++i) {
    uint64_t h1 = synth_hash(st, 2 * (uint64_t)(e0 + i));
    uint64_t h2 = synth_hash(st, 2 * (uint64_t)(e0 + i) + 1);
    double u1 = 1.0 - u01(h1); /* (0, 1] */
    double u2 = u01(h2);
    out[i] = (float)(sqrt(-2.0 * log(u1)) * cos(two_pi * u2));
  }
}
