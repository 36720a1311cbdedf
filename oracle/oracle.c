/*
 * ORACLE -- test infrastructure only.
 *
 * A plain, slow CPU statement of one training step of a
 * pooled sparse embedding layer: the layer the paper's introduction names as
 * the part of a recommendation model that turns massive high-dimensional
 * sparse ids into dense features at a high data-access cost (Introduction;
 * Section "Multi-mode Execution", heterogeneous pipeline paragraph).  The
 * paper gives no formula for the layer, so this file writes out the plain
 * definition of a bag-pooled embedding lookup and one optimizer step:
 *
 *   A[m][r] = scale_m * #{ j in bag m : row_offset[t(m)] + idx[j] = r }
 *   out     = A W                      (forward, rounded once to fp32)
 *   grad W  = A^T G                    (backward)
 *   W'      = opt(W, grad W) on the rows with a nonzero column of A.
 *
 * Dedup (sorted unique keys, stable sort permutation, counts, segment
 * offsets) is computed here only because the library's boundary returns it;
 * it is the plain definition: a stable ascending sort by key, then the runs
 * of equal keys.
 *
 * Accumulation is in double, with one rounding at each output.  The loops
 * over bags (forward) and over segments and rows (reduce, optimizer) may run
 * on several threads (OpenMP, oracle_set_threads); every output is computed
 * by one thread in the same order whatever the thread count, so the results
 * do not depend on it.  The sort is single-threaded.  Only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark load this
 * file; the product library never links or calls it.
 *
 * Tables are given as a "row store": either dense (keys == NULL: row r at
 * slot r) or a sorted list of the global rows present with their values, so
 * a check of a 50-million-row table needs only the rows a batch touches.
 *
 * Return values: 0 on success, negative on invalid input (the checks of the
 * step-1 validation below).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_OK = 0, ORC_BAD_OFFSETS = -1, ORC_BAD_ID = -2, ORC_MISSING_ROW = -3, ORC_BAD_ARG = -4, ORC_NOMEM = -5 };

/* Threads of the parallel loops (n < 1: the OpenMP default); the number in use. */
void oracle_set_threads(int32_t n) { omp_set_num_threads(n > 0 ? n : omp_get_num_procs()); }
int32_t oracle_get_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------------------ row store */

typedef struct {
  int64_t n;             /* rows held */
  const uint32_t* keys;  /* sorted global rows, or NULL for a dense table */
  int32_t dim;
  int32_t dtype;         /* 0 fp32, 1 bf16 (bits) */
} store_t;

static int64_t store_slot(const store_t* s, uint32_t key) {
  if (s->keys == NULL) return key < (uint64_t)s->n ? (int64_t)key : -1;
  int64_t lo = 0, hi = s->n; /* first slot with keys[slot] >= key */
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    if (s->keys[mid] < key) lo = mid + 1; else hi = mid;
  }
  return (lo < s->n && s->keys[lo] == key) ? lo : -1;
}

static double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

static uint16_t float_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* splitmix64 (Steele, Lea and Flood 2014): the output for generator state x */
static uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9e3779b97f4a7c15ULL;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

/* The 16 random bits of stochastic rounding for element counter c (row * D +
 * column) under seed: the top 16 bits of splitmix64(seed ^ splitmix64(c)). */
uint32_t oracle_sr_bits(uint64_t seed, uint64_t c) { return (uint32_t)(splitmix64(seed ^ splitmix64(c)) >> 48); }

/* Stochastic rounding of an fp32 value to bf16: the 16 bits below the bf16
 * mantissa are added to 16 random bits and cut off, so the magnitude rounds
 * up with probability (dropped bits) / 2^16 -- unbiased.  Non-finite values
 * round to nearest even. */
uint16_t oracle_bf16_stochastic(float f, uint32_t r16) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return float_to_bf16_rne(f);
  return (uint16_t)((u + (r16 & 0xffffu)) >> 16);
}

static double store_get(const store_t* s, const void* vals, int64_t slot, int32_t d) {
  if (s->dtype == 0) return (double)((const float*)vals)[slot * s->dim + d];
  return bf16_to_double(((const uint16_t*)vals)[slot * s->dim + d]);
}

/* one rounding to fp32 (round to nearest even), then to bf16 for bf16 tables */
static void store_put(const store_t* s, void* vals, int64_t slot, int32_t d, double v) {
  float f = (float)v;
  if (s->dtype == 0) ((float*)vals)[slot * s->dim + d] = f;
  else ((uint16_t*)vals)[slot * s->dim + d] = float_to_bf16_rne(f);
}

/* the same, stochastic rounding to bf16 with the bits of element (row, d) */
static void store_put_sr(const store_t* s, void* vals, int64_t slot, int32_t d, double v, uint64_t seed,
                         uint32_t row) {
  float f = (float)v;
  if (s->dtype == 0) ((float*)vals)[slot * s->dim + d] = f;
  else
    ((uint16_t*)vals)[slot * s->dim + d] =
        oracle_bf16_stochastic(f, oracle_sr_bits(seed, (uint64_t)row * (uint64_t)s->dim + (uint64_t)d));
}

/* ------------------------------------------------------------- validate */

/* offsets[0] = 0, nondecreasing; ids in [0, rows_t) of the bag's table */
static int validate(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx) {
  if (T < 1 || B < 0) return ORC_BAD_ARG;
  int64_t M = (int64_t)T * B;
  if (offsets[0] != 0) return ORC_BAD_OFFSETS;
  for (int64_t m = 0; m < M; ++m)
    if (offsets[m + 1] < offsets[m]) return ORC_BAD_OFFSETS;
  for (int64_t m = 0; m < M; ++m) {
    int64_t rows = row_offset[m / B + 1] - row_offset[m / B];
    for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j)
      if (idx[j] < 0 || idx[j] >= rows) return ORC_BAD_ID;
  }
  return ORC_OK;
}

/* ------------------------------------------------------------- forward */

/* out[m][d] = scale_m * sum over the bag of W[row_offset[t] + idx[j]][d];
 * scale 1 (pool 0, sum) or 1/L_m (pool 1, mean); an empty bag gives 0. */
int oracle_pool_fwd(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                    int32_t D, int32_t dtype, int64_t store_n, const uint32_t* store_keys, const void* store_vals,
                    int32_t pool, float* out) {
  int rc = validate(T, row_offset, B, offsets, idx);
  if (rc) return rc;
  store_t s = {store_n, store_keys, D, dtype};
  int64_t M = (int64_t)T * B;
  int err = ORC_OK;
#pragma omp parallel
  {
    double* acc = (double*)malloc(sizeof(double) * (size_t)D);
    if (!acc) {
#pragma omp atomic write
      err = ORC_NOMEM;
    }
#pragma omp for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
      if (!acc) continue;
      int64_t t = m / B;
      for (int32_t d = 0; d < D; ++d) acc[d] = 0.0;
      int missing = 0;
      for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j) {
        int64_t slot = store_slot(&s, (uint32_t)(row_offset[t] + idx[j]));
        if (slot < 0) {
          missing = 1;
          break;
        }
        for (int32_t d = 0; d < D; ++d) acc[d] += store_get(&s, store_vals, slot, d);
      }
      if (missing) {
#pragma omp atomic write
        err = ORC_MISSING_ROW;
        continue;
      }
      int32_t L = offsets[m + 1] - offsets[m];
      for (int32_t d = 0; d < D; ++d) {
        double v = acc[d];
        if (pool == 1 && L > 0) v = v / (double)L;
        out[m * D + d] = (float)v;
      }
    }
    free(acc);
  }
  return err;
}

/* --------------------------------------------------------------- dedup */

typedef struct {
  uint32_t key;
  int32_t pos;
} kp_t;

/* (key, position) order: ascending key, ties in position order -- the
 * unique result of a stable sort by key */
static int kp_cmp(const void* a, const void* b) {
  const kp_t* x = (const kp_t*)a;
  const kp_t* y = (const kp_t*)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  return (x->pos > y->pos) - (x->pos < y->pos);
}

/* key[j] = row_offset[t(j)] + idx[j]; perm = stable ascending sort of
 * positions by key; unique_keys/seg_offsets/counts describe the runs of
 * equal keys; seg_offsets[U] = N. */
int oracle_unique_ids(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                      uint32_t* unique_keys, int32_t* counts, int32_t* seg_offsets, int32_t* perm,
                      int32_t* num_unique) {
  int rc = validate(T, row_offset, B, offsets, idx);
  if (rc) return rc;
  int64_t M = (int64_t)T * B;
  int64_t N = offsets[M];
  kp_t* a = (kp_t*)malloc(sizeof(kp_t) * (size_t)(N > 0 ? N : 1));
  if (!a) return ORC_NOMEM;
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m)
    for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j) {
      a[j].key = (uint32_t)(row_offset[m / B] + idx[j]);
      a[j].pos = j;
    }
  qsort(a, (size_t)N, sizeof(kp_t), kp_cmp);
  int32_t U = 0;
  for (int64_t k = 0; k < N; ++k) {
    perm[k] = a[k].pos;
    if (k == 0 || a[k].key != a[k - 1].key) {
      unique_keys[U] = a[k].key;
      seg_offsets[U] = (int32_t)k;
      ++U;
    }
  }
  seg_offsets[U] = (int32_t)N;
  for (int32_t u = 0; u < U; ++u) counts[u] = seg_offsets[u + 1] - seg_offsets[u];
  *num_unique = U;
  free(a);
  return ORC_OK;
}

/* ---------------------------------------------------------- backward */

/* grad_rows[u][d] = sum over the sorted positions k of segment u of
 * scale_{m(k)} * G[m(k)][d], with m(k) the bag holding position perm[k]
 * (the rows of A^T G that are nonzero).  acc (optional, [U][D]) receives the
 * unrounded double sums. */
int oracle_grad_reduce(int32_t T, int32_t B, const int32_t* offsets, int32_t D, int32_t pool, const float* G,
                       const int32_t* perm, const int32_t* seg_offsets, int32_t U, float* grad_rows, double* acc) {
  if (T < 1 || B < 0 || D < 1 || U < 0) return ORC_BAD_ARG;
  int64_t M = (int64_t)T * B;
  int64_t N = offsets[M];
  int32_t* bag = (int32_t*)malloc(sizeof(int32_t) * (size_t)(N > 0 ? N : 1));
  if (!bag) return ORC_NOMEM;
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < M; ++m)
    for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j) bag[j] = (int32_t)m;
  int err = ORC_OK;
#pragma omp parallel
  {
    double* sum = (double*)malloc(sizeof(double) * (size_t)D);
    if (!sum) {
#pragma omp atomic write
      err = ORC_NOMEM;
    }
#pragma omp for schedule(dynamic, 64)
    for (int32_t u = 0; u < U; ++u) {
      if (!sum) continue;
      for (int32_t d = 0; d < D; ++d) sum[d] = 0.0;
      for (int32_t k = seg_offsets[u]; k < seg_offsets[u + 1]; ++k) {
        int32_t m = bag[perm[k]];
        int32_t L = offsets[m + 1] - offsets[m];
        double scale = pool == 1 ? 1.0 / (double)L : 1.0;
        for (int32_t d = 0; d < D; ++d) sum[d] += scale * (double)G[(int64_t)m * D + d];
      }
      for (int32_t d = 0; d < D; ++d) {
        if (grad_rows) grad_rows[(int64_t)u * D + d] = (float)sum[d];
        if (acc) acc[(int64_t)u * D + d] = sum[d];
      }
    }
    free(sum);
  }
  free(bag);
  return err;
}

/* ------------------------------------------------------------ optimizer */

/* One step on the rows unique_keys[0..U) with gradient rows grad[u][.]
 * (rounding 1: bf16 rows round stochastically, element (r, d) with the bits
 * oracle_sr_bits(seed, r * D + d)):
 *   opt 0, SGD:                     W[r] <- W[r] - lr * g
 *   opt 1, row-wise Adagrad:        h_r <- h_r + (1/D) sum_d g[d]^2
 *                                   W[r] <- W[r] - lr * g / (sqrt(h_r) + eps)
 *   opt 2, element-wise Adagrad:    h_r[d] <- h_r[d] + g[d]^2
 *   (Duchi, Hazan and Singer 2011)  W[r][d] <- W[r][d] - lr * g[d] / (sqrt(h_r[d]) + eps)
 * state is indexed like the store's slots (opt 1: one value per slot, opt 2:
 * D values per slot).  W is rounded once to fp32 (then to bf16 for bf16
 * tables); h is stored as fp32, the unrounded h is used for the same step's
 * W. */
int oracle_sparse_update(int32_t opt, float lr, float eps, int32_t D, int32_t dtype, int64_t store_n,
                         const uint32_t* store_keys, void* store_vals, float* state, const uint32_t* unique_keys,
                         int32_t U, const double* grad, int32_t rounding, uint64_t seed) {
  if (opt < 0 || opt > 2 || D < 1 || U < 0 || rounding < 0 || rounding > 1) return ORC_BAD_ARG;
  if (opt != 0 && state == NULL) return ORC_BAD_ARG;
  store_t s = {store_n, store_keys, D, dtype};
  for (int32_t u = 0; u < U; ++u)
    if (store_slot(&s, unique_keys[u]) < 0) return ORC_MISSING_ROW;
  /* distinct keys (strictly ascending, as a dedup gives them) touch distinct
   * rows, so their rows may be updated on several threads; otherwise in order */
  int distinct = 1;
  for (int32_t u = 1; u < U && distinct; ++u) distinct = unique_keys[u] > unique_keys[u - 1];
#pragma omp parallel for schedule(static) if (distinct)
  for (int32_t u = 0; u < U; ++u) {
    int64_t slot = store_slot(&s, unique_keys[u]);
    const double* g = grad + (int64_t)u * D;
    double denom = 1.0;
    if (opt == 1) {
      double sq = 0.0;
      for (int32_t d = 0; d < D; ++d) sq += g[d] * g[d];
      double h = (double)state[slot] + sq / (double)D;
      state[slot] = (float)h;
      denom = sqrt(h) + (double)eps;
    }
    for (int32_t d = 0; d < D; ++d) {
      if (opt == 2) {
        float* hp = state + slot * (int64_t)D + d;
        double h = (double)*hp + g[d] * g[d];
        *hp = (float)h;
        denom = (double)eps + sqrt(h);
      }
      double w = store_get(&s, store_vals, slot, d);
      if (rounding == 1) store_put_sr(&s, store_vals, slot, d, w - (double)lr * g[d] / denom, seed, unique_keys[u]);
      else store_put(&s, store_vals, slot, d, w - (double)lr * g[d] / denom);
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------- routing */

/* Routing of a batch's ids to the owners of a row-range sharding (the step
 * before the forward when the layer is spread over several devices): rank r
 * owns global rows [shard_start[r], shard_start[r+1]).  For each position j,
 * in position order, owner(j) is the rank whose range holds key[j]; the send
 * order lists the positions rank by rank, in position order within a rank.
 * send_counts[r] = positions owned by r; for the k-th sent position j:
 * send_ids[k] = key[j] - shard_start[owner(j)], send_pos[k] = j,
 * send_bag[k] = the bag holding j. */
int oracle_route_ids(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                     int32_t W, const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids,
                     int32_t* send_pos, int32_t* send_bag) {
  int rc = validate(T, row_offset, B, offsets, idx);
  if (rc) return rc;
  if (W < 1 || shard_start[0] != 0 || shard_start[W] != row_offset[T]) return ORC_BAD_ARG;
  for (int32_t r = 0; r < W; ++r)
    if (shard_start[r + 1] < shard_start[r]) return ORC_BAD_ARG;
  int64_t M = (int64_t)T * B;
  int64_t N = offsets[M];
  int64_t k = 0;
  for (int32_t r = 0; r < W; ++r) {
    send_counts[r] = 0;
    for (int64_t m = 0; m < M; ++m)
      for (int32_t j = offsets[m]; j < offsets[m + 1]; ++j) {
        int64_t key = row_offset[m / B] + idx[j];
        if (key < shard_start[r] || key >= shard_start[r + 1]) continue;
        if (k >= N) return ORC_BAD_ARG; /* every position has one owner: N entries in all */
        send_ids[k] = (int32_t)(key - shard_start[r]);
        send_pos[k] = j;
        send_bag[k] = (int32_t)m;
        ++k;
        ++send_counts[r];
      }
  }
  return ORC_OK;
}
