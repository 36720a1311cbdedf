/*
 * Driver of the CPU sanitizer run (AddressSanitizer + UndefinedBehaviorSanitizer):
 * draws small multi-table batches with the input generator (synth.c) and
 * runs every oracle routine (oracle.c) on them -- forward, dedup, gradient
 * reduce, the three optimizers on fp32 and bf16 stores with both roundings,
 * routing, and the rejection of malformed batches -- checking a few
 * invariants on the way.  Any out-of-bounds access, leak or undefined
 * operation aborts the run through the sanitizers.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* synth.c */
void synth_weights_f32(uint64_t seed, uint64_t r0, uint64_t n, int32_t D, float* out);
void synth_weights_bf16(uint64_t seed, uint64_t r0, uint64_t n, int32_t D, uint16_t* out);
void synth_loguniform_rows(uint64_t seed, int32_t T, double lo, double hi, int64_t* rows);
void synth_bag_lengths(uint64_t seed, int64_t step, int32_t table, int32_t kind, int32_t lmax, double lambda,
                       int64_t B, int32_t* out);
void synth_ids(uint64_t seed, int64_t step, int32_t table, int32_t dist, double s, int64_t rows, int64_t n,
               int32_t* out);
void synth_normal_f32(uint64_t seed, int64_t step, int64_t e0, int64_t n, float* out);
/* oracle.c */
void oracle_set_threads(int32_t n);
int oracle_pool_fwd(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                    int32_t D, int32_t dtype, int64_t store_n, const uint32_t* store_keys, const void* store_vals,
                    int32_t pool, float* out);
int oracle_unique_ids(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                      uint32_t* unique_keys, int32_t* counts, int32_t* seg_offsets, int32_t* perm,
                      int32_t* num_unique);
int oracle_grad_reduce(int32_t T, int32_t B, const int32_t* offsets, int32_t D, int32_t pool, const float* G,
                       const int32_t* perm, const int32_t* seg_offsets, int32_t U, float* grad_rows, double* acc);
int oracle_sparse_update(int32_t opt, float lr, float eps, int32_t D, int32_t dtype, int64_t store_n,
                         const uint32_t* store_keys, void* store_vals, float* state, const uint32_t* unique_keys,
                         int32_t U, const double* grad, int32_t rounding, uint64_t seed);
int oracle_route_ids(int32_t T, const int64_t* row_offset, int32_t B, const int32_t* offsets, const int32_t* idx,
                     int32_t W, const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids,
                     int32_t* send_pos, int32_t* send_bag);

static int fails = 0;
#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #c);        \
      ++fails;                                                    \
    }                                                             \
  } while (0)

static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) abort();
  return p;
}

/* one step over a random multi-table batch; dtype 0 fp32, 1 bf16 */
static void run_case(uint64_t seed, int32_t T, int32_t B, int32_t D, int32_t dtype, int32_t pool, int32_t opt,
                     int32_t rounding) {
  int64_t* rows = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)T);
  synth_loguniform_rows(seed, T, 50.0, 3000.0, rows);
  int64_t* ro = (int64_t*)xmalloc(sizeof(int64_t) * (size_t)(T + 1));
  ro[0] = 0;
  for (int t = 0; t < T; ++t) ro[t + 1] = ro[t] + rows[t];
  const int64_t R = ro[T];
  const int32_t M = T * B;
  int32_t* off = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)(M + 1));
  off[0] = 0;
  for (int t = 0; t < T; ++t) {
    int32_t* len = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)B);
    synth_bag_lengths(seed, 0, t, t % 3 == 2 ? 2 : (t % 3), 40, 12.0, B, len);
    for (int b = 0; b < B; ++b) off[t * B + b + 1] = off[t * B + b] + (b % 7 == 3 ? 0 : len[b]);  /* some empty bags */
    free(len);
  }
  const int32_t N = off[M];
  int32_t* idx = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  for (int t = 0; t < T; ++t) {
    const int32_t lo = off[t * B], hi = off[(t + 1) * B];
    synth_ids(seed, 0, t, t % 2, 1.1, rows[t], hi - lo, idx + lo);
  }
  void* W = xmalloc((size_t)R * (size_t)D * (dtype ? 2 : 4));
  if (dtype) synth_weights_bf16(seed, 0, (uint64_t)R, D, (uint16_t*)W);
  else synth_weights_f32(seed, 0, (uint64_t)R, D, (float*)W);
  float* G = (float*)xmalloc(sizeof(float) * (size_t)M * (size_t)D);
  synth_normal_f32(seed, 0, 0, (int64_t)M * D, G);
  float* out = (float*)xmalloc(sizeof(float) * (size_t)M * (size_t)D);
  CHECK(oracle_pool_fwd(T, ro, B, off, idx, D, dtype, R, NULL, W, pool, out) == 0);

  uint32_t* uk = (uint32_t*)xmalloc(sizeof(uint32_t) * (size_t)N);
  int32_t* cnt = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  int32_t* seg = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)(N + 1));
  int32_t* perm = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  int32_t U = -1;
  CHECK(oracle_unique_ids(T, ro, B, off, idx, uk, cnt, seg, perm, &U) == 0);
  CHECK(U >= (N > 0) && U <= N);
  int64_t total = 0;
  for (int32_t u = 0; u < U; ++u) {
    total += cnt[u];
    if (u) CHECK(uk[u] > uk[u - 1]);
  }
  CHECK(total == N && seg[U] == N);

  float* gr = (float*)xmalloc(sizeof(float) * (size_t)(U ? U : 1) * (size_t)D);
  double* acc = (double*)xmalloc(sizeof(double) * (size_t)(U ? U : 1) * (size_t)D);
  CHECK(oracle_grad_reduce(T, B, off, D, pool, G, perm, seg, U, gr, acc) == 0);
  float* state = (float*)calloc((size_t)R * (size_t)(opt == 2 ? D : 1), sizeof(float));
  if (!state) abort();
  CHECK(oracle_sparse_update(opt, 0.01f, 1e-8f, D, dtype, R, NULL, W, opt ? state : NULL, uk, U, acc, rounding,
                             seed) == 0);
  /* a sparse store of just the touched rows (sorted keys) */
  void* Ws = xmalloc((size_t)(U ? U : 1) * (size_t)D * (dtype ? 2 : 4));
  memset(Ws, 0, (size_t)(U ? U : 1) * (size_t)D * (dtype ? 2 : 4));
  CHECK(oracle_pool_fwd(T, ro, B, off, idx, D, dtype, U, uk, Ws, pool, out) == 0);
  /* routing over 5 uneven ranks */
  int64_t shard[6] = {0, R / 7, R / 3, R / 3, (2 * R) / 3, R};
  int32_t scnt[5];
  int32_t* sids = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  int32_t* spos = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  int32_t* sbag = (int32_t*)xmalloc(sizeof(int32_t) * (size_t)N);
  CHECK(oracle_route_ids(T, ro, B, off, idx, 5, shard, scnt, sids, spos, sbag) == 0);
  CHECK(scnt[0] + scnt[1] + scnt[2] + scnt[3] + scnt[4] == N);
  /* malformed batches are rejected */
  if (N > 0) {
    const int32_t keep = idx[0];
    idx[0] = (int32_t)rows[0];
    CHECK(oracle_unique_ids(T, ro, B, off, idx, uk, cnt, seg, perm, &U) != 0);
    idx[0] = keep;
    if (M > 1) {
      const int32_t k1 = off[1];
      off[1] = off[2] + 1;
      CHECK(oracle_pool_fwd(T, ro, B, off, idx, D, dtype, R, NULL, W, pool, out) != 0);
      off[1] = k1;
    }
  }
  free(rows); free(ro); free(off); free(idx); free(W); free(G); free(out); free(uk); free(cnt); free(seg);
  free(perm); free(gr); free(acc); free(state); free(Ws); free(sids); free(spos); free(sbag);
}

int main(void) {
  for (int threads = 1; threads <= 4; threads += 3) {
    oracle_set_threads(threads);
    run_case(1, 1, 64, 16, 0, 0, 0, 0);
    run_case(2, 3, 40, 8, 0, 1, 1, 0);
    run_case(3, 4, 33, 8, 1, 0, 1, 1);
    run_case(4, 2, 50, 4, 0, 0, 2, 0);
    run_case(5, 5, 17, 8, 1, 1, 2, 1);
    run_case(6, 1, 1, 4, 0, 0, 0, 0);
  }
  printf(fails ? "FAILED %d\n" : "ok\n", fails);
  return fails ? 1 : 0;
}
