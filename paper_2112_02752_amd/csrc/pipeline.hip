// The pipelined training schedule, enqueued natively: the id dedups of each
// next group of batches on side streams while the main stream runs the
// forward and the fused update of the current group.  The dedup reads only a
// batch's ids and offsets, never the table, so running it early changes no
// result.  Everything here is host code that only enqueues work through the
// library's entry points and HIP events (no allocation, no synchronisation).
#include "emb_common.h"
#include "kernels.h"

extern "C" {

emb_status emb_pipeline_steps(const emb_tables* tables, int32_t pool, const emb_update* update, int32_t n_steps,
                              const emb_batch* batches, float* const* outs, const float* const* grads,
                              int32_t group, const emb_dedup_set* sets, void* main_stream, int32_t n_side,
                              void* const* side_streams, void* const* events) {
  if (tables == nullptr || update == nullptr || n_steps < 0 || group < 1 || n_side < 1 || n_side > group)
    return EMB_EINVAL;
  if (n_steps == 0) return EMB_OK;
  if (batches == nullptr || outs == nullptr || grads == nullptr || sets == nullptr || side_streams == nullptr ||
      events == nullptr)
    return EMB_EINVAL;
  for (int i = 0; i < 3 + 2 * n_side; ++i)
    if (events[i] == nullptr) return EMB_EINVAL;
  for (int s = 0; s < n_side; ++s)
    if (side_streams[s] == nullptr || side_streams[s] == main_stream) return EMB_EINVAL;
  const hipStream_t main = (hipStream_t)main_stream;
  hipEvent_t ev_start = (hipEvent_t)events[0];
  hipEvent_t ev_main[2] = {(hipEvent_t)events[1], (hipEvent_t)events[2]};
  auto ev_side = [&](int parity, int s) { return (hipEvent_t)events[3 + parity * n_side + s]; };
  auto hip_ok = [](hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_EHIP; };
  const int K = group;
  const int ngroups = (n_steps + K - 1) / K;
  // one dedup in flight per side stream at most with emb_unique_ids (which may
  // make the workgroups of a pass wait for one another); several side
  // streams use emb_unique_ids_concurrent, whose workgroups never wait
  auto dedup = n_side > 1 ? emb_unique_ids_concurrent : emb_unique_ids;
  emb_status st = hip_ok(hipEventRecord(ev_start, main));
  for (int s = 0; s < n_side && st == EMB_OK; ++s) st = hip_ok(hipStreamWaitEvent((hipStream_t)side_streams[s], ev_start, 0));
  if (st != EMB_OK) return st;

  // the dedups of group g into the buffer sets of parity g % 2
  auto dedups = [&](int g) -> emb_status {
    const int par = g % 2;
    for (int i = 0; i < K && g * K + i < n_steps; ++i) {
      const int k = g * K + i;
      const emb_dedup_set& d = sets[par * K + i];
      const emb_status r = dedup(tables, &batches[k], d.unique_keys, d.counts, d.seg_offsets, d.sort_perm,
                                 d.num_unique, d.ws, d.ws_bytes, side_streams[i % n_side]);
      if (r != EMB_OK) return r;
    }
    for (int s = 0; s < n_side; ++s) {
      const emb_status r = hip_ok(hipEventRecord(ev_side(par, s), (hipStream_t)side_streams[s]));
      if (r != EMB_OK) return r;
    }
    return EMB_OK;
  };

  if ((st = dedups(0)) != EMB_OK) return st;
  emb_update u = *update;
  for (int g = 0; g < ngroups; ++g) {
    if (g + 1 < ngroups) {
      if (g >= 1) {
        // the sets of group g + 1 were read by the main stream's group g - 1
        for (int s = 0; s < n_side; ++s)
          if ((st = hip_ok(hipStreamWaitEvent((hipStream_t)side_streams[s], ev_main[(g + 1) % 2], 0))) != EMB_OK)
            return st;
      }
      if ((st = dedups(g + 1)) != EMB_OK) return st;
    }
    for (int s = 0; s < n_side; ++s)
      if ((st = hip_ok(hipStreamWaitEvent(main, ev_side(g % 2, s), 0))) != EMB_OK) return st;
    for (int i = 0; i < K && g * K + i < n_steps; ++i) {
      const int k = g * K + i;
      const emb_dedup_set& d = sets[(g % 2) * K + i];
      u.seed = update->seed + (uint64_t)k;  // bf16 stochastic rounding draws fresh bits every step
      if ((st = emb_pool_fwd(tables, &batches[k], pool, outs[k], main_stream)) != EMB_OK) return st;
      if ((st = emb_grad_reduce(tables, &batches[k], pool, grads[k], d.sort_perm, d.seg_offsets, d.unique_keys,
                                d.num_unique, nullptr, &u, d.ws, d.ws_bytes, main_stream)) != EMB_OK)
        return st;
    }
    if ((st = hip_ok(hipEventRecord(ev_main[g % 2], main))) != EMB_OK) return st;
  }
  return EMB_OK;
}

}  // extern "C"
