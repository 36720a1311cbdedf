// C ABI of the embedding layer: host-side argument checks, workspace
// layout, kernel dispatch.  No allocation, no synchronisation.
#include <string.h>

#include "emb_common.h"
#include "kernels.h"

using namespace emb;

namespace {

constexpr int64_t kMaxIndices = (int64_t)1 << 30;

int dtype_bytes(int32_t dtype) { return dtype == EMB_FP32 ? 4 : (dtype == EMB_BF16 ? 2 : 0); }

emb_status check_tables(const emb_tables* t, TableOffsets* ro, int64_t* total_rows) {
  if (t == nullptr || t->row_offset == nullptr || t->weights == nullptr) return EMB_EINVAL;
  if (t->num_tables < 1 || t->num_tables > EMB_MAX_TABLES) return t->num_tables < 1 ? EMB_EINVAL : EMB_EUNSUPPORTED;
  if (t->dim < 1) return EMB_EINVAL;
  const int sb = dtype_bytes(t->dtype);
  if (sb == 0) return EMB_EINVAL;
  if (((int64_t)t->dim * sb) % 16 != 0) return EMB_EUNSUPPORTED;
  if (((uintptr_t)t->weights & 15u) != 0) return EMB_EINVAL;
  if (t->row_offset[0] != 0) return EMB_EINVAL;
  memset(ro, 0, sizeof(*ro));
  for (int i = 0; i < t->num_tables; ++i)
    if (t->row_offset[i + 1] < t->row_offset[i]) return EMB_EINVAL;
  const int64_t R = t->row_offset[t->num_tables];
  if (R >= ((int64_t)1 << 32)) return EMB_EUNSUPPORTED;
  for (int i = 0; i <= t->num_tables; ++i) ro->off[i] = (uint32_t)t->row_offset[i];
  *total_rows = R;
  return EMB_OK;
}

emb_status check_batch(const emb_batch* b, int32_t T, int32_t* M) {
  if (b == nullptr || b->offsets == nullptr) return EMB_EINVAL;
  if (b->bags_per_table < 0 || b->num_indices < 0) return EMB_EINVAL;
  if (b->num_indices >= kMaxIndices) return EMB_EUNSUPPORTED;
  if (b->num_indices > 0 && b->indices == nullptr) return EMB_EINVAL;
  if (b->index_bytes != 0 && b->index_bytes != 4 && b->index_bytes != 8) return EMB_EINVAL;
  const int64_t m = (int64_t)T * b->bags_per_table;
  if (m >= ((int64_t)1 << 31) - 1) return EMB_EUNSUPPORTED;
  *M = (int32_t)m;
  return EMB_OK;
}

int key_bits_for(int64_t R) {
  int bits = 1;
  while (bits < 32 && ((int64_t)1 << bits) < R) ++bits;
  return bits;
}

// The largest batch (ids) whose layout fits ws_bytes with rows of D floats.
// Layouts grow with the batch, so a bisection finds it; the last answer of
// each thread is kept, since a workspace is normally used with one size.
int64_t ws_capacity(size_t ws_bytes, int32_t D) {
  thread_local size_t c_bytes = 0;
  thread_local int32_t c_dim = 0;
  thread_local int64_t c_cap = -1;
  if (c_cap >= 0 && c_bytes == ws_bytes && c_dim == D) return c_cap;
  int64_t lo = 0, hi = kMaxIndices - 1;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (ws_layout(mid, 0, D).total <= ws_bytes) lo = mid; else hi = mid - 1;
  }
  c_bytes = ws_bytes;
  c_dim = D;
  c_cap = lo;
  return lo;
}

// Regions are placed by the workspace's capacity, not by the batch: for one
// ws_bytes and dim every byte belongs to the same region in every call, so a
// region of call-tagged words only ever holds such words (or the zeros of
// emb_workspace_init), never another call's keys, positions or counts, which
// could pass for a word of the current call.
emb_status check_ws(const void* ws, size_t ws_bytes, int64_t N, int64_t M, int32_t D, WsLayout* lay) {
  if (ws == nullptr) return EMB_EINVAL;
  if (((uintptr_t)ws & 255u) != 0) return EMB_EWORKSPACE;
  if (ws_bytes < ws_layout(N, M, D).total) return EMB_EWORKSPACE;
  *lay = ws_layout(ws_capacity(ws_bytes, D), M, D);
  return EMB_OK;
}

emb_status check_update(const emb_update* u) {
  if (u == nullptr) return EMB_EINVAL;
  if (u->opt != EMB_OPT_SGD && u->opt != EMB_OPT_ADAGRAD_ROWWISE && u->opt != EMB_OPT_ADAGRAD_ELEMENTWISE)
    return EMB_EINVAL;
  if (u->opt != EMB_OPT_SGD && u->state == nullptr) return EMB_EINVAL;
  if (u->rounding != EMB_ROUND_NEAREST_EVEN && u->rounding != EMB_ROUND_STOCHASTIC) return EMB_EINVAL;
  return EMB_OK;
}

emb_status hip_status(hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_EHIP; }

// host checks of a routing call; fills the launch descriptor (ws left null)
emb_status route_prepare(const emb_tables* tables, const emb_batch* batch, int32_t world_size,
                         const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids, int32_t* send_pos,
                         int32_t* send_bag, RouteLaunch* p) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  st = check_batch(batch, tables->num_tables, &M);
  if (st != EMB_OK) return st;
  if (world_size < 1 || world_size > kMaxRanks || shard_start == nullptr || send_counts == nullptr) return EMB_EINVAL;
  if (shard_start[0] != 0 || shard_start[world_size] != R) return EMB_EINVAL;
  ShardBounds sb;
  for (int r = 0; r < world_size; ++r) {
    if (shard_start[r + 1] < shard_start[r]) return EMB_EINVAL;
    sb.off[r] = (uint32_t)shard_start[r];
  }
  sb.off[world_size] = (uint32_t)R;
  const int64_t N = batch->num_indices;
  if (N > 0 && (send_ids == nullptr || send_pos == nullptr || send_bag == nullptr)) return EMB_EINVAL;
  *p = RouteLaunch{};
  p->offsets = batch->offsets;
  p->idx = batch->indices;
  p->idx64 = batch->index_bytes == 8;
  p->ro = ro;
  p->sb = sb;
  p->B = batch->bags_per_table;
  p->M = M;
  p->W = world_size;
  p->N = N;
  p->send_counts = send_counts;
  p->send_ids = send_ids;
  p->send_pos = send_pos;
  p->send_bag = send_bag;
  return EMB_OK;
}


}  // namespace

namespace emb {

emb_status check_dedup_group(const emb_tables* tables, int32_t n_batches, const emb_batch* batches, const void* ws,
                             size_t ws_bytes) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  if (n_batches < 1 || batches == nullptr) return EMB_EINVAL;
  if (n_batches > kMaxGroup) return EMB_EUNSUPPORTED;
  int gb = 0;
  while ((1 << gb) < n_batches) ++gb;
  if (key_bits_for(R) + gb > 32) return EMB_EUNSUPPORTED;
  int64_t N = 0, M = 0;
  for (int i = 0; i < n_batches; ++i) {
    int32_t m = 0;
    if ((st = check_batch(&batches[i], tables->num_tables, &m)) != EMB_OK) return st;
    N += batches[i].num_indices;
    M += m;
  }
  if (N >= kMaxIndices) return EMB_EUNSUPPORTED;
  WsLayout lay;
  return check_ws(ws, ws_bytes, N, M, tables->dim, &lay);
}

// Every host check that emb_pool_fwd, emb_unique_ids (or _concurrent) and a
// fused emb_grad_reduce would make for one step of the pipelined schedule,
// so that the schedule can reject a bad step before it enqueues anything.
emb_status check_pipeline_step(const emb_tables* tables, const emb_batch* batch, int32_t pool, const float* out,
                               const float* grad, const emb_update* update, const emb_dedup_set* d) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  if ((st = check_batch(batch, tables->num_tables, &M)) != EMB_OK) return st;
  if (pool != EMB_POOL_SUM && pool != EMB_POOL_MEAN) return EMB_EINVAL;
  if ((st = check_update(update)) != EMB_OK) return st;
  if ((int64_t)tables->dim * dtype_bytes(tables->dtype) / 16 > fwd_max_row_vectors()) return EMB_EUNSUPPORTED;
  if (tables->dim > reduce_max_dim()) return EMB_EUNSUPPORTED;
  if (M > 0 && out == nullptr) return EMB_EINVAL;
  if (batch->num_indices > 0 && grad == nullptr) return EMB_EINVAL;
  return check_dedup_step(tables, batch, d);
}

emb_status check_dedup_step(const emb_tables* tables, const emb_batch* batch, const emb_dedup_set* d) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  if ((st = check_batch(batch, tables->num_tables, &M)) != EMB_OK) return st;
  if (d->seg_offsets == nullptr || d->num_unique == nullptr) return EMB_EINVAL;
  if (batch->num_indices > 0 && (d->unique_keys == nullptr || d->counts == nullptr || d->sort_perm == nullptr))
    return EMB_EINVAL;
  WsLayout lay;
  return check_ws(d->ws, d->ws_bytes, batch->num_indices, M, tables->dim, &lay);
}

}  // namespace emb

extern "C" {

const char* emb_status_string(int32_t status) {
  switch (status) {
    case EMB_OK: return "ok";
    case EMB_EINVAL: return "invalid argument";
    case EMB_EWORKSPACE: return "workspace too small or misaligned";
    case EMB_EUNSUPPORTED: return "unsupported size or layout";
    case EMB_EHIP: return "HIP launch failure";
    default: return "unknown status";
  }
}

size_t emb_workspace_size(int64_t num_indices, int64_t num_bags, int32_t dim) {
  if (num_indices < 0 || num_indices >= kMaxIndices || num_bags < 0 || dim < 1) return 0;
  return ws_layout(num_indices, num_bags, dim).total;
}

size_t emb_workspace_error_offset(void) { return offsetof(WsHeader, err); }

emb_status emb_workspace_status(const void* ws, size_t ws_bytes, int32_t* status, void* stream) {
  if (ws == nullptr || status == nullptr) return EMB_EINVAL;
  if (((uintptr_t)ws & 255u) != 0 || ws_bytes < sizeof(WsHeader)) return EMB_EWORKSPACE;
  return hip_status(launch_workspace_status(ws, status, (hipStream_t)stream));
}

emb_status emb_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (ws == nullptr) return EMB_EINVAL;
  if (((uintptr_t)ws & 255u) != 0) return EMB_EWORKSPACE;
  return hip_status(launch_zero_bytes(ws, ws_bytes, (hipStream_t)stream));
}

emb_status emb_pool_fwd(const emb_tables* tables, const emb_batch* batch, int32_t pool, float* out, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  st = check_batch(batch, tables->num_tables, &M);
  if (st != EMB_OK) return st;
  if (pool != EMB_POOL_SUM && pool != EMB_POOL_MEAN) return EMB_EINVAL;
  if (M > 0 && out == nullptr) return EMB_EINVAL;
  if ((int64_t)tables->dim * dtype_bytes(tables->dtype) / 16 > fwd_max_row_vectors()) return EMB_EUNSUPPORTED;
  if (M == 0) return EMB_OK;
  FwdLaunch p{};
  p.W = tables->weights;
  p.offsets = batch->offsets;
  p.idx = batch->indices;
  p.idx64 = batch->index_bytes == 8;
  p.ro = ro;
  p.B = batch->bags_per_table;
  p.M = M;
  p.D = tables->dim;
  p.dtype = tables->dtype;
  p.pool = pool;
  p.out = out;
  return hip_status(launch_pool_fwd(p, (hipStream_t)stream));
}

static emb_status unique_ids(const emb_tables* tables, const emb_batch* batch, uint32_t* unique_keys, int32_t* counts,
                             int32_t* seg_offsets, int32_t* sort_perm, int32_t* num_unique, void* ws, size_t ws_bytes,
                             int32_t waitfree, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  st = check_batch(batch, tables->num_tables, &M);
  if (st != EMB_OK) return st;
  if (seg_offsets == nullptr || num_unique == nullptr) return EMB_EINVAL;
  if (batch->num_indices > 0 && (unique_keys == nullptr || counts == nullptr || sort_perm == nullptr))
    return EMB_EINVAL;
  WsLayout lay;
  st = check_ws(ws, ws_bytes, batch->num_indices, M, tables->dim, &lay);
  if (st != EMB_OK) return st;
  DedupLaunch p{};
  p.offsets = batch->offsets;
  p.idx = batch->indices;
  p.idx64 = batch->index_bytes == 8;
  p.ro = ro;
  p.T = tables->num_tables;
  p.B = batch->bags_per_table;
  p.M = M;
  p.N = batch->num_indices;
  p.plan = make_sort_plan(key_bits_for(R));
  p.ws = ws;
  p.ws_bytes = ws_bytes;
  p.lay = lay;
  p.unique_keys = unique_keys;
  p.counts = counts;
  p.seg_offsets = seg_offsets;
  p.sort_perm = sort_perm;
  p.num_unique = num_unique;
  p.waitfree = waitfree;
  return hip_status(launch_dedup(p, (hipStream_t)stream));
}

emb_status emb_unique_ids_batched(const emb_tables* tables, int32_t n_batches, const emb_batch* batches,
                                  const emb_dedup_set* sets, void* ws, size_t ws_bytes, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  if (n_batches < 1 || batches == nullptr || sets == nullptr) return EMB_EINVAL;
  if (n_batches > kMaxGroup) return EMB_EUNSUPPORTED;
  const int kb = key_bits_for(R);
  int gb = 0;
  while ((1 << gb) < n_batches) ++gb;
  if (kb + gb > 32) return EMB_EUNSUPPORTED;  // the batch index must fit above the key bits
  GroupDedupLaunch p{};
  p.n = n_batches;
  p.ro = ro;
  p.T = tables->num_tables;
  p.key_bits = kb;
  int64_t Ntot = 0, Mtot = 0;
  for (int i = 0; i < n_batches; ++i) {
    const emb_batch* b = &batches[i];
    const emb_dedup_set& d = sets[i];
    int32_t M = 0;
    if ((st = check_batch(b, tables->num_tables, &M)) != EMB_OK) return st;
    if (d.seg_offsets == nullptr || d.num_unique == nullptr) return EMB_EINVAL;
    if (b->num_indices > 0 && (d.unique_keys == nullptr || d.counts == nullptr || d.sort_perm == nullptr))
      return EMB_EINVAL;
    WsLayout li;
    if ((st = check_ws(d.ws, d.ws_bytes, b->num_indices, M, tables->dim, &li)) != EMB_OK) return st;
    // each batch's workspace is its own: not the group's, not another batch's
    if (d.ws == ws) return EMB_EINVAL;
    for (int j = 0; j < i; ++j)
      if (sets[j].ws == d.ws) return EMB_EINVAL;
    GroupMember& m = p.m[i];
    m.offsets = b->offsets;
    m.idx = b->indices;
    m.idx64 = b->index_bytes == 8;
    m.B = b->bags_per_table;
    m.M = M;
    m.N = (int32_t)b->num_indices;
    m.P = Ntot;
    // about kPrepPositions positions per prepare block, as for one batch
    const int64_t want = m.N > 0 ? (int64_t)kPrepPositions * M / m.N : 1;
    m.bags_per_block = (int32_t)(want < 1 ? 1 : (want > kPrepMaxBags ? kPrepMaxBags : want));
    char* w = static_cast<char*>(d.ws);
    m.unique_keys = d.unique_keys;
    m.counts = d.counts;
    m.seg_offsets = d.seg_offsets;
    m.sort_perm = d.sort_perm;
    m.num_unique = d.num_unique;
    m.sorted_bag = reinterpret_cast<int32_t*>(w + li.sorted_bag);
    m.chunk_seg = reinterpret_cast<int32_t*>(w + li.chunk_seg);
    m.uniq_words = reinterpret_cast<uint64_t*>(w + li.uniq_status);
    m.totals = reinterpret_cast<uint32_t*>(w + li.totals);
    m.hdr = reinterpret_cast<WsHeader*>(w + li.hdr);
    Ntot += m.N;
    Mtot += M;
  }
  if (Ntot >= kMaxIndices) return EMB_EUNSUPPORTED;
  if ((st = check_ws(ws, ws_bytes, Ntot, Mtot, tables->dim, &p.lay)) != EMB_OK) return st;
  p.N = Ntot;
  p.plan = make_sort_plan(kb + gb);
  p.ws = ws;
  p.ws_bytes = ws_bytes;
  return hip_status(launch_dedup_group(p, (hipStream_t)stream));
}

emb_status emb_unique_ids(const emb_tables* tables, const emb_batch* batch, uint32_t* unique_keys, int32_t* counts,
                          int32_t* seg_offsets, int32_t* sort_perm, int32_t* num_unique, void* ws, size_t ws_bytes,
                          void* stream) {
  return unique_ids(tables, batch, unique_keys, counts, seg_offsets, sort_perm, num_unique, ws, ws_bytes, 0, stream);
}

emb_status emb_unique_ids_concurrent(const emb_tables* tables, const emb_batch* batch, uint32_t* unique_keys,
                                     int32_t* counts, int32_t* seg_offsets, int32_t* sort_perm, int32_t* num_unique,
                                     void* ws, size_t ws_bytes, void* stream) {
  return unique_ids(tables, batch, unique_keys, counts, seg_offsets, sort_perm, num_unique, ws, ws_bytes, 1, stream);
}

emb_status emb_grad_reduce(const emb_tables* tables, const emb_batch* batch, int32_t pool, const float* grad_out,
                           const int32_t* sort_perm, const int32_t* seg_offsets, const uint32_t* unique_keys,
                           const int32_t* num_unique, float* grad_rows, const emb_update* fuse, void* ws,
                           size_t ws_bytes, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  st = check_batch(batch, tables->num_tables, &M);
  if (st != EMB_OK) return st;
  if (pool != EMB_POOL_SUM && pool != EMB_POOL_MEAN) return EMB_EINVAL;
  if (fuse == nullptr && grad_rows == nullptr) return EMB_EINVAL;
  if (fuse != nullptr && (st = check_update(fuse)) != EMB_OK) return st;
  if (tables->dim > reduce_max_dim()) return EMB_EUNSUPPORTED;
  WsLayout lay;
  st = check_ws(ws, ws_bytes, batch->num_indices, M, tables->dim, &lay);
  if (st != EMB_OK) return st;
  if (batch->num_indices == 0) return EMB_OK;
  if (grad_out == nullptr || sort_perm == nullptr || seg_offsets == nullptr || unique_keys == nullptr ||
      num_unique == nullptr)
    return EMB_EINVAL;
  ReduceLaunch p{};
  p.grad_out = grad_out;
  p.perm = sort_perm;
  p.seg = seg_offsets;
  p.ukeys = unique_keys;
  p.num_unique = num_unique;
  p.offsets = batch->offsets;
  p.N = (int32_t)batch->num_indices;
  p.M = M;
  p.D = tables->dim;
  p.pool = pool;
  p.ws = ws;
  p.ws_bytes = ws_bytes;
  p.lay = lay;
  p.grad_rows = grad_rows;
  p.fuse = fuse != nullptr;
  p.opt = fuse ? fuse->opt : 0;
  p.dtype = tables->dtype;
  p.lr = fuse ? fuse->lr : 0.f;
  p.eps = fuse ? fuse->eps : 0.f;
  p.rounding = fuse ? fuse->rounding : 0;
  p.seed = fuse ? fuse->seed : 0;
  p.W = tables->weights;
  p.state = fuse ? fuse->state : nullptr;
  return hip_status(launch_grad_reduce(p, (hipStream_t)stream));
}

emb_status emb_sparse_update(const emb_tables* tables, const emb_update* update, const uint32_t* unique_keys,
                             const int32_t* num_unique, int64_t max_unique, const float* grad_rows, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  if ((st = check_update(update)) != EMB_OK) return st;
  if (max_unique < 0 || max_unique >= kMaxIndices) return max_unique < 0 ? EMB_EINVAL : EMB_EUNSUPPORTED;
  if (tables->dim > reduce_max_dim()) return EMB_EUNSUPPORTED;
  if (max_unique == 0) return EMB_OK;
  if (unique_keys == nullptr || num_unique == nullptr || grad_rows == nullptr) return EMB_EINVAL;
  UpdateLaunch p{};
  p.grad_rows = grad_rows;
  p.ukeys = unique_keys;
  p.num_unique = num_unique;
  p.max_unique = max_unique;
  p.rows = (uint32_t)R;
  p.D = tables->dim;
  p.opt = update->opt;
  p.dtype = tables->dtype;
  p.lr = update->lr;
  p.eps = update->eps;
  p.rounding = update->rounding;
  p.seed = update->seed;
  p.W = tables->weights;
  p.state = update->state;
  return hip_status(launch_sparse_update(p, (hipStream_t)stream));
}

size_t emb_route_workspace_size(int64_t num_indices, int64_t num_bags, int32_t world_size) {
  if (num_indices < 0 || num_indices >= kMaxIndices || num_bags < 0 || num_bags >= ((int64_t)1 << 31) ||
      world_size < 1 || world_size > kMaxRanks)
    return 0;
  const RoutePlan plan = route_plan(num_indices, num_bags);
  return align256(sizeof(int32_t) * (size_t)world_size * (size_t)(plan.nblocks > 0 ? plan.nblocks : 1));
}

emb_status emb_route_ids(const emb_tables* tables, const emb_batch* batch, int32_t world_size,
                         const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids, int32_t* send_pos,
                         int32_t* send_bag, void* ws, size_t ws_bytes, void* stream) {
  RouteLaunch p;
  emb_status st = route_prepare(tables, batch, world_size, shard_start, send_counts, send_ids, send_pos, send_bag, &p);
  if (st != EMB_OK) return st;
  if (p.N > 0 && ws == nullptr) return EMB_EINVAL;
  if (ws_bytes < emb_route_workspace_size(p.N, p.M, world_size)) return EMB_EWORKSPACE;
  p.ws = ws;
  return hip_status(launch_route(p, (hipStream_t)stream));
}

emb_status emb_route_ids_noalloc(const emb_tables* tables, const emb_batch* batch, int32_t world_size,
                                 const int64_t* shard_start, int32_t* send_counts, int32_t* send_ids,
                                 int32_t* send_pos, int32_t* send_bag, void* stream) {
  RouteLaunch p;
  emb_status st = route_prepare(tables, batch, world_size, shard_start, send_counts, send_ids, send_pos, send_bag, &p);
  if (st != EMB_OK) return st;
  if (!route_fits_scratch(p.N, p.M, world_size)) return EMB_EUNSUPPORTED;
  return hip_status(launch_route_noalloc(p, (hipStream_t)stream));
}

emb_status emb_validate_batch(const emb_tables* tables, const emb_batch* batch, int32_t* flag, void* stream) {
  TableOffsets ro;
  int64_t R = 0;
  emb_status st = check_tables(tables, &ro, &R);
  if (st != EMB_OK) return st;
  int32_t M = 0;
  st = check_batch(batch, tables->num_tables, &M);
  if (st != EMB_OK) return st;
  if (flag == nullptr) return EMB_EINVAL;
  ValidateLaunch p{};
  p.offsets = batch->offsets;
  p.idx = batch->indices;
  p.idx64 = batch->index_bytes == 8;
  p.ro = ro;
  p.T = tables->num_tables;
  p.B = batch->bags_per_table;
  p.M = M;
  p.N = batch->num_indices;
  p.flag = flag;
  return hip_status(launch_validate(p, (hipStream_t)stream));
}

}  // extern "C"
