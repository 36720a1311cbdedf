// Launch descriptors of the gfx950 kernels; the C-ABI layer fills them after
// checking its arguments on the host.
#pragma once

#include "emb_common.h"

namespace emb {

struct FwdLaunch {
  const void* W;
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;  // indices are int64
  TableOffsets ro;
  int32_t B, M, D, dtype, pool;
  float* out;
};
hipError_t launch_pool_fwd(const FwdLaunch& p, hipStream_t s);
int fwd_max_row_vectors();

// digit schedule of the LSD sort for keys of `key_bits` bits
struct SortPlan {
  int passes;
  int shift[kMaxPasses];
  int bits[kMaxPasses];
};
SortPlan make_sort_plan(int key_bits);

struct DedupLaunch {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  int32_t T, B, M;
  int64_t N;
  SortPlan plan;
  void* ws;
  size_t ws_bytes;
  WsLayout lay;
  uint32_t* unique_keys;
  int32_t* counts;
  int32_t* seg_offsets;
  int32_t* sort_perm;
  int32_t* num_unique;
  // 1: only kernels in which no workgroup waits for another (reduce-then-scan
  // sort passes and unique scan), so that any number of dedups may be in
  // flight on a device at once
  int32_t waitfree;
};
hipError_t launch_dedup(const DedupLaunch& p, hipStream_t s);

// A group dedup: the batches of a group sorted as one, each key carrying its
// batch's index above the key bits, then each batch's share split off into
// its own outputs and workspace, exactly as its own dedup would leave them.
constexpr int kMaxGroup = 16;
struct GroupMember {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64, B, M, N;
  int64_t P;                   // first position of this batch among the group's positions
  int32_t bags_per_block;      // of its prepare blocks
  uint32_t* unique_keys;       // its outputs, as emb_unique_ids fills them
  int32_t* counts;
  int32_t* seg_offsets;
  int32_t* sort_perm;
  int32_t* num_unique;
  int32_t* sorted_bag;         // in its own workspace (what its gradient reduce reads)
  int32_t* chunk_seg;
  uint64_t* uniq_words;        // its unique scan's per-tile words
  uint32_t* totals;            // a row of its workspace's digit totals (cleared by its unique scan)
  WsHeader* hdr;
};
struct GroupDedupLaunch {
  int32_t n;
  GroupMember m[kMaxGroup];
  TableOffsets ro;
  int32_t T;
  int32_t key_bits;            // bits of a key without the batch index
  int64_t N;                   // positions of all the batches
  SortPlan plan;               // over key_bits + the batch index bits
  void* ws;                    // the group's own workspace
  size_t ws_bytes;
  WsLayout lay;
};
hipError_t launch_dedup_group(const GroupDedupLaunch& p, hipStream_t s);

struct ReduceLaunch {
  const float* grad_out;
  const int32_t* perm;
  const int32_t* seg;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  const int32_t* offsets;
  int32_t N, M, D, pool;
  void* ws;
  size_t ws_bytes;
  WsLayout lay;
  float* grad_rows;  // may be null
  // fused optimizer (fuse = 0: reduce only)
  int32_t fuse, opt, dtype;
  float lr, eps;
  int32_t rounding;  // bf16 stores: 0 nearest even, 1 stochastic
  uint64_t seed;
  void* W;
  float* state;
};
hipError_t launch_grad_reduce(const ReduceLaunch& p, hipStream_t s);

struct UpdateLaunch {
  const float* grad_rows;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  int64_t max_unique;
  uint32_t rows;  // R: keys at or above it are skipped
  int32_t D, opt, dtype;
  float lr, eps;
  int32_t rounding;  // bf16 stores: 0 nearest even, 1 stochastic
  uint64_t seed;
  void* W;
  float* state;
};
hipError_t launch_sparse_update(const UpdateLaunch& p, hipStream_t s);
int reduce_max_dim();

struct RoutePlan {
  int32_t bags_per_block, nblocks;
};
RoutePlan route_plan(int64_t N, int64_t M);

struct RouteLaunch {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  ShardBounds sb;
  int32_t B, M, W;
  int64_t N;
  void* ws;  // [W][nblocks] int32
  int32_t* send_counts;
  int32_t* send_ids;
  int32_t* send_pos;
  int32_t* send_bag;
};
hipError_t launch_route(const RouteLaunch& p, hipStream_t s);
// the same on the library's per-device scratch array (p.ws is ignored);
// route_fits_scratch says whether a batch's per-block counts fit it
hipError_t launch_route_noalloc(RouteLaunch p, hipStream_t s);
bool route_fits_scratch(int64_t N, int64_t M, int32_t W);

struct ValidateLaunch {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  int32_t T, B, M;
  int64_t N;
  int32_t* flag;
};
hipError_t launch_validate(const ValidateLaunch& p, hipStream_t s);
hipError_t launch_zero_bytes(void* p, size_t bytes, hipStream_t s);
hipError_t launch_workspace_status(const void* ws, int32_t* status, hipStream_t s);

// host checks of a group of batches for emb_unique_ids_batched's group
// workspace: the number of batches, key bits, total ids and workspace size
emb_status check_dedup_group(const emb_tables* tables, int32_t n_batches, const emb_batch* batches, const void* ws,
                             size_t ws_bytes);

// host checks of one step of emb_pipeline_steps (defined with the C ABI)
emb_status check_pipeline_step(const emb_tables* tables, const emb_batch* batch, int32_t pool, const float* out,
                               const float* grad, const emb_update* update, const emb_dedup_set* d);
// the dedup part alone (a look-ahead batch, deduplicated for the next call)
emb_status check_dedup_step(const emb_tables* tables, const emb_batch* batch, const emb_dedup_set* d);

}  // namespace emb
