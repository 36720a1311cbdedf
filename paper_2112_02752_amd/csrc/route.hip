// Routing of a batch's ids to the owners of a row-range sharding of the
// stacked tables (gfx950): the step before the forward when the layer is
// spread over several devices, each owning a contiguous range of global rows.
//
//   owner(j)  = the rank r with shard[r] <= key(j) < shard[r+1]
//   send order: positions rank by rank, in position order within a rank
//
// Three kernels, none waiting on another block: a per-block owner histogram,
// one scan per rank over the blocks' counts, and a stable scatter.  A block is
// one wavefront over a range of consecutive bags, whose positions are
// consecutive too; their offsets are staged in LDS, so a position's bag is an
// LDS binary search and the stable rank among equal owners a few ballots.
#include <mutex>

#include "emb_common.h"
#include "kernels.h"

namespace emb {

namespace {

// Per-block owner counts of emb_route_ids_noalloc, for callers that cannot
// allocate: a device array that every call on a GPU shares (each GPU holds its
// own copy for the life of the process).  The count kernel writes every entry
// a call reads, so nothing in it needs clearing; calls that overlap on one GPU
// race on it.
static __device__ __align__(256) int32_t scratch[kRouteScratchInts];

// device address of this GPU's copy of `scratch`, found once per device with
// that device current (the host-side name `scratch` is not a device address)
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};

hipError_t scratch_for_current_device(int32_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

struct RouteArgs {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  ShardBounds sb;
  int32_t B, M, W, owner_bits, bags_per_block, nblocks;
  int32_t N;
  int32_t* counts;  // [W][nblocks]: a block's count of each owner, then its base within the owner's range
  int32_t* send_counts;
  int32_t* send_ids;
  int32_t* send_pos;
  int32_t* send_bag;
};

// Stage the block's bag offsets and the shard bounds in LDS; returns the
// block's bag range [b0, b1).
__device__ __forceinline__ void stage(const RouteArgs& a, int32_t* s_off, uint32_t* s_sb, int& b0, int& b1) {
  const int lane = threadIdx.x;
  b0 = blockIdx.x * a.bags_per_block;
  b1 = min(a.M, b0 + a.bags_per_block);
  for (int i = lane; i <= b1 - b0; i += kWave) s_off[i] = a.offsets[b0 + i];
  for (int i = lane; i <= a.W; i += kWave) s_sb[i] = a.sb.off[i];
  __syncthreads();
}

// bag (block-relative) holding position j: the last staged offset <= j that
// starts a non-empty bag
__device__ __forceinline__ int bag_of(const int32_t* s_off, int nb, int32_t j) {
  int lo = 0, hi = nb - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_off[mid] <= j) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// owner rank of a global key: the last bound <= key
__device__ __forceinline__ int owner_of(const uint32_t* s_sb, int W, uint32_t key) {
  int lo = 0, hi = W - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_sb[mid] <= key) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(kWave) void k_route_count(RouteArgs a) {
  __shared__ int32_t s_off[kRouteBags + 1];
  __shared__ uint32_t s_sb[kMaxRanks + 1];
  __shared__ int32_t s_hist[kMaxRanks];
  const int lane = threadIdx.x;
  int b0, b1;
  for (int r = lane; r < a.W; r += kWave) s_hist[r] = 0;
  stage(a, s_off, s_sb, b0, b1);
  const int nb = b1 - b0;
  const int32_t p0 = s_off[0], p1 = s_off[nb];
  for (int32_t j = p0 + lane; j < p1; j += kWave) {
    const int bl = bag_of(s_off, nb, j);
    const uint32_t key = a.ro.off[(b0 + bl) / a.B] + (uint32_t)load_id(a.idx, a.idx64, j);
    atomicAdd(&s_hist[owner_of(s_sb, a.W, key)], 1);
  }
  __syncthreads();
  for (int r = lane; r < a.W; r += kWave) a.counts[(size_t)r * a.nblocks + blockIdx.x] = s_hist[r];
}

// One block per rank: exclusive scan of the rank's per-block counts in block
// order (a thread sums a contiguous run of blocks, the run sums are scanned
// in LDS); the total is the rank's send count.
__global__ __launch_bounds__(kRouteScanThreads) void k_route_scan(RouteArgs a) {
  __shared__ int32_t s_w[kRouteScanThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
  int32_t* c = a.counts + (size_t)blockIdx.x * a.nblocks;
  const int per = (a.nblocks + kRouteScanThreads - 1) / kRouteScanThreads;
  const int q0 = min(a.nblocks, tid * per), q1 = min(a.nblocks, q0 + per);
  int32_t sum = 0;
  for (int q = q0; q < q1; ++q) sum += c[q];
  const uint32_t incl = wave_incl_sum((uint32_t)sum);
  if (lane == kWave - 1) s_w[w] = (int32_t)incl;
  __syncthreads();
  int32_t run = (int32_t)incl - sum;
  for (int ww = 0; ww < w; ++ww) run += s_w[ww];
  for (int q = q0; q < q1; ++q) {
    const int32_t x = c[q];
    c[q] = run;
    run += x;
  }
  if (tid == kRouteScanThreads - 1) a.send_counts[blockIdx.x] = run;
}

__global__ __launch_bounds__(kWave) void k_route_scatter(RouteArgs a) {
  __shared__ int32_t s_off[kRouteBags + 1];
  __shared__ uint32_t s_sb[kMaxRanks + 1];
  __shared__ int32_t s_run[kMaxRanks];
  const int lane = threadIdx.x;
  int b0, b1;
  // where this block's positions of each owner go: the owner's start in the
  // send order (exclusive scan of the send counts) plus the block's base
  uint32_t carry = 0;
  for (int r0 = 0; r0 < a.W; r0 += kWave) {
    const int r = r0 + lane;
    const uint32_t cnt = r < a.W ? (uint32_t)a.send_counts[r] : 0u;
    const uint32_t incl = wave_incl_sum(cnt);
    if (r < a.W) s_run[r] = (int32_t)(carry + incl - cnt) + a.counts[(size_t)r * a.nblocks + blockIdx.x];
    carry += (uint32_t)__shfl((int)incl, kWave - 1, kWave);
  }
  stage(a, s_off, s_sb, b0, b1);
  const int nb = b1 - b0;
  const int32_t p0 = s_off[0], p1 = s_off[nb];
  for (int32_t jb = p0; jb < p1; jb += kWave) {
    const int32_t j = jb + lane;
    const bool valid = j < p1;
    int bl = 0, o = 0;
    uint32_t key = 0;
    if (valid) {
      bl = bag_of(s_off, nb, j);
      key = a.ro.off[(b0 + bl) / a.B] + (uint32_t)load_id(a.idx, a.idx64, j);
      o = owner_of(s_sb, a.W, key);
    }
    // lanes with the same owner, by one ballot per owner bit
    uint64_t peers = __ballot(valid);
    for (int bit = 0; bit < a.owner_bits; ++bit) {
      const bool x = (o >> bit) & 1;
      const uint64_t bx = __ballot(x);
      peers &= x ? bx : ~bx;
    }
    const int32_t dst = valid ? s_run[o] + (int32_t)lanes_below(peers) : 0;
    if (valid && (uint32_t)dst < (uint32_t)a.N) {  // always, for well-formed offsets
      a.send_ids[dst] = (int32_t)(key - s_sb[o]);
      a.send_pos[dst] = j;
      a.send_bag[dst] = b0 + bl;
    }
    __builtin_amdgcn_wave_barrier();
    // the lowest lane of each owner advances that owner's position
    if (valid && lanes_below(peers) == 0) s_run[o] += __popcll(peers);
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace

RoutePlan route_plan(int64_t N, int64_t M) {
  RoutePlan p{};
  const int64_t want = M > 0 && N > 0 ? (int64_t)kRoutePositions * M / N : 1;
  p.bags_per_block = (int32_t)(want < 1 ? 1 : (want > kRouteBags ? kRouteBags : want));
  p.nblocks = M > 0 ? (int32_t)((M + p.bags_per_block - 1) / p.bags_per_block) : 0;
  return p;
}

bool route_fits_scratch(int64_t N, int64_t M, int32_t W) {
  const RoutePlan plan = route_plan(N, M);
  return (int64_t)W * (int64_t)(plan.nblocks > 0 ? plan.nblocks : 1) <= (int64_t)kRouteScratchInts;
}

hipError_t launch_route_noalloc(RouteLaunch p, hipStream_t s) {
  int32_t* ptr = nullptr;
  const hipError_t e = scratch_for_current_device(&ptr);
  if (e != hipSuccess) return e;
  p.ws = ptr;
  return launch_route(p, s);
}

hipError_t launch_route(const RouteLaunch& p, hipStream_t s) {
  const RoutePlan plan = route_plan(p.N, p.M);
  if (p.N == 0 || plan.nblocks == 0) return launch_zero_bytes(p.send_counts, sizeof(int32_t) * (size_t)p.W, s);
  RouteArgs a{};
  a.offsets = p.offsets;
  a.idx = p.idx;
  a.idx64 = p.idx64;
  a.ro = p.ro;
  a.sb = p.sb;
  a.B = p.B;
  a.M = p.M;
  a.W = p.W;
  a.N = (int32_t)p.N;
  a.owner_bits = 0;
  while ((1 << a.owner_bits) < p.W) ++a.owner_bits;
  a.bags_per_block = plan.bags_per_block;
  a.nblocks = plan.nblocks;
  a.counts = static_cast<int32_t*>(p.ws);
  a.send_counts = p.send_counts;
  a.send_ids = p.send_ids;
  a.send_pos = p.send_pos;
  a.send_bag = p.send_bag;
  hipLaunchKernelGGL(k_route_count, dim3((unsigned)a.nblocks), dim3(kWave), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_route_scan, dim3((unsigned)a.W), dim3(kRouteScanThreads), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_route_scatter, dim3((unsigned)a.nblocks), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace emb
