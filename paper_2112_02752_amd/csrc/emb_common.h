// Internal definitions shared by the gfx950 kernels of the embedding layer:
// workspace layout, launch constants, wavefront helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "emb.h"
#include "ws_words.h"

namespace emb {

constexpr int kWave = 64;

// ---------------------------------------------------------------- dedup sort
// LSD radix sort, one kernel per digit (co-resident tiles with prefix blocks,
// or reduce-then-scan: tile counts and a column scan before each pass).
constexpr int kMaxPasses = 4;
constexpr int kMaxDigitBits = 10;
constexpr int kMaxDigits = 1 << kMaxDigitBits;
constexpr int kSortThreads = 512;
// keys per thread: tiles of 2048 when every tile of a pass is resident at
// once (more blocks, shorter ranking), 4096 otherwise (fewer tiles per pass)
constexpr int kSortItemsCore = 4;
constexpr int kSortItemsMid = 5;
constexpr int kSortItemsWide = 8;
constexpr int kSortTileMin = kSortThreads * kSortItemsCore;

// unique / segment scan
constexpr int kUniqThreads = 256;
constexpr int kUniqItems = 8;
constexpr int kUniqTile = kUniqThreads * kUniqItems;

// tiles per group of the two-level prefix used when all tiles are resident
constexpr int kPrefixGroup = 16;
// digit-range prefix blocks (passes after the first, co-resident): digits per
// block, and the most tiles one of its threads sums
constexpr int kRangeDigits = 32;
constexpr int kRangeTiles = 16;
// bag offsets a first-pass tile stages in LDS to find the bag of each position
constexpr int kBagStage = 2048;

// prepare kernel (keys, bag ids, digit histograms)
constexpr int kPrepThreads = 256;
constexpr int kPrepMaxBags = 1024;     // bags of one block (offsets staged in LDS)
constexpr int kPrepPositions = 2048;   // positions a block aims at

// gradient reduce: segments longer than kChunk positions are "heavy" and are
// summed in aligned chunks of kChunk sorted positions, then combined.
constexpr int kChunk = 64;
// light segments each lane group carries at once, and the longest such
// segment (longer light ones are summed by a whole wavefront)
constexpr int kSlots = 2;
constexpr int kTinySeg = 16;
// heavy-segment combine: threads per block, chunks a block covers (a
// heavy segment that crosses blocks is finished by the last block to reach
// it, from one row per block)
constexpr int kCombineThreads = 1024;
constexpr int kCombineChunks = 64;

// Workspace header (device).  Every emb_unique_ids call on a workspace has a
// generation g = next_gen(gen) (ws_words.h): it tags the words the sort's
// workgroups publish to one another, so they never need clearing, and the
// error bits of that call, so that a failure belongs to one call only.
struct WsHeader {
  uint32_t gen;  // generation of the last dedup whose unique scan has run
  uint32_t cur;  // generation of the dedup in flight (written by its first sort pass)
  uint64_t err;  // (generation << 32) | error bits of the last call that set any
  // the first wait that ran out since the workspace was initialised: its site
  // code, block index and call generation; the number of waits that ran out
  uint32_t timeout_site, timeout_block, timeout_gen, timeouts;
  uint32_t pad[56];
};
static_assert(sizeof(WsHeader) == 256, "header is one 256-byte block");

// Workspace layout.  The front holds the batch's data arrays; the back (the
// last bytes of the caller's workspace, wherever it ends) holds the
// tag-checked coordination words of the sort.  Data of a call never lands on
// bytes another call used for coordination words: a smaller batch has a
// smaller front and its back lies inside the back of a larger one, so stale
// words in the back are always coordination words of another call, whose
// tags differ.
struct WsLayout {
  // front (offsets from the workspace base)
  size_t hdr, totals, keys_built, keys_a, keys_b, vals_a, vals_b, bags_a, bags_b, bag_of, sorted_keys, sorted_bag,
      group_perm, uniq_status, tile_counts, chunk_seg, partials, level2, arrivals, front;
  // back (offsets from the back base)
  size_t pass_status, rows, grp, later, back;
  size_t total;
  int64_t sort_tiles, uniq_tiles, chunks, groups, combine_blocks;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline WsLayout ws_layout(int64_t N, int64_t M, int32_t D) {
  (void)M;
  WsLayout L{};
  int64_t n = N > 0 ? N : 1;
  L.sort_tiles = (n + kSortTileMin - 1) / kSortTileMin;  // the most tiles any pass uses
  L.uniq_tiles = (n + kUniqTile - 1) / kUniqTile;
  L.chunks = (n + kChunk - 1) / kChunk;
  L.groups = (L.sort_tiles + kPrefixGroup - 1) / kPrefixGroup;
  size_t off = 0;
  L.hdr = off;
  off += sizeof(WsHeader);
  L.totals = off;
  off = align256(off + sizeof(uint32_t) * kMaxPasses * kMaxDigits);
  const size_t n4 = sizeof(uint32_t) * (size_t)n;
  L.keys_built = off;
  off = align256(off + n4);
  L.keys_a = off;
  off = align256(off + n4);
  L.keys_b = off;
  off = align256(off + n4);
  L.vals_a = off;
  off = align256(off + n4);
  L.vals_b = off;
  off = align256(off + n4);
  L.bags_a = off;
  off = align256(off + n4);
  L.bags_b = off;
  off = align256(off + n4);
  L.bag_of = off;
  off = align256(off + n4);
  L.sorted_keys = off;
  off = align256(off + n4);
  L.sorted_bag = off;
  off = align256(off + n4);
  // a group dedup's sort permutation (positions of all its batches), before
  // each batch's share is split off
  L.group_perm = off;
  off = align256(off + n4);
  L.uniq_status = off;
  off = align256(off + sizeof(uint64_t) * L.uniq_tiles);
  // plain digit counts of the passes whose tiles are not all resident at
  // once (tiles of at least kSortTileMin keys); never shares bytes with the
  // call-tagged words of the back region
  L.tile_counts = off;
  off = align256(off + sizeof(uint32_t) * (size_t)L.sort_tiles * kMaxDigits);
  L.chunk_seg = off;
  off = align256(off + sizeof(int32_t) * (L.chunks + 1));
  L.partials = off;
  off = align256(off + sizeof(float) * (size_t)L.chunks * 2 * (size_t)(D > 0 ? D : 1));
  L.combine_blocks = (L.chunks + kCombineChunks - 1) / kCombineChunks;
  L.level2 = off;
  off = align256(off + sizeof(uint64_t) * (size_t)L.combine_blocks * 2 * (size_t)(D > 0 ? D : 1));
  L.arrivals = off;
  off = align256(off + sizeof(uint32_t) * (size_t)L.combine_blocks);
  L.front = off;
  size_t b = 0;
  L.pass_status = b;
  b = align256(b + sizeof(uint64_t) * L.sort_tiles * kMaxDigits);
  L.rows = b;
  b = align256(b + sizeof(uint64_t) * L.sort_tiles * kMaxDigits);
  L.grp = b;
  b = align256(b + sizeof(uint64_t) * L.groups * kMaxDigits);
  L.later = b;
  b = align256(b + sizeof(uint64_t) * L.sort_tiles * (kMaxPasses - 1) * kMaxDigits);
  L.back = b;
  L.total = L.front + L.back;
  return L;
}

// base of the back region of a workspace of ws_bytes bytes (256-aligned)
inline char* ws_back(void* ws, size_t ws_bytes, const WsLayout& L) {
  return static_cast<char*>(ws) + ((ws_bytes - L.back) & ~(size_t)255);
}

// Global row offsets of the stacked tables, passed by value in kernel
// arguments (R < 2^32, so 32 bits per entry).
struct TableOffsets {
  uint32_t off[EMB_MAX_TABLES + 1];
};

// Routing: ranks of a sharding, their first global rows (by value in kernel
// arguments), bags one routing block covers at most, positions it aims at,
// threads of a per-rank scan block.
constexpr int kMaxRanks = EMB_MAX_RANKS;
struct ShardBounds {
  uint32_t off[kMaxRanks + 1];
};
constexpr int kRouteBags = 1024;
// owner counts the allocation-free routing entry point can hold (4 MiB), and
// the devices it keeps a scratch address for
constexpr size_t kRouteScratchInts = (size_t)1 << 20;
constexpr int kMaxDevices = 64;
constexpr int kRoutePositions = 256;
constexpr int kRouteScanThreads = 1024;

// ------------------------------------------------------------ device helpers

// id j of a batch whose indices are int32 (idx64 == 0) or int64; a valid id
// is below 2^31 (rows of a table), so both read the same value
__device__ __forceinline__ int32_t load_id(const void* idx, int32_t idx64, int64_t j) {
  return idx64 ? (int32_t) static_cast<const int64_t*>(idx)[j] : static_cast<const int32_t*>(idx)[j];
}

// One wavefront's values added to an LDS histogram.  The lanes that share
// lane 0's value add once, through lane 0: in a skewed batch many of a
// wavefront's keys are the hottest id (a fifth of them in the 50M-row
// workload), whose digit is one bin in every radix pass, and lane-by-lane
// atomics on one LDS word serialise.  Valid lanes are the low ones, so lane 0
// is valid whenever any lane is.  Called by every lane of the wavefront.
__device__ __forceinline__ void hist_add(uint32_t* hist, uint32_t d, bool valid, int lane) {
  const uint32_t d0 = (uint32_t)__shfl((int)d, 0, kWave);
  const uint64_t same = __ballot(valid && d == d0);
  if (valid && d != d0) atomicAdd(&hist[d], 1u);
  if (lane == 0 && same) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
}

// number of set bits of `mask` below this lane
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// device-coherent (agent scope) loads and stores of words other workgroups
// publish or poll; relaxed: a poll re-reads until the word carries its tag
__device__ __forceinline__ uint64_t ld_relaxed_u64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t atomic_add_u32(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Workgroups of `kernel` (with `threads` per block) that the current device
// holds at once, all compute units together (cached per device and kernel).
int resident_blocks(const void* kernel, int threads);

// The most workgroups of `kernel` that may wait on one another within one
// launch: one per compute unit (0 if a compute unit cannot hold one).  The
// occupancy API counts what an idle device holds; kernels that ran alongside
// on other streams can leave a compute unit's registers and LDS fragmented so
// that it takes only one such block until it drains, and a block per compute
// unit is what stays guaranteed once the others have finished (blocks go to
// the XCDs round-robin, the same number of compute units in each).
int coresident_limit(const void* kernel, int threads);

// Bound of a wait for a word another workgroup publishes, in ticks of the
// 100 MHz constant clock: 20 ms, thousands of times any wait of a healthy
// call.  Running out sets bit 0 of the call's error bits, records the wait,
// and lets the wave continue, so every wave always exits; the other waits of
// a call that has timed out give up at their next check of its error bits.
constexpr uint64_t kWaitTicks = 2000000;
// error bits of the dedup: a wait ran out (bit 0); digit totals inconsistent
// with the keys (bit 1).  The gradient reduce writes no table row when either
// is set for the dedup it follows.
constexpr uint32_t kDedupErrors = 3u;
// error bit of the gradient combine: one of its waits ran out
constexpr uint32_t kCombineError = 4u;

// Site codes of the waits: (kernel << 8) | (sort pass << 4) | wait.
enum WaitSite : uint32_t {
  kSiteTileOffsets = 0x100,  // co-resident tile: its final digit offsets
  kSiteGroupCounts = 0x102,  // first-pass prefix block: its group's counts
  kSiteGroupSums = 0x103,    // first-pass prefix block: every group's sum
  kSiteLaterCounts = 0x104,  // first-pass prefix block: later passes' counts
  kSiteRangeCounts = 0x105,  // range prefix block: its tiles' counts
  kSiteUnique = 0x200,       // unique look-back
  kSiteCombine = 0x300,      // gradient combine: crossing-segment rows
};

__device__ __forceinline__ uint64_t wait_clock() { return wall_clock64(); }

// error bits of call g (0 if the error word belongs to another call)
__device__ __forceinline__ uint32_t call_errors(const WsHeader* h, uint32_t g) {
  const uint64_t v = __hip_atomic_load(&h->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return err_bits_of(v, g);
}

// set `bits` among the error bits of call g; the word of an earlier call is
// replaced, not added to
__device__ __forceinline__ void flag_error(WsHeader* h, uint32_t g, uint32_t bits) {
  uint64_t old = __hip_atomic_load(&h->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  while (!__hip_atomic_compare_exchange_strong(&h->err, &old, err_word_with(old, g, bits), __ATOMIC_RELAXED,
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
  }
}

// a wait of call g that started at t0 has run out (or another wait of the call has)
__device__ __forceinline__ bool wait_over(const WsHeader* h, uint32_t g, uint64_t t0, uint32_t spins) {
  // the call's error word is read every 32nd retry (each read is a round
  // trip of its own, which a poll that succeeds on its next load would pay)
  if ((spins & 31u) == 0u && (call_errors(h, g) & 1u)) return true;
  return wait_clock() - t0 > kWaitTicks;
}

// a wait of call g ran out: set `bit` in its error bits and record the first such wait
__device__ __forceinline__ void flag_timeout(WsHeader* h, uint32_t g, uint32_t site, uint32_t bit = 1u) {
  flag_error(h, g, bit);
  atomicAdd(&h->timeouts, 1u);
  if (atomicCAS(&h->timeout_site, 0u, site) == 0u) {
    h->timeout_block = blockIdx.x;
    h->timeout_gen = g;
  }
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// inclusive wave scan (sum) of a 32-bit value
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    uint32_t t = __shfl_up(v, o, kWave);
    if (lane >= o) v += t;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_max(uint32_t v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    uint32_t t = __shfl_up(v, o, kWave);
    if (lane >= o) v = v > t ? v : t;
  }
  return v;
}

}  // namespace emb
