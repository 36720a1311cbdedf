// ID dedup of a batch (gfx950): keys, stable LSD radix sort, unique runs.
//
//   key[j]   = row_offset[t(j)] + idx[j]
//   perm     = stable ascending sort of positions by key
//   unique_keys / seg_offsets / counts = the runs of equal sorted keys
//
// Kernels, in stream order:
//  1. k_sort_pass (once per digit): a tile ranks its keys with wavefront
//     ballots (the lanes sharing a digit are found with one ballot per digit
//     bit, the rank is a masked popcount), reorders them in LDS by digit and
//     writes them out in digit runs.  Each digit's offset among earlier tiles
//     comes from one of two schemes.  When every tile of a pass is resident
//     at once, the tile publishes its digit counts (an LDS histogram) as soon
//     as its keys are loaded, and prefix blocks launched after the tiles sum
//     the published counts and publish final offsets while the tiles rank;
//     the first pass also finds each position's bag.  Otherwise k_prepare
//     first writes every position's bag id (and key, for several tables), and
//     each pass is preceded by k_tile_counts (every tile's digit counts) and
//     k_column_scan (per digit, the prefix of those counts over the tiles,
//     and the digit's total), so that the pass reads its offsets with no
//     wait.  Ranks follow position order within a tile and tiles follow
//     position order, so every pass is stable and so is the whole sort.
//  2. k_unique: head flags key[k] != key[k-1], a block scan plus a look-back
//     of (number of heads, last head position) gives every head its segment
//     index and the length of the previous segment; when its tiles are not
//     all resident at once, k_uniq_counts and k_uniq_scan compute each
//     tile's (heads, last head) prefix first instead of the look-back.
#include "emb_common.h"
#include "kernels.h"

namespace emb {

SortPlan make_sort_plan(int key_bits) {
  SortPlan p{};
  if (key_bits < 1) key_bits = 1;
  const int passes = (key_bits + kMaxDigitBits - 1) / kMaxDigitBits;
  int shift = 0;
  for (int i = 0; i < passes; ++i) {
    const int left = key_bits - shift;
    const int b = (left + (passes - i) - 1) / (passes - i);
    p.shift[i] = shift;
    p.bits[i] = b;
    shift += b;
  }
  p.passes = passes;
  return p;
}

namespace {

// status word flags of the unique scan's look-back: aggregate, inclusive prefix
constexpr uint64_t kFlagAgg = 1, kFlagInc = 2;

// ------------------------------------------------------------------ prepare

struct PrepArgs {
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  int32_t B, M, bags_per_block;
  uint32_t* keys_out;  // null for int32 ids of one table (the ids are the keys)
  int32_t* bag_of;
  uint32_t key_hi;     // or-ed into every key (a group dedup's batch index bits; 0 otherwise)
};

// Used when the tiles of a pass are not all resident at once.  A block owns a
// contiguous range of bags and therefore of positions.  The bags' offsets are
// staged in LDS; every thread takes positions of the range in strides, finds
// each one's bag by a binary search in LDS, and writes the bag id (and the key
// for several tables).
// `a` supplies offsets, idx, idx64, ro, B, M, bags_per_block, keys_out,
// bag_of and key_hi (one batch's, with keys_out and bag_of at its positions)
template <typename A>
__device__ __forceinline__ void prepare_block(const A& a, int block, int32_t* s_off) {
  constexpr int UN = 8;
  const int tid = threadIdx.x;
  const int m0 = block * a.bags_per_block;
  const int nb = min(a.M - m0, a.bags_per_block);
  for (int i = tid; i <= nb; i += kPrepThreads) s_off[i] = a.offsets[m0 + i];
  __syncthreads();
  const int j0 = s_off[0], j1 = s_off[nb];
  for (int jb = j0; jb < j1; jb += kPrepThreads * UN) {
    int32_t id[UN];
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int j = jb + u * kPrepThreads + tid;
      id[u] = j < j1 ? load_id(a.idx, a.idx64, j) : 0;
    }
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int j = jb + u * kPrepThreads + tid;
      if (j < j1) {
        // last bag i with s_off[i] <= j (empty bags share an offset with the next one)
        int lo = 0, hi = nb - 1;
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (s_off[mid] <= j) lo = mid; else hi = mid - 1;
        }
        const int m = m0 + lo;
        const uint32_t key = (a.ro.off[m / a.B] + (uint32_t)id[u]) | a.key_hi;
        a.bag_of[j] = m;
        if (a.keys_out) a.keys_out[j] = key;
      }
    }
  }
}

__global__ __launch_bounds__(kPrepThreads) void k_prepare(PrepArgs a) {
  __shared__ int32_t s_off[kPrepMaxBags + 1];
  prepare_block(a, blockIdx.x, s_off);
}

// ------------------------------------------------------------- sort pass

struct PassArgs {
  const uint32_t* keys_in;
  const int32_t* vals_in;  // null: values are the positions
  const int32_t* bags_in;  // bag of each element (travels with it through the passes)
  uint32_t* keys_out;
  int32_t* vals_out;
  int32_t* bags_out;
  uint32_t* totals;        // this pass's digit totals (global histogram)
  uint32_t* prev_totals;   // the previous pass's totals, cleared here (null for the first pass)
  uint64_t* status;        // co-resident: each tile's final digit offsets (tag << 32 | offset): [tiles][status_stride]
  uint64_t* rows;          // published tile counts (tag << 32 | count): [tiles][status_stride]
  uint64_t* grp;           // published group sums, same form: [groups][status_stride]
  WsHeader* hdr;
  // first pass with co-resident tiles: the bag of every position is found here
  // (offsets, idx, ro, B, M); the first pass also clears the unique scan's
  // look-back words
  int32_t search_bags;
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  TableOffsets ro;
  int32_t B, M, T;
  uint64_t* uniq_status;
  int32_t uniq_tiles;
  int32_t N, ntiles, shift, bits, pass, status_stride;
  const uint32_t* prefix;  // reduce-then-scan (tiles not co-resident): [tiles][status_stride], each digit's
                           // count in the tiles before this one, from k_tile_counts and k_column_scan
  int32_t xcd_order;       // 1: tiles in XCD order (xcd_tile), for passes of many tiles that read their offsets
  int32_t coresident;      // 1: every tile is resident at once (tile = block index, prefix blocks
                           //    after the tiles publish each tile's final digit offsets)
  int32_t prefix_mode;     // co-resident: kPrefixGroups or kPrefixRanges
  // first co-resident pass: the later passes' digit counts are published in
  // `later` [tiles][kMaxPasses - 1][status_stride] and summed into their
  // totals (`totals_all` [kMaxPasses][kMaxDigits]) by the prefix blocks
  uint64_t* later;
  uint32_t* totals_all;
  int32_t npass;
  int32_t pass_shift[kMaxPasses], pass_bits[kMaxPasses];
  // the last pass of a group sort (split_n > 0): values and bags go straight
  // to each member's own buffers instead of vals_out and bags_out; a key's
  // member is key >> split_bits (0 with one member), its sorted position in
  // the member dst - split_P[m] (< split_N[m]), its value less split_P[m]
  int32_t split_n, split_bits;
  int32_t split_P[kMaxGroup], split_N[kMaxGroup];
  int32_t* split_perm[kMaxGroup];
  int32_t* split_bag[kMaxGroup];
};

// Prefix blocks of a co-resident pass.  Groups: one block per kPrefixGroup
// tiles, digit totals found from the tiles' counts (three exchanges through
// memory: counts, group sums, final offsets).  Ranges: one block per
// kRangeDigits digits over all tiles, with digit totals known before the pass
// (two exchanges: counts, final offsets).
constexpr int kPrefixGroups = 1, kPrefixRanges = 2;

// Exclusive scan of n = 2^RB counters held in LDS, by kSortThreads threads.
template <int RB>
__device__ __forceinline__ void block_excl_scan(uint32_t* arr, uint32_t* s_wsum) {
  constexpr int ND = 1 << RB;
  constexpr int EPT = ND >= kSortThreads ? ND / kSortThreads : 1;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  uint32_t v[EPT];
  uint32_t sum = 0;
  const bool own = tid * EPT < ND;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    v[e] = own ? arr[tid * EPT + e] : 0u;
    sum += v[e];
  }
  const uint32_t incl = wave_incl_sum(sum);
  if (lane == kWave - 1) s_wsum[w] = incl;
  __syncthreads();
  uint32_t run = incl - sum;
  for (int ww = 0; ww < w; ++ww) run += s_wsum[ww];
  if (own) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      arr[tid * EPT + e] = run;
      run += v[e];
    }
  }
  __syncthreads();
}

// Two-level prefix of a co-resident pass, for digit d.  Published words are
// (tag << 32 | count).  A batch of words is loaded together; the words that
// do not carry this pass's tag yet are loaded again together after a short
// sleep, so every retry round costs one memory round trip however many words
// are stale.  The wait is bounded in time (kWaitTicks).
template <int K>
__device__ __forceinline__ void poll_batch(const uint64_t* base, int stride, int lo, int n, int d, uint64_t tag,
                                           WsHeader* h, uint32_t g, uint32_t site, uint64_t (&v)[K]) {
  // words past n stand in as ready
  uint32_t stale = 0;
#pragma unroll
  for (int i = 0; i < K; ++i) stale |= (i < n && !word_current(v[i], tag)) ? (1u << i) : 0u;
  uint32_t spins = 0;
  const uint64_t t0 = stale ? wait_clock() : 0;
  while (stale) {
    if (wait_over(h, g, t0, ++spins)) {
      flag_timeout(h, g, site);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
    const uint64_t* p = base + (size_t)lo * stride + d;
#pragma unroll
    for (int i = 0; i < K; ++i)
      if (stale & (1u << i)) v[i] = ld_relaxed_u64(p + (size_t)i * stride);
    stale = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) stale |= (i < n && !word_current(v[i], tag)) ? (1u << i) : 0u;
  }
}

// The last tile of a group of kPrefixGroup tiles reads the group's published
// counts for digit d (one batch), publishes the group's sum and returns the
// in-group exclusive prefixes of the group's tiles as 16-bit pairs (a group
// of co-resident tiles holds fewer than 2^16 keys before its last tile), and
// its own.
static_assert((kPrefixGroup - 1) * kSortThreads * kSortItemsWide < 65536, "in-group prefixes fit 16 bits");
__device__ __forceinline__ void group_counts(const uint64_t* rows, uint64_t* grp, int stride, int g, int g0, int g1,
                                             int d, uint64_t tag, WsHeader* h, uint32_t gcall, uint32_t site,
                                             uint32_t (&pk)[kPrefixGroup / 2],
                                             uint32_t& last_pre) {
  uint64_t v[kPrefixGroup];
  const int n = g1 - g0;
#pragma unroll
  for (int i = 0; i < kPrefixGroup; ++i) v[i] = i < n ? ld_relaxed_u64(rows + (size_t)(g0 + i) * stride + d) : 0;
  poll_batch<kPrefixGroup>(rows, stride, g0, n, d, tag, h, gcall, site, v);
  uint32_t run = 0;
  last_pre = 0;
#pragma unroll
  for (int i = 0; i < kPrefixGroup; ++i) {
    if (i % 2 == 0) pk[i / 2] = run;
    else pk[i / 2] |= run << 16;
    if (i == n - 1) last_pre = run;
    if (i < n) run += word_count(v[i]);
  }
  st_u64(grp + (size_t)g * stride + d, word_make(tag, run));
}

// Sum of the published group sums of digit d before group g, and of all of
// them (the digit's total), loaded in batches of kPrefixGroup.
__device__ __forceinline__ void group_sums(const uint64_t* grp, int stride, int g, int ngroups, int d, uint64_t tag,
                                           WsHeader* h, uint32_t gcall, uint32_t site, uint32_t& before,
                                           uint32_t& total) {
  before = total = 0;
  for (int base = 0; base < ngroups; base += kPrefixGroup) {
    const int n = min(kPrefixGroup, ngroups - base);
    uint64_t gv[kPrefixGroup];
#pragma unroll
    for (int i = 0; i < kPrefixGroup; ++i) gv[i] = i < n ? ld_relaxed_u64(grp + (size_t)(base + i) * stride + d) : 0;
    poll_batch<kPrefixGroup>(grp, stride, base, n, d, tag, h, gcall, site, gv);
#pragma unroll
    for (int i = 0; i < kPrefixGroup; ++i) {
      if (i < n) {
        const uint32_t c = word_count(gv[i]);
        total += c;
        if (base + i < g) before += c;
      }
    }
  }
}

// A prefix block of a co-resident pass (one per group of kPrefixGroup tiles,
// launched after the tiles): for each digit d it reads its group's published
// tile counts (in-group exclusive prefixes and the group's sum), publishes the
// group's sum, reads every group's sum (the groups before its own, and the
// digit's total), forms the digit bases by an exclusive scan of the totals and
// publishes for every tile of its group the final output offset of digit d in
// that tile's status word.  The tiles rank and reorder their keys meanwhile.
template <int RB>
__device__ __forceinline__ void sort_prefix_block(const PassArgs& a, uint32_t gcall, uint64_t tag, uint32_t* s_base,
                                                  uint32_t* s_wsum, uint32_t* s_pre) {
  constexpr int ND = 1 << RB;
  constexpr int DPT = (ND + kSortThreads - 1) / kSortThreads;
  const int tid = threadIdx.x;
  const int g = blockIdx.x - a.ntiles, g0 = g * kPrefixGroup;
  const int g1 = min(a.ntiles, g0 + kPrefixGroup);
  const int ngroups = (a.ntiles + kPrefixGroup - 1) / kPrefixGroup;
  uint32_t excl[DPT];
  // the in-group prefixes (16-bit pairs) wait in LDS: s_pre[j * ND + d]
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = tid + k * kSortThreads;
    if (d < ND) {
      uint32_t pk[kPrefixGroup / 2], unused;
      group_counts(a.rows, a.grp, a.status_stride, g, g0, g1, d, tag, a.hdr, gcall,
                   kSiteGroupCounts | ((uint32_t)a.pass << 4), pk, unused);
#pragma unroll
      for (int j = 0; j < kPrefixGroup / 2; ++j) s_pre[j * ND + d] = pk[j];
    }
  }
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = tid + k * kSortThreads;
    excl[k] = 0;
    if (d < ND) {
      uint32_t total = 0;
      group_sums(a.grp, a.status_stride, g, ngroups, d, tag, a.hdr, gcall, kSiteGroupSums | ((uint32_t)a.pass << 4),
                 excl[k], total);
      s_base[d] = total;
    }
  }
  __syncthreads();
  block_excl_scan<RB>(s_base, s_wsum);
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = tid + k * kSortThreads;
    if (d < ND) {
      const uint32_t gb = s_base[d] + excl[k];
#pragma unroll
      for (int i = 0; i < kPrefixGroup; ++i) {
        const uint32_t pre = (s_pre[(i / 2) * ND + d] >> (16 * (i % 2))) & 0xffffu;
        if (g0 + i < g1) st_u64(a.status + (size_t)(g0 + i) * a.status_stride + d, word_make(tag, gb + pre));
      }
    }
  }
  if (a.later) {
    // after the final offsets are out: this group's counts of the later
    // passes' digits are added to their totals
    const size_t lstride = (size_t)(kMaxPasses - 1) * a.status_stride;
    const int n = g1 - g0;
    for (int p = 1; p < a.npass; ++p) {
#pragma unroll
      for (int k = 0; k < DPT; ++k) {
        const int d = tid + k * kSortThreads;
        if (d < (1 << a.pass_bits[p])) {
          const uint64_t* lb = a.later + (size_t)(p - 1) * a.status_stride;
          uint64_t v[kPrefixGroup];
#pragma unroll
          for (int i = 0; i < kPrefixGroup; ++i) v[i] = i < n ? ld_relaxed_u64(lb + (size_t)(g0 + i) * lstride + d) : 0;
          poll_batch<kPrefixGroup>(lb, (int)lstride, g0, n, d, tag, a.hdr, gcall,
                                   kSiteLaterCounts | ((uint32_t)a.pass << 4), v);
          uint32_t sum = 0;
#pragma unroll
          for (int i = 0; i < kPrefixGroup; ++i) sum += i < n ? word_count(v[i]) : 0u;
          if (sum) atomic_add_u32(&a.totals_all[p * kMaxDigits + d], sum);
        }
      }
    }
  }
}

// A digit-range prefix block (passes after the first, co-resident): block b
// owns digits [b*DB, (b+1)*DB) of every tile.  The digit bases come from the
// totals counted during the first pass; a thread sums one digit's published
// counts over a chunk of consecutive tiles, the chunk sums are scanned in LDS,
// and the thread publishes the final offset of its digit for each tile of its
// chunk.
template <int RB>
__device__ __forceinline__ void sort_prefix_range(const PassArgs& a, uint32_t gcall, uint64_t tag, uint32_t* s_base,
                                                  uint32_t* s_wsum, uint32_t* s_cs) {
  constexpr int ND = 1 << RB;
  constexpr int DPT = (ND + kSortThreads - 1) / kSortThreads;
  constexpr int DB = ND < kRangeDigits ? ND : kRangeDigits;
  constexpr int NC = kSortThreads / DB;
  const int tid = threadIdx.x;
  const int dl = tid % DB, c = tid / DB;
  const int d = (blockIdx.x - a.ntiles) * DB + dl;
  const int ct = (a.ntiles + NC - 1) / NC;  // at most kRangeTiles (checked by the host)
  const int t0 = c * ct, n = max(0, min(a.ntiles - t0, ct));
  // the digit bases, found while the tiles load their keys
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int dd = tid + k * kSortThreads;
    if (dd < ND) s_base[dd] = a.totals[dd];
  }
  __syncthreads();
  block_excl_scan<RB>(s_base, s_wsum);
  // this digit's counts in the chunk's tiles
  uint64_t v[kRangeTiles];
#pragma unroll
  for (int i = 0; i < kRangeTiles; ++i)
    v[i] = i < n ? ld_relaxed_u64(a.rows + (size_t)(t0 + i) * a.status_stride + d) : 0;
  poll_batch<kRangeTiles>(a.rows, a.status_stride, t0, n, d, tag, a.hdr, gcall,
                          kSiteRangeCounts | ((uint32_t)a.pass << 4), v);
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < kRangeTiles; ++i) sum += i < n ? word_count(v[i]) : 0u;
  s_cs[c * DB + dl] = sum;
  __syncthreads();
  uint32_t run = s_base[d];
  for (int cc = 0; cc < c; ++cc) run += s_cs[cc * DB + dl];
#pragma unroll
  for (int i = 0; i < kRangeTiles; ++i) {
    if (i < n) {
      st_u64(a.status + (size_t)(t0 + i) * a.status_stride + d, word_make(tag, run));
      run += word_count(v[i]);
    }
  }
}

// Bag of each of this thread's positions of a tile: the bag holding position
// j is the last m with offsets[m] <= j.  One offset in every S (S chosen so
// the samples fit one per thread) narrows the tile's bags to a few sample
// intervals whose offsets are staged in LDS.  Every nonempty staged bag that
// overlaps the tile writes its id at its first position in the tile, and an
// inclusive max-scan over the tile's positions carries each id forward to
// the bag's other positions (bag ids grow with position).  Intervals that do
// not fit the stage are searched in global memory.  `s_work` holds
// one int per position of the tile.
template <int IT>
__device__ __forceinline__ void find_tile_bags(const PassArgs& a, int tile, int32_t* s_boff, int* s_lohi,
                                               int32_t* s_work, uint32_t* s_wmax, int32_t (&bag)[IT]) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  const int64_t p0 = (int64_t)tile * (kSortThreads * IT);
  const int64_t p1 = min(p0 + (kSortThreads * IT), (int64_t)a.N);
  const int S = (a.M + kSortThreads) / kSortThreads;  // samples offsets[0], offsets[S], ... up to offsets[M]
  const int nsamp = a.M / S + 1;
  int samp = 0;
  if (tid < nsamp) samp = a.offsets[min(tid * S, a.M)];
  if (tid == 0) s_lohi[0] = s_lohi[1] = 0;
  __syncthreads();
  // samples are nondecreasing: count those <= p0 and <= p1 - 1
  const uint64_t le0 = __ballot(tid < nsamp && samp <= p0);
  const uint64_t le1 = __ballot(tid < nsamp && samp <= p1 - 1);
  if (lane == 0) {
    atomicAdd(&s_lohi[0], (int)__popcll(le0));
    atomicAdd(&s_lohi[1], (int)__popcll(le1));
  }
  __syncthreads();
  const int m_lo = (s_lohi[0] - 1) * S;                    // a bag at or before the tile's first bag
  const int m_hi = min((s_lohi[1] - 1) * S + S, a.M);      // an offset index at or after its last bag's end
  const int nst = m_hi - m_lo + 1;
  if (nst <= kBagStage + 1) {
    for (int i = tid; i < nst; i += kSortThreads) s_boff[i] = a.offsets[m_lo + i];
    // ids are stored plus one, so that 0 means "no bag starts here"
    for (int i = tid; i < (kSortThreads * IT); i += kSortThreads) s_work[i] = 0;
    __syncthreads();
    for (int i = tid; i < nst - 1; i += kSortThreads) {
      const int64_t st = s_boff[i], en = s_boff[i + 1];
      if (st < en && st < p1 && en > p0) s_work[(st > p0 ? st : p0) - p0] = m_lo + i + 1;
    }
    __syncthreads();
    uint32_t v[IT];
    uint32_t run = 0;
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const uint32_t x = (uint32_t)s_work[tid * IT + k];
      run = x > run ? x : run;
      v[k] = run;
    }
    const uint32_t incl = wave_incl_max(run);
    if (lane == kWave - 1) s_wmax[w] = incl;
    uint32_t carry = __shfl_up(incl, 1, kWave);
    if (lane == 0) carry = 0;
    __syncthreads();
    for (int ww = 0; ww < w; ++ww) carry = s_wmax[ww] > carry ? s_wmax[ww] : carry;
#pragma unroll
    for (int k = 0; k < IT; ++k) s_work[tid * IT + k] = (int32_t)(v[k] > carry ? v[k] : carry);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int64_t j = p0 + (int64_t)w * (kWave * IT) + i * kWave + lane;
      bag[i] = j < p1 ? s_work[j - p0] - 1 : 0;
    }
    __syncthreads();  // s_work is reused by the caller
    return;
  }
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const int64_t j = p0 + (int64_t)w * (kWave * IT) + i * kWave + lane;
    bag[i] = 0;
    if (j < p1) {
      int lo = 0, hi = nst - 2;  // last idx in [0, nst-2] with offset <= j
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.offsets[m_lo + mid] <= j) lo = mid; else hi = mid - 1;
      }
      bag[i] = m_lo + lo;
    }
  }
}

// Workgroups are handed to the 8 XCDs in turn (block b to XCD b % 8).  In
// XCD order consecutive tiles run on one XCD: the runs that neighbouring
// tiles write for one digit are adjacent in the output, so their partial
// cache lines meet in that XCD's L2.  A bijection of [0, n): XCD x takes a
// contiguous range of tiles.  Used for reduce-then-scan passes of more than
// kXcdOrderMinTiles tiles (measured: 8% faster passes over 3.3M keys, slower
// ones for a pass of a few hundred tiles).
constexpr int kSortXcds = 8;
constexpr int kXcdOrderMinTiles = 512;
__device__ inline int xcd_tile(int b, int n) {
  const int x = b % kSortXcds, i = b / kSortXcds, q = n / kSortXcds, r = n % kSortXcds;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

// LDS of a sort pass, one arena whose regions serve several phases (byte
// offsets):
//   [cnt]    16-bit per-wave digit counters [NW][ND] (ranking, reorder)
//   [tstart] the tile's digit starts [ND], [gbase] digit bases [ND]
//   [keys]   reorder buffer [TILE]: keys, then bags; before the reorder the
//            bag search's per-position work area
//   [vals]   reorder buffer [TILE]: values; before the reorder the bag
//            search's staged offsets
// Before the ranking [cnt]..[gbase] hold the co-resident pass's published
// histograms (u32 [kMaxPasses][ND]).  A prefix block uses the arena from its
// start for its in-group prefixes and digit bases.
template <int RB, int IT>
struct PassLds {
  static constexpr int ND = 1 << RB;
  static constexpr int TILE = kSortThreads * IT;
  static constexpr int NW = kSortThreads / kWave;
  static constexpr int kCnt = 0;
  static constexpr int kTstart = kCnt + NW * ND * 2;
  static constexpr int kGbase = kTstart + ND * 4;
  static constexpr int kKeys = kGbase + ND * 4;
  static constexpr int kVals = kKeys + TILE * 4;
  static constexpr int kValsWords = TILE > kBagStage + 1 ? TILE : kBagStage + 1;
  static constexpr int kTileBytes = kVals + kValsWords * 4;
  static constexpr int kPrefixBytes = ((kPrefixGroup / 2) * ND + ND) * 4;
  static constexpr int kRangeBytes = (ND + kSortThreads) * 4;
  static constexpr int kBytes0 = kTileBytes > kPrefixBytes ? kTileBytes : kPrefixBytes;
  static constexpr int kBytes = kBytes0 > kRangeBytes ? kBytes0 : kRangeBytes;
  static_assert(kKeys >= 4 * kMaxPasses * ND, "the published histograms fit before the reorder buffers");
  static_assert(TILE < 65536, "per-wave counters fit 16 bits");
};

template <int RB, int IT>
__global__ __launch_bounds__(kSortThreads, 4) void k_sort_pass(PassArgs a) {
  using Lds = PassLds<RB, IT>;
  constexpr int ND = Lds::ND;
  constexpr int TILE = Lds::TILE;
  constexpr int NW = Lds::NW;
  constexpr int DPT = (ND + kSortThreads - 1) / kSortThreads;
  __shared__ __align__(16) unsigned char s_arena[Lds::kBytes];
  __shared__ uint32_t s_wsum[NW];
  __shared__ int s_lohi[2];
  __shared__ uint32_t s_toff[EMB_MAX_TABLES];
  uint16_t(*s_cnt)[ND] = reinterpret_cast<uint16_t(*)[ND]>(s_arena + Lds::kCnt);
  uint32_t* s_tstart = reinterpret_cast<uint32_t*>(s_arena + Lds::kTstart);
  uint32_t* s_gbase = reinterpret_cast<uint32_t*>(s_arena + Lds::kGbase);
  uint32_t* s_keys = reinterpret_cast<uint32_t*>(s_arena + Lds::kKeys);
  int32_t* s_vals = reinterpret_cast<int32_t*>(s_arena + Lds::kVals);
  // published histograms: row 0 this pass's digits, row p a later pass's
  uint32_t* s_hist = reinterpret_cast<uint32_t*>(s_arena);

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  // co-resident: the histograms start from zero (the per-wave counters are
  // cleared after them); otherwise the per-wave counters at once
  if (a.coresident)
    for (int i = tid; i < kMaxPasses * ND; i += kSortThreads) s_hist[i] = 0u;
  else
    for (int i = tid; i < NW * ND / 2; i += kSortThreads) reinterpret_cast<uint32_t*>(s_arena + Lds::kCnt)[i] = 0u;
  if (a.search_bags && a.T > 1)
    for (int t = tid; t < a.T; t += kSortThreads) s_toff[t] = a.ro.off[t];
  // the previous pass is complete: clear its totals for the next call
  if (blockIdx.x == 0 && a.prev_totals)
    for (int d = tid; d < kMaxDigits; d += kSortThreads) a.prev_totals[d] = 0u;
  __syncthreads();
  const int tile = a.xcd_order && (int)blockIdx.x < a.ntiles ? xcd_tile((int)blockIdx.x, a.ntiles) : (int)blockIdx.x;
  const uint32_t mask = (1u << a.bits) - 1u;
  // the call's generation (the header's advances once per call, in the
  // unique scan) and this pass's tag
  const uint32_t gcall = next_gen(a.hdr->gen);
  const uint64_t tag = word_tag(gcall, (uint32_t)a.pass);
  if (a.pass == 0 && blockIdx.x == 0 && tid == 0) a.hdr->cur = gcall;
  if (a.coresident && (int)blockIdx.x >= a.ntiles) {
    uint32_t* s_pre = reinterpret_cast<uint32_t*>(s_arena);
    uint32_t* s_base = s_pre + (kPrefixGroup / 2) * ND;
    if (a.prefix_mode == kPrefixRanges) sort_prefix_range<RB>(a, gcall, tag, s_pre, s_wsum, s_pre + ND);
    else sort_prefix_block<RB>(a, gcall, tag, s_base, s_wsum, s_pre);
    return;
  }
  const int64_t wbase = (int64_t)tile * TILE + w * (kWave * IT);

  uint32_t key[IT], dig[IT], lrank[IT];
  int32_t val[IT], bag[IT];
  if (a.pass == 0) {
    // the unique scan of this call starts from cleared look-back words
    for (int i = blockIdx.x * kSortThreads + tid; i < a.uniq_tiles; i += a.ntiles * kSortThreads)
      a.uniq_status[i] = 0;
  }
  // The tile's digit counts are published as soon as its digits are known
  // (from an LDS histogram), so that the other tiles' prefixes advance while
  // this tile finds its bags, ranks and reorders its keys.
  auto publish_counts = [&]() {
    if (!a.coresident) return;  // the offsets were computed before the pass
#pragma unroll
    for (int i = 0; i < IT; ++i) hist_add(s_hist, dig[i], wbase + i * kWave + lane < a.N, lane);
    if (a.later) {
      // and the later passes' digits
      for (int p = 1; p < a.npass; ++p) {
        const uint32_t pm = (1u << a.pass_bits[p]) - 1u;
#pragma unroll
        for (int i = 0; i < IT; ++i)
          hist_add(s_hist + p * ND, (key[i] >> a.pass_shift[p]) & pm, wbase + i * kWave + lane < a.N, lane);
      }
    }
    __syncthreads();
    uint64_t* row = a.rows + (size_t)tile * a.status_stride;
#pragma unroll
    for (int k = 0; k < DPT; ++k) {
      const int d = tid + k * kSortThreads;
      if (d < ND) st_u64(row + d, word_make(tag, s_hist[d]));
    }
    if (a.later) {
      for (int p = 1; p < a.npass; ++p) {
        uint64_t* lrow = a.later + ((size_t)tile * (kMaxPasses - 1) + (p - 1)) * a.status_stride;
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
          const int d = tid + k * kSortThreads;
          if (d < (1 << a.pass_bits[p])) st_u64(lrow + d, word_make(tag, s_hist[p * ND + d]));
        }
      }
    }
  };

  if (a.search_bags) {
    // the ids are loaded first: their loads overlap the bag search
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int64_t pos = wbase + i * kWave + lane;
      key[i] = pos < a.N ? (uint32_t)load_id(a.idx, a.idx64, pos) : 0u;
      val[i] = pos < a.N ? (int32_t)pos : 0;
    }
    // with one table the ids are the keys: the counts go out before the bag search
    const bool one_table = a.T == 1;
    if (one_table) {
#pragma unroll
      for (int i = 0; i < IT; ++i) dig[i] = (key[i] >> a.shift) & mask;
      publish_counts();
    }
    find_tile_bags<IT>(a, tile, s_vals, s_lohi, reinterpret_cast<int32_t*>(s_keys), s_wsum, bag);
    if (!one_table) {
#pragma unroll
      for (int i = 0; i < IT; ++i) {
        key[i] += s_toff[bag[i] / a.B];
        dig[i] = (key[i] >> a.shift) & mask;
      }
      publish_counts();
    }
  } else {
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int64_t pos = wbase + i * kWave + lane;
      const bool valid = pos < a.N;
      key[i] = valid ? a.keys_in[pos] : 0u;
      val[i] = valid ? (a.vals_in ? a.vals_in[pos] : (int32_t)pos) : 0;
      bag[i] = valid ? a.bags_in[pos] : 0;
      dig[i] = (key[i] >> a.shift) & mask;
    }
    publish_counts();
  }
  // the histograms are out: the per-wave counters start from zero
  if (a.coresident) {
    __syncthreads();
    for (int i = tid; i < NW * ND / 2; i += kSortThreads) reinterpret_cast<uint32_t*>(s_arena + Lds::kCnt)[i] = 0u;
    __syncthreads();
  }

  // rank each element among the earlier elements of its wave with its digit
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const bool valid = wbase + i * kWave + lane < a.N;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < a.bits; ++b) {
      const bool bit = (dig[i] >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    lrank[i] = 0;
    if (valid) {
      const uint32_t r = lanes_below(peers);
      const uint32_t c = s_cnt[w][dig[i]];
      lrank[i] = c + r;
      if (r == 0) s_cnt[w][dig[i]] = (uint16_t)(c + (uint32_t)__popcll(peers));
    }
  }
  __syncthreads();

  // per digit: exclusive prefix over the waves (the sum is the tile's count)
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = tid + k * kSortThreads;
    if (d < ND) {
      uint32_t run = 0;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) {
        const uint32_t c = s_cnt[ww][d];
        s_cnt[ww][d] = (uint16_t)run;
        run += c;
      }
      s_tstart[d] = run;
      if (!a.coresident) s_gbase[d] = a.totals[d];
    }
  }

  uint32_t excl[DPT];
  __syncthreads();
  block_excl_scan<RB>(s_tstart, s_wsum);
  if (!a.coresident) block_excl_scan<RB>(s_gbase, s_wsum);

  // reorder the tile in LDS by digit (stable); only tile-local offsets are
  // needed, so this is done before the wait for the other tiles' counts.
  // Each element's slot is kept for the bags' round.
  uint32_t lp[IT];
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const bool valid = wbase + i * kWave + lane < a.N;
    lp[i] = valid ? s_tstart[dig[i]] + s_cnt[w][dig[i]] + lrank[i] : 0xffffffffu;
    if (valid) {
      s_keys[lp[i]] = key[i];
      s_vals[lp[i]] = val[i];
    }
  }

  if (a.coresident) {
    // the final offset of every digit arrives from this tile's group's
    // prefix block; only this tile's words are polled
#pragma unroll
    for (int k = 0; k < DPT; ++k) {
      const int d = tid + k * kSortThreads;
      excl[k] = 0;
      if (d < ND) {
        uint64_t fv[1] = {ld_relaxed_u64(a.status + (size_t)tile * a.status_stride + d)};
        poll_batch<1>(a.status, a.status_stride, tile, 1, d, tag, a.hdr, gcall,
                      kSiteTileOffsets | ((uint32_t)a.pass << 4), fv);
        excl[k] = word_count(fv[0]);
      }
    }
    // the final offsets replace the digit bases
#pragma unroll
    for (int k = 0; k < DPT; ++k) {
      const int d = tid + k * kSortThreads;
      if (d < ND) s_gbase[d] = 0;
    }
  } else {
#pragma unroll
    for (int k = 0; k < DPT; ++k) {
      const int d = tid + k * kSortThreads;
      excl[k] = d < ND ? a.prefix[(size_t)tile * a.status_stride + d] : 0u;
    }
  }
#pragma unroll
  for (int k = 0; k < DPT; ++k) {
    const int d = tid + k * kSortThreads;
    if (d < ND) s_gbase[d] += excl[k];
  }
  __syncthreads();

  // write the tile out in digit runs: keys and values, then the bags
  // through the values' buffer, each slot to the destination found for it
  // (in a group sort's last pass, values and bags to the key's member)
  const int64_t tstart = (int64_t)tile * TILE;
  const int nvalid = (int)min((int64_t)TILE, (int64_t)a.N - tstart);
  uint32_t dst[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int s = tid + j * kSortThreads;
    dst[j] = 0xffffffffu;
    if (s < nvalid) {
      const uint32_t k = s_keys[s];
      const uint32_t d = (k >> a.shift) & mask;
      dst[j] = s_gbase[d] + (uint32_t)s - s_tstart[d];
      if (dst[j] < (uint32_t)a.N) {
        a.keys_out[dst[j]] = k;
        if (a.split_n > 0) {
          const uint32_t m = a.split_n > 1 ? k >> a.split_bits : 0u;
          const uint32_t o = dst[j] - (uint32_t)a.split_P[m < (uint32_t)a.split_n ? m : 0];
          if (m < (uint32_t)a.split_n && o < (uint32_t)a.split_N[m]) a.split_perm[m][o] = s_vals[s] - a.split_P[m];
          else flag_error(a.hdr, gcall, 2u);  // a key outside its member's share
        } else {
          a.vals_out[dst[j]] = s_vals[s];
        }
      } else {
        flag_error(a.hdr, gcall, 2u);  // digit totals inconsistent with the keys
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < IT; ++i)
    if (lp[i] != 0xffffffffu) s_vals[lp[i]] = bag[i];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    if (dst[j] >= (uint32_t)a.N) continue;
    const int s = tid + j * kSortThreads;
    if (a.split_n > 0) {
      const uint32_t m = a.split_n > 1 ? s_keys[s] >> a.split_bits : 0u;
      if (m < (uint32_t)a.split_n) {
        const uint32_t o = dst[j] - (uint32_t)a.split_P[m];
        if (o < (uint32_t)a.split_N[m]) a.split_bag[m][o] = s_vals[s];
      }
    } else {
      a.bags_out[dst[j]] = s_vals[s];
    }
  }
}

// ------------------------------------------------- reduce-then-scan passes
//
// When the tiles of a pass cannot all be resident at once, a pass takes three
// kernels instead of a look-back: each tile's digit counts, then per digit the
// exclusive prefix of those counts over the tiles (and the digit's total), and
// the pass itself, which reads its tile's offsets with no wait.

struct CountArgs {
  const uint32_t* keys;
  int32_t N, shift, bits, stride;
  uint32_t* counts;  // [tiles][stride]
};

template <int IT>
__global__ __launch_bounds__(kSortThreads) void k_tile_counts(CountArgs a) {
  __shared__ uint32_t s_hist[kMaxDigits];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  const int nd = 1 << a.bits;
  const uint32_t mask = (uint32_t)nd - 1u;
  for (int i = tid; i < nd; i += kSortThreads) s_hist[i] = 0u;
  __syncthreads();
  const int64_t wbase = (int64_t)blockIdx.x * (kSortThreads * IT) + w * (kWave * IT);
  uint32_t key[IT];
#pragma unroll
  for (int i = 0; i < IT; ++i) {
    const int64_t pos = wbase + i * kWave + lane;
    key[i] = pos < a.N ? a.keys[pos] : 0u;
  }
#pragma unroll
  for (int i = 0; i < IT; ++i) hist_add(s_hist, (key[i] >> a.shift) & mask, wbase + i * kWave + lane < a.N, lane);
  __syncthreads();
  for (int d = tid; d < nd; d += kSortThreads) a.counts[(size_t)blockIdx.x * a.stride + d] = s_hist[d];
}

struct ColScanArgs {
  uint32_t* counts;  // in: counts, out: exclusive prefixes over the tiles
  uint32_t* totals;  // out: each digit's total
  int32_t tiles, nd, stride;
};

// One block per kColDigits digits; thread (digit, chunk of consecutive
// tiles): the chunk's counts are loaded kColBatch at a time, the chunk sums
// scanned in LDS, and the chunk rewritten with running prefixes.
constexpr int kColDigits = 16;
constexpr int kColChunks = 64;
constexpr int kColBatch = 16;
__global__ __launch_bounds__(kColDigits * kColChunks) void k_column_scan(ColScanArgs a) {
  __shared__ uint32_t s_cs[kColChunks][kColDigits];
  const int tid = threadIdx.x, dl = tid % kColDigits, c = tid / kColDigits;
  const int d = blockIdx.x * kColDigits + dl;
  const int ct = (a.tiles + kColChunks - 1) / kColChunks;
  const int t0 = min(a.tiles, c * ct), t1 = min(a.tiles, t0 + ct);
  const bool ok = d < a.nd;
  uint32_t sum = 0;
  for (int tb = t0; tb < t1; tb += kColBatch) {
    uint32_t v[kColBatch];
#pragma unroll
    for (int i = 0; i < kColBatch; ++i) v[i] = ok && tb + i < t1 ? a.counts[(size_t)(tb + i) * a.stride + d] : 0u;
#pragma unroll
    for (int i = 0; i < kColBatch; ++i) sum += v[i];
  }
  s_cs[c][dl] = sum;
  __syncthreads();
  uint32_t run = 0, total = 0;
  for (int cc = 0; cc < kColChunks; ++cc) {
    if (cc < c) run += s_cs[cc][dl];
    total += s_cs[cc][dl];
  }
  if (ok && c == 0) a.totals[d] = total;
  for (int tb = t0; tb < t1; tb += kColBatch) {
    uint32_t v[kColBatch];
#pragma unroll
    for (int i = 0; i < kColBatch; ++i) v[i] = ok && tb + i < t1 ? a.counts[(size_t)(tb + i) * a.stride + d] : 0u;
#pragma unroll
    for (int i = 0; i < kColBatch; ++i) {
      if (ok && tb + i < t1) {
        a.counts[(size_t)(tb + i) * a.stride + d] = run;
        run += v[i];
      }
    }
  }
}

// ----------------------------------------------------------------- unique

struct UniqArgs {
  const uint32_t* skeys;
  int32_t N, ntiles, nchunks;
  uint32_t* ukeys;
  int32_t* counts;
  int32_t* seg;
  int32_t* num_unique;
  int32_t* chunk_seg;  // [nchunks+1]: segment of position c*kChunk; [nchunks] = U
  uint64_t* status;    // [tiles], zeroed by k_prepare of the same call
  uint32_t* prev_totals;  // the last sort pass's totals, cleared here
  const uint64_t* prefix;  // reduce-then-scan: each tile's (heads, last head position + 1) over the
                           // tiles before it, from k_uniq_counts and k_uniq_scan; null: look-back
  WsHeader* hdr;
  uint32_t key_mask;       // applied to the keys written out (a group dedup drops the batch index bits)
};

// status word: flag [63:62], head count [61:31], last head position + 1 [30:0]
__device__ __forceinline__ uint64_t pack_uniq(uint64_t flag, uint32_t c, uint32_t q) {
  return (flag << 62) | ((uint64_t)c << 31) | (uint64_t)q;
}

constexpr int kUniqWindows = 4;  // look-back words per lane and round

// Reduce-then-scan unique (the tiles are not all resident at once): each
// tile's number of heads and last head position + 1, then their exclusive
// (sum, max) scan over the tiles by one block.
struct UniqCountArgs {
  const uint32_t* skeys;
  int32_t N;
  uint64_t* out;  // [tiles]: pack_uniq(0, heads, last head position + 1)
};

__device__ __forceinline__ void uniq_counts_tile(const UniqCountArgs& a, int tile, uint32_t* s_c, uint32_t* s_q) {
  constexpr int NW = kUniqThreads / kWave;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  const int64_t tbase = (int64_t)tile * kUniqTile;
  uint32_t cur[kUniqItems], prv[kUniqItems];
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) {
    const int64_t pos = tbase + tid + i * kUniqThreads;
    cur[i] = pos < a.N ? a.skeys[pos] : 0u;
    prv[i] = pos > 0 && pos < a.N ? a.skeys[pos - 1] : 0u;
  }
  uint32_t c = 0, q = 0;
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) {
    const int64_t pos = tbase + tid + i * kUniqThreads;
    if (pos < a.N && (pos == 0 || cur[i] != prv[i])) {
      ++c;
      q = max(q, (uint32_t)pos + 1u);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    c += __shfl_xor(c, o, kWave);
    q = max(q, (uint32_t)__shfl_xor((int)q, o, kWave));
  }
  if (lane == 0) {
    s_c[w] = c;
    s_q[w] = q;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t tc = 0, tq = 0;
    for (int ww = 0; ww < NW; ++ww) {
      tc += s_c[ww];
      tq = max(tq, s_q[ww]);
    }
    a.out[tile] = pack_uniq(0, tc, tq);
  }
}

__global__ __launch_bounds__(kUniqThreads) void k_uniq_counts(UniqCountArgs a) {
  __shared__ uint32_t s_c[kUniqThreads / kWave], s_q[kUniqThreads / kWave];
  uniq_counts_tile(a, blockIdx.x, s_c, s_q);
}

constexpr int kUniqScanThreads = 1024;
__device__ __forceinline__ void uniq_scan_block(uint64_t* words, int32_t tiles, uint32_t* s_c, uint32_t* s_q) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  const int per = (tiles + kUniqScanThreads - 1) / kUniqScanThreads;
  const int t0 = min(tiles, tid * per), t1 = min(tiles, t0 + per);
  uint32_t c = 0, q = 0;
  for (int t = t0; t < t1; ++t) {
    const uint64_t v = words[t];
    c += (uint32_t)(v >> 31) & 0x7fffffffu;
    q = max(q, (uint32_t)v & 0x7fffffffu);
  }
  const uint32_t ci = wave_incl_sum(c), qi = wave_incl_max(q);
  if (lane == kWave - 1) {
    s_c[w] = ci;
    s_q[w] = qi;
  }
  uint32_t qb = (uint32_t)__shfl_up((int)qi, 1, kWave);
  if (lane == 0) qb = 0;
  __syncthreads();
  uint32_t rc = ci - c, rq = qb;
  for (int ww = 0; ww < w; ++ww) {
    rc += s_c[ww];
    rq = max(rq, s_q[ww]);
  }
  for (int t = t0; t < t1; ++t) {
    const uint64_t v = words[t];
    words[t] = pack_uniq(0, rc, rq);
    rc += (uint32_t)(v >> 31) & 0x7fffffffu;
    rq = max(rq, (uint32_t)v & 0x7fffffffu);
  }
}

__global__ __launch_bounds__(kUniqScanThreads) void k_uniq_scan(uint64_t* words, int32_t tiles) {
  __shared__ uint32_t s_c[kUniqScanThreads / kWave], s_q[kUniqScanThreads / kWave];
  uniq_scan_block(words, tiles, s_c, s_q);
}

__device__ __forceinline__ void unique_tile(const UniqArgs& a, const int tile) {
  constexpr int NW = kUniqThreads / kWave;
  __shared__ uint32_t s_keys[kUniqTile];
  __shared__ uint32_t s_wc[NW], s_wq[NW];
  __shared__ uint32_t s_pc, s_pq, s_prev, s_fail;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & (kWave - 1);
  const int64_t tbase = (int64_t)tile * kUniqTile;
  const bool last_tile = tbase + kUniqTile >= (int64_t)a.N;
  // this call's generation (its first sort pass recorded it); the sort is
  // complete, so its error bits are final: clear the last pass's totals and
  // make the call's generation the header's
  const uint32_t gcall = a.hdr->cur;
  if (tile == 0) {
    for (int d = tid; d < kMaxDigits; d += kUniqThreads) a.prev_totals[d] = 0u;
    if (tid == 0) a.hdr->gen = gcall;
  }
  if (tid == 0) s_fail = call_errors(a.hdr, gcall) & kDedupErrors;
  __syncthreads();
  if (s_fail) {
    // the sort failed: no unique ids, so neither a fused nor an unfused
    // update touches any row
    if (tile == 0 && tid == 0) {
      a.num_unique[0] = 0;
      a.seg[0] = a.N;
    }
    return;
  }
  // every load of the tile is issued before the first LDS store
  uint32_t kv[kUniqItems];
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) {
    const int64_t pos = tbase + tid + i * kUniqThreads;
    kv[i] = pos < a.N ? a.skeys[pos] : 0u;
  }
  const uint32_t before = (tid == 0 && tbase > 0) ? a.skeys[tbase - 1] : 0u;
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) s_keys[tid + i * kUniqThreads] = kv[i];
  if (tid == 0) s_prev = before;
  __syncthreads();

  uint32_t c = 0, q = 0, heads = 0;
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) {
    const int s = tid * kUniqItems + i;
    const int64_t pos = tbase + s;
    if (pos < a.N) {
      const uint32_t prev = s > 0 ? s_keys[s - 1] : s_prev;
      if (pos == 0 || s_keys[s] != prev) {
        ++c;
        q = (uint32_t)pos + 1u;
        heads |= 1u << i;
      }
    }
  }
  // block exclusive scan of (count sum, last-head max)
  const uint32_t ci = wave_incl_sum(c);
  const uint32_t qi = wave_incl_max(q);
  if (lane == kWave - 1) {
    s_wc[w] = ci;
    s_wq[w] = qi;
  }
  const uint32_t q_before_lane = __shfl_up(qi, 1, kWave);
  __syncthreads();
  uint32_t c_ex = ci - c, q_ex = lane > 0 ? q_before_lane : 0u;
  uint32_t tile_c = 0, tile_q = 0;
  for (int ww = 0; ww < NW; ++ww) {
    if (ww < w) {
      c_ex += s_wc[ww];
      q_ex = max(q_ex, s_wq[ww]);
    }
    tile_c += s_wc[ww];
    tile_q = max(tile_q, s_wq[ww]);
  }
  if (a.prefix) {
    if (tid == 0) {
      const uint64_t v = a.prefix[tile];
      s_pc = (uint32_t)(v >> 31) & 0x7fffffffu;
      s_pq = (uint32_t)v & 0x7fffffffu;
    }
  } else if (w == 0) {
    // wave-parallel look-back: in a round, lane k reads the status of tiles
    // j - k - 64 i for i < kUniqWindows (one round trip for all of them); the
    // windows are then taken in order up to the first word not yet published
    // or the first inclusive prefix
    uint32_t pc = 0, pq = 0;
    bool gave_up = false;
    if (tile == 0) {
      if (lane == 0) st_u64(a.status, pack_uniq(kFlagInc, tile_c, tile_q));
    } else {
      if (lane == 0) st_u64(a.status + tile, pack_uniq(kFlagAgg, tile_c, tile_q));
      int j = tile - 1;
      uint32_t spins = 0;
      const uint64_t t0 = wait_clock();
      while (!gave_up) {
        uint64_t sv[kUniqWindows];
#pragma unroll
        for (int i = 0; i < kUniqWindows; ++i) {
          const int jj = j - i * kWave - lane;
          sv[i] = jj >= 0 ? ld_relaxed_u64(a.status + jj) : 0;
        }
        uint32_t c = 0, q = 0;
        int took = 0;
        bool done = false, stop = false;
#pragma unroll
        for (int i = 0; i < kUniqWindows; ++i) {
          if (!stop) {
            const int jj = j - i * kWave - lane;
            const uint64_t flag = sv[i] >> 62;
            const uint64_t not_ready = __ballot(!(jj >= 0 && flag != 0));
            const uint64_t inc = __ballot(jj >= 0 && flag == kFlagInc);
            const int first_nr = not_ready ? __builtin_ctzll(not_ready) : kWave;
            const int first_inc = inc ? __builtin_ctzll(inc) : kWave;
            done = first_inc < first_nr;
            const int take = done ? first_inc + 1 : first_nr;
            if (lane < take) {
              c += (uint32_t)((sv[i] >> 31) & 0x7fffffffu);
              q = max(q, (uint32_t)(sv[i] & 0x7fffffffu));
            }
            took += take;
            stop = done || take < kWave;
          }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
          c += __shfl_xor(c, o, kWave);
          const uint32_t qo = __shfl_xor(q, o, kWave);
          q = q > qo ? q : qo;
        }
        pc += c;
        pq = max(pq, q);
        if (done) break;
        j -= took;
        if (took == 0) {
          gave_up = __builtin_amdgcn_readfirstlane((int)wait_over(a.hdr, gcall, t0, ++spins)) != 0;
          if (gave_up) {
            if (lane == 0) flag_timeout(a.hdr, gcall, kSiteUnique);
          } else {
            __builtin_amdgcn_s_sleep(1);
          }
        }
      }
      // a tile whose look-back gave up publishes no inclusive prefix, so no
      // later tile builds on its short one
      if (lane == 0 && !gave_up) st_u64(a.status + tile, pack_uniq(kFlagInc, pc + tile_c, max(pq, tile_q)));
    }
    if (lane == 0) {
      s_pc = pc;
      s_pq = pq;
      // A tile whose look-back gave up writes nothing.  The last tile
      // reports no unique ids if any look-back of the call gave up (the
      // gradient reduce also checks the call's error bits).
      s_fail = gave_up || (last_tile && (call_errors(a.hdr, gcall) & 1u));
    }
  }
  __syncthreads();
  if (s_fail) {
    if (last_tile && tid == 0) a.num_unique[0] = 0;
    return;
  }
  uint32_t u = s_pc + c_ex;
  uint32_t lastq = max(s_pq, q_ex);
#pragma unroll
  for (int i = 0; i < kUniqItems; ++i) {
    const int s = tid * kUniqItems + i;
    const int64_t pos = tbase + s;
    if (pos < a.N) {
      if (heads & (1u << i)) {
        a.ukeys[u] = s_keys[s] & a.key_mask;
        a.seg[u] = (int32_t)pos;
        if (u > 0) a.counts[u - 1] = (int32_t)pos - (int32_t)(lastq - 1u);
        lastq = (uint32_t)pos + 1u;
        ++u;
      }
      if (pos % kChunk == 0) a.chunk_seg[pos / kChunk] = (int32_t)u - 1;
      if (pos == a.N - 1) {
        a.num_unique[0] = (int32_t)u;
        a.seg[u] = a.N;
        a.counts[u - 1] = a.N - (int32_t)(lastq - 1u);
        a.chunk_seg[a.nchunks] = (int32_t)u;
      }
    }
  }
}

__global__ __launch_bounds__(kUniqThreads) void k_unique(UniqArgs a) { unique_tile(a, blockIdx.x); }

__global__ void k_unique_empty(int32_t* num_unique, int32_t* seg) {
  if (threadIdx.x == 0) {
    num_unique[0] = 0;
    seg[0] = 0;
  }
}

template <int RB, int IT>
hipError_t launch_pass(const PassArgs& pa, int tiles, hipStream_t s) {
  hipLaunchKernelGGL((k_sort_pass<RB, IT>), dim3((unsigned)tiles), dim3(kSortThreads), 0, s, pa);
  return hipGetLastError();
}

template <int IT>
const void* pass_kernel_bits(int bits) {
  switch (bits) {
    case 1: return reinterpret_cast<const void*>(&k_sort_pass<1, IT>);
    case 2: return reinterpret_cast<const void*>(&k_sort_pass<2, IT>);
    case 3: return reinterpret_cast<const void*>(&k_sort_pass<3, IT>);
    case 4: return reinterpret_cast<const void*>(&k_sort_pass<4, IT>);
    case 5: return reinterpret_cast<const void*>(&k_sort_pass<5, IT>);
    case 6: return reinterpret_cast<const void*>(&k_sort_pass<6, IT>);
    case 7: return reinterpret_cast<const void*>(&k_sort_pass<7, IT>);
    case 8: return reinterpret_cast<const void*>(&k_sort_pass<8, IT>);
    case 9: return reinterpret_cast<const void*>(&k_sort_pass<9, IT>);
    default: return reinterpret_cast<const void*>(&k_sort_pass<10, IT>);
  }
}

template <int IT>
hipError_t launch_pass_bits(const PassArgs& pa, int tiles, hipStream_t s) {
  switch (pa.bits) {
    case 1: return launch_pass<1, IT>(pa, tiles, s);
    case 2: return launch_pass<2, IT>(pa, tiles, s);
    case 3: return launch_pass<3, IT>(pa, tiles, s);
    case 4: return launch_pass<4, IT>(pa, tiles, s);
    case 5: return launch_pass<5, IT>(pa, tiles, s);
    case 6: return launch_pass<6, IT>(pa, tiles, s);
    case 7: return launch_pass<7, IT>(pa, tiles, s);
    case 8: return launch_pass<8, IT>(pa, tiles, s);
    case 9: return launch_pass<9, IT>(pa, tiles, s);
    case 10: return launch_pass<10, IT>(pa, tiles, s);
    default: return hipErrorInvalidValue;
  }
}

const void* pass_kernel(int it, int bits) {
  switch (it) {
    case kSortItemsCore: return pass_kernel_bits<kSortItemsCore>(bits);
    case kSortItemsMid: return pass_kernel_bits<kSortItemsMid>(bits);
    default: return pass_kernel_bits<kSortItemsWide>(bits);
  }
}

}  // namespace

// the wait-free dedup uses 2048-key tiles up to this many tiles (about a
// million keys), 4096-key tiles beyond
constexpr int kWaitfreeSmallTiles = 512;

hipError_t launch_dedup(const DedupLaunch& p, hipStream_t s) {
  char* ws = static_cast<char*>(p.ws);
  const WsLayout& L = p.lay;
  char* back = ws_back(p.ws, p.ws_bytes, L);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  if (p.N == 0) {
    hipLaunchKernelGGL(k_unique_empty, dim3(1), dim3(64), 0, s, p.num_unique, p.seg_offsets);
    return hipGetLastError();
  }
  const int N = (int)p.N;
  const int uniq_tiles = (N + kUniqTile - 1) / kUniqTile;
  const int nchunks = (N + kChunk - 1) / kChunk;
  int max_bits = 1;
  for (int i = 0; i < p.plan.passes; ++i) max_bits = p.plan.bits[i] > max_bits ? p.plan.bits[i] : max_bits;
  const int status_stride = 1 << max_bits;
  // Co-resident passes, when every tile of a pass and its prefix blocks fit
  // one block per compute unit (coresident_limit): tile = block index, bags
  // found by the first pass, two-level published-count prefix, with the
  // smallest tiles that fit.  Otherwise a prepare kernel (bags, keys) and
  // 4096-key tiles, each pass preceded by its tile counts and column scan.
  // A co-resident pass also runs its prefix blocks after the tiles: one per
  // group of kPrefixGroup tiles for the first pass, one per kRangeDigits
  // digits for the later ones (their digit totals are counted during the
  // first pass), unless the tiles are too many for a range block's threads
  // or the digits do not shrink from pass to pass.
  int sort_it = 0, core_tiles = 0, core_groups = 0, ranges = 0;
  auto prefix_blocks = [&](int ps) {
    if (ps == 0 || !ranges) return core_groups;
    const int nd = 1 << p.plan.bits[ps];
    return nd / (nd < kRangeDigits ? nd : kRangeDigits);
  };
  for (const int it : {kSortItemsCore, kSortItemsMid, kSortItemsWide}) {
    if (p.waitfree) break;
    core_tiles = (N + kSortThreads * it - 1) / (kSortThreads * it);
    core_groups = (core_tiles + kPrefixGroup - 1) / kPrefixGroup;
    ranges = p.plan.passes > 1 ? 1 : 0;
    for (int i = 1; i < p.plan.passes; ++i) {
      const int nd = 1 << p.plan.bits[i];
      const int db = nd < kRangeDigits ? nd : kRangeDigits;
      if (p.plan.bits[i] > p.plan.bits[0] || core_tiles > (kSortThreads / db) * kRangeTiles) ranges = 0;
    }
    bool fits = true;
    for (int i = 0; i < p.plan.passes; ++i)
      if (core_tiles + prefix_blocks(i) > coresident_limit(pass_kernel(it, p.plan.bits[i]), kSortThreads)) fits = false;
    if (fits) {
      sort_it = it;
      break;
    }
  }
  const int sort_cores = sort_it > 0 ? 1 : 0;
  // Passes that read their offsets (reduce-then-scan): 4096-key tiles, or
  // for the wait-free dedup of a batch of at most kWaitfreeSmallTiles
  // 2048-key tiles (twice the workgroups, each ranking half as many keys:
  // the pass is latency-bound, not bound by its column scan)
  int rts_it = kSortItemsWide;
  if (!sort_cores && p.waitfree &&
      (N + kSortThreads * kSortItemsCore - 1) / (kSortThreads * kSortItemsCore) <= kWaitfreeSmallTiles)
    rts_it = kSortItemsCore;
  const int tile_keys = kSortThreads * (sort_cores ? sort_it : rts_it);
  const int sort_tiles = (N + tile_keys - 1) / tile_keys;
  // int32 ids of one table are the keys: the first pass then reads them and
  // finds each position's bag itself, with no prepare kernel
  const bool first_pass_bags = p.T == 1 && !p.idx64;
  const int uniq_cores =
      !p.waitfree && uniq_tiles <= resident_blocks(reinterpret_cast<const void*>(&k_unique), kUniqThreads);
  uint32_t* keys_built = reinterpret_cast<uint32_t*>(ws + L.keys_built);
  hipError_t e = hipSuccess;

  if (!sort_cores && !first_pass_bags) {
    PrepArgs pa{};
    pa.offsets = p.offsets;
    pa.idx = p.idx;
    pa.idx64 = p.idx64;
    pa.ro = p.ro;
    pa.B = p.B;
    pa.M = p.M;
    // about kPrepPositions positions per block
    const int64_t want = (int64_t)kPrepPositions * p.M / N;
    pa.bags_per_block = (int)(want < 1 ? 1 : (want > kPrepMaxBags ? kPrepMaxBags : want));
    // int32 ids of one table are the keys themselves; otherwise keys are built
    pa.keys_out = (p.T > 1 || p.idx64) ? keys_built : nullptr;
    pa.bag_of = reinterpret_cast<int32_t*>(ws + L.bag_of);
    const int prep_blocks = p.M > 0 ? (p.M + pa.bags_per_block - 1) / pa.bags_per_block : 1;
    hipLaunchKernelGGL(k_prepare, dim3((unsigned)prep_blocks), dim3(kPrepThreads), 0, s, pa);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const uint32_t* kin = (p.T > 1 || p.idx64) ? keys_built : static_cast<const uint32_t*>(p.idx);
  const int32_t* vin = nullptr;
  const int32_t* bin = reinterpret_cast<const int32_t*>(ws + L.bag_of);
  uint32_t* keys_a = reinterpret_cast<uint32_t*>(ws + L.keys_a);
  uint32_t* keys_b = reinterpret_cast<uint32_t*>(ws + L.keys_b);
  int32_t* vals_a = reinterpret_cast<int32_t*>(ws + L.vals_a);
  int32_t* vals_b = reinterpret_cast<int32_t*>(ws + L.vals_b);
  int32_t* bags_a = reinterpret_cast<int32_t*>(ws + L.bags_a);
  int32_t* bags_b = reinterpret_cast<int32_t*>(ws + L.bags_b);
  for (int ps = 0; ps < p.plan.passes; ++ps) {
    const bool last = ps == p.plan.passes - 1;
    PassArgs xa{};
    xa.keys_in = kin;
    xa.vals_in = vin;
    xa.bags_in = bin;
    xa.keys_out = last ? reinterpret_cast<uint32_t*>(ws + L.sorted_keys) : ((ps % 2 == 0) ? keys_a : keys_b);
    xa.vals_out = last ? p.sort_perm : ((ps % 2 == 0) ? vals_a : vals_b);
    xa.bags_out = last ? reinterpret_cast<int32_t*>(ws + L.sorted_bag) : ((ps % 2 == 0) ? bags_a : bags_b);
    xa.totals = reinterpret_cast<uint32_t*>(ws + L.totals) + ps * kMaxDigits;
    xa.prev_totals = ps > 0 ? reinterpret_cast<uint32_t*>(ws + L.totals) + (ps - 1) * kMaxDigits : nullptr;
    xa.status = reinterpret_cast<uint64_t*>(back + L.pass_status);
    xa.rows = reinterpret_cast<uint64_t*>(back + L.rows);
    xa.grp = reinterpret_cast<uint64_t*>(back + L.grp);
    xa.coresident = sort_cores;
    xa.xcd_order = !sort_cores && sort_tiles > kXcdOrderMinTiles;
    xa.prefix_mode = (sort_cores && ranges && ps > 0) ? kPrefixRanges : kPrefixGroups;
    xa.later = (sort_cores && ranges && ps == 0) ? reinterpret_cast<uint64_t*>(back + L.later) : nullptr;
    xa.totals_all = reinterpret_cast<uint32_t*>(ws + L.totals);
    xa.npass = p.plan.passes;
    for (int i = 0; i < kMaxPasses; ++i) {
      xa.pass_shift[i] = p.plan.shift[i];
      xa.pass_bits[i] = p.plan.bits[i];
    }
    xa.search_bags = ps == 0 && (sort_cores || first_pass_bags);
    xa.offsets = p.offsets;
    xa.idx = p.idx;
    xa.idx64 = p.idx64;
    xa.ro = p.ro;
    xa.B = p.B;
    xa.M = p.M;
    xa.T = p.T;
    xa.uniq_status = reinterpret_cast<uint64_t*>(ws + L.uniq_status);
    xa.uniq_tiles = uniq_tiles;
    xa.hdr = hdr;
    xa.N = N;
    xa.ntiles = sort_tiles;
    xa.shift = p.plan.shift[ps];
    xa.bits = p.plan.bits[ps];
    xa.pass = ps;
    xa.status_stride = status_stride;
    if (!sort_cores) {
      // reduce-then-scan: the tiles' digit counts, then their prefixes over
      // the tiles and the digit totals
      uint32_t* counts = reinterpret_cast<uint32_t*>(ws + L.tile_counts);
      CountArgs ca{};
      ca.keys = kin;
      ca.N = N;
      ca.shift = xa.shift;
      ca.bits = xa.bits;
      ca.stride = status_stride;
      ca.counts = counts;
      if (rts_it == kSortItemsCore)
        hipLaunchKernelGGL(k_tile_counts<kSortItemsCore>, dim3((unsigned)sort_tiles), dim3(kSortThreads), 0, s, ca);
      else
        hipLaunchKernelGGL(k_tile_counts<kSortItemsWide>, dim3((unsigned)sort_tiles), dim3(kSortThreads), 0, s, ca);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      ColScanArgs sa{};
      sa.counts = counts;
      sa.totals = xa.totals;
      sa.tiles = sort_tiles;
      sa.nd = 1 << xa.bits;
      sa.stride = status_stride;
      hipLaunchKernelGGL(k_column_scan, dim3((unsigned)((sa.nd + kColDigits - 1) / kColDigits)),
                         dim3(kColDigits * kColChunks), 0, s, sa);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      xa.prefix = counts;
    }
    const int extra = sort_cores ? prefix_blocks(ps) : 0;
    switch (sort_cores ? sort_it : rts_it) {
      case kSortItemsCore: e = launch_pass_bits<kSortItemsCore>(xa, sort_tiles + extra, s); break;
      case kSortItemsMid: e = launch_pass_bits<kSortItemsMid>(xa, sort_tiles + extra, s); break;
      default: e = launch_pass_bits<kSortItemsWide>(xa, sort_tiles + extra, s);
    }
    if (e != hipSuccess) return e;
    kin = xa.keys_out;
    vin = xa.vals_out;
    bin = xa.bags_out;
  }

  UniqArgs ua{};
  ua.skeys = kin;
  ua.N = N;
  ua.ntiles = uniq_tiles;
  ua.nchunks = nchunks;
  ua.ukeys = p.unique_keys;
  ua.counts = p.counts;
  ua.seg = p.seg_offsets;
  ua.num_unique = p.num_unique;
  ua.chunk_seg = reinterpret_cast<int32_t*>(ws + L.chunk_seg);
  ua.status = reinterpret_cast<uint64_t*>(ws + L.uniq_status);
  ua.prev_totals = reinterpret_cast<uint32_t*>(ws + L.totals) + (p.plan.passes - 1) * kMaxDigits;
  ua.key_mask = 0xffffffffu;
  if (!uniq_cores) {
    // reduce-then-scan: tile head counts, then their scan over the tiles
    UniqCountArgs uc{};
    uc.skeys = kin;
    uc.N = N;
    uc.out = ua.status;
    hipLaunchKernelGGL(k_uniq_counts, dim3((unsigned)uniq_tiles), dim3(kUniqThreads), 0, s, uc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_uniq_scan, dim3(1), dim3(kUniqScanThreads), 0, s, ua.status, uniq_tiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    ua.prefix = ua.status;
  }
  ua.hdr = hdr;
  hipLaunchKernelGGL(k_unique, dim3((unsigned)uniq_tiles), dim3(kUniqThreads), 0, s, ua);
  return hipGetLastError();
}

}  // namespace emb

// ------------------------------------------------------------ group dedup
//
// The batches of a group are sorted as one: every key carries its batch's
// index above the key bits, so the sorted keys hold batch 0's keys first,
// then batch 1's, and within each batch exactly the stable order of its own
// sort.  Each batch's share (its positions [P_i, P_i + N_i) of the sorted
// order) is then split off into its own permutation and bag ids, and its
// unique scan runs on its share alone, into its own outputs and workspace.
// No workgroup of any of these kernels waits for another.

namespace emb {

namespace {

// the member a block belongs to: the last i with first[i] <= blk
__device__ __forceinline__ int group_member(const int32_t* first, int n, int blk) {
  int i = 0;
  while (i + 1 < n && first[i + 1] <= blk) ++i;
  return i;
}

struct PrepView {  // one batch's prepare arguments, in the form prepare_block reads
  const int32_t* offsets;
  const void* idx;
  int32_t idx64;
  const TableOffsets& ro;
  int32_t B, M, bags_per_block;
  uint32_t* keys_out;
  int32_t* bag_of;
  uint32_t key_hi;
};

struct PrepMember {
  const int32_t* offsets;
  const void* idx;
  int64_t P;
  int32_t idx64, B, M, bags_per_block;
};

struct PrepGroupArgs {
  int32_t n, key_bits;
  int32_t first[kMaxGroup + 1];  // first block of each member; first[n] = grid
  PrepMember b[kMaxGroup];
  uint32_t* keys_out;            // the group's keys, all members' positions
  int32_t* bag_of;               // the group's bag ids (each member's own bag numbers)
  TableOffsets ro;
};

__global__ __launch_bounds__(kPrepThreads) void k_prepare_group(PrepGroupArgs a) {
  __shared__ int32_t s_off[kPrepMaxBags + 1];
  const int i = group_member(a.first, a.n, (int)blockIdx.x);
  const PrepMember& m = a.b[i];
  const PrepView v{m.offsets, m.idx, m.idx64, a.ro, m.B, m.M, m.bags_per_block, a.keys_out + m.P, a.bag_of + m.P,
                   i == 0 ? 0u : (uint32_t)i << a.key_bits};
  prepare_block(v, (int)blockIdx.x - a.first[i], s_off);
}

struct UniqMember {
  int64_t P;
  int32_t N, ntiles, nchunks;
  uint32_t* unique_keys;
  int32_t* counts;
  int32_t* seg_offsets;
  int32_t* num_unique;
  int32_t* chunk_seg;
  uint64_t* words;
  uint32_t* totals;
  WsHeader* hdr;
};

struct UniqGroupArgs {
  int32_t n;
  uint32_t key_mask;
  int32_t first[kMaxGroup + 1];  // first unique tile block of each member
  UniqMember b[kMaxGroup];
  const uint32_t* skeys;         // the group's sorted keys
  WsHeader* ghdr;                // the group call's header
  int32_t sorted;                // the group's passes ran
};

__global__ __launch_bounds__(kUniqThreads) void k_uniq_counts_group(UniqGroupArgs a) {
  __shared__ uint32_t s_c[kUniqThreads / kWave], s_q[kUniqThreads / kWave];
  const int i = group_member(a.first, a.n, (int)blockIdx.x);
  const UniqMember& m = a.b[i];
  const UniqCountArgs c{a.skeys + m.P, m.N, m.words};
  uniq_counts_tile(c, (int)blockIdx.x - a.first[i], s_c, s_q);
}

// One block per member: its call generation (the group sort's error bits
// become its own, so that its unique scan and gradient reduce see them; an
// empty member's outputs instead), then its unique counts' scan.  Block 0
// also makes the group call's generation the group header's (the call is
// complete: no later kernel of it reads the group header).
__global__ __launch_bounds__(kUniqScanThreads) void k_uniq_scan_group(UniqGroupArgs a) {
  __shared__ uint32_t s_c[kUniqScanThreads / kWave], s_q[kUniqScanThreads / kWave];
  const UniqMember& m = a.b[blockIdx.x];
  if (threadIdx.x == 0) {
    if (m.N == 0) {
      m.num_unique[0] = 0;
      m.seg_offsets[0] = 0;
    } else {
      const uint32_t g = next_gen(m.hdr->gen);
      m.hdr->cur = g;
      const uint32_t bits = call_errors(a.ghdr, a.ghdr->cur) & kDedupErrors;
      if (bits) flag_error(m.hdr, g, bits);
    }
    if (blockIdx.x == 0 && a.sorted) a.ghdr->gen = a.ghdr->cur;
  }
  if (m.N > 0) uniq_scan_block(m.words, m.ntiles, s_c, s_q);
}

__global__ __launch_bounds__(kUniqThreads) void k_unique_group(UniqGroupArgs a) {
  const int i = group_member(a.first, a.n, (int)blockIdx.x);
  const UniqMember& m = a.b[i];
  UniqArgs u{};
  u.skeys = a.skeys + m.P;
  u.N = m.N;
  u.ntiles = m.ntiles;
  u.nchunks = m.nchunks;
  u.ukeys = m.unique_keys;
  u.counts = m.counts;
  u.seg = m.seg_offsets;
  u.num_unique = m.num_unique;
  u.chunk_seg = m.chunk_seg;
  u.status = m.words;
  u.prev_totals = m.totals;
  u.prefix = m.words;
  u.hdr = m.hdr;
  u.key_mask = a.key_mask;
  unique_tile(u, (int)blockIdx.x - a.first[i]);
}

}  // namespace

hipError_t launch_dedup_group(const GroupDedupLaunch& p, hipStream_t s) {
  char* ws = static_cast<char*>(p.ws);
  const WsLayout& L = p.lay;
  char* back = ws_back(p.ws, p.ws_bytes, L);
  WsHeader* ghdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  const int n = p.n;
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  uint32_t* keys_built = reinterpret_cast<uint32_t*>(ws + L.keys_built);
  int32_t* bag_of = reinterpret_cast<int32_t*>(ws + L.bag_of);
  uint32_t* sorted_keys = reinterpret_cast<uint32_t*>(ws + L.sorted_keys);
  int32_t* group_perm = reinterpret_cast<int32_t*>(ws + L.group_perm);
  int32_t* sorted_bag = reinterpret_cast<int32_t*>(ws + L.sorted_bag);

  if (p.N > 0) {
    const int N = (int)p.N;
    // keys (with the member index above the key bits) and bag ids of all positions
    PrepGroupArgs pa{};
    pa.n = n;
    pa.key_bits = p.key_bits;
    pa.keys_out = keys_built;
    pa.bag_of = bag_of;
    pa.ro = p.ro;
    int blocks = 0;
    for (int i = 0; i < n; ++i) {
      const GroupMember& m = p.m[i];
      pa.first[i] = blocks;
      pa.b[i] = PrepMember{m.offsets, m.idx, m.P, m.idx64, m.B, m.M, m.bags_per_block};
      if (m.N > 0 && m.M > 0) blocks += (m.M + m.bags_per_block - 1) / m.bags_per_block;
    }
    pa.first[n] = blocks;
    if (blocks > 0) {
      hipLaunchKernelGGL(k_prepare_group, dim3((unsigned)blocks), dim3(kPrepThreads), 0, s, pa);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }

    // the radix passes over all positions: reduce-then-scan, tile offsets
    // computed before each pass (no workgroup waits for another)
    const int it = (N + kSortThreads * kSortItemsCore - 1) / (kSortThreads * kSortItemsCore) <= kWaitfreeSmallTiles
                       ? kSortItemsCore
                       : kSortItemsWide;
    const int tile_keys = kSortThreads * it;
    const int sort_tiles = (N + tile_keys - 1) / tile_keys;
    int max_bits = 1;
    for (int i = 0; i < p.plan.passes; ++i) max_bits = p.plan.bits[i] > max_bits ? p.plan.bits[i] : max_bits;
    const int status_stride = 1 << max_bits;
    const uint32_t* kin = keys_built;
    const int32_t* vin = nullptr;
    const int32_t* bin = bag_of;
    uint32_t* keys_a = reinterpret_cast<uint32_t*>(ws + L.keys_a);
    uint32_t* keys_b = reinterpret_cast<uint32_t*>(ws + L.keys_b);
    int32_t* vals_a = reinterpret_cast<int32_t*>(ws + L.vals_a);
    int32_t* vals_b = reinterpret_cast<int32_t*>(ws + L.vals_b);
    int32_t* bags_a = reinterpret_cast<int32_t*>(ws + L.bags_a);
    int32_t* bags_b = reinterpret_cast<int32_t*>(ws + L.bags_b);
    uint32_t* counts = reinterpret_cast<uint32_t*>(ws + L.tile_counts);
    for (int ps = 0; ps < p.plan.passes; ++ps) {
      const bool last = ps == p.plan.passes - 1;
      PassArgs xa{};
      xa.keys_in = kin;
      xa.vals_in = vin;
      xa.bags_in = bin;
      xa.keys_out = last ? sorted_keys : ((ps % 2 == 0) ? keys_a : keys_b);
      xa.vals_out = last ? group_perm : ((ps % 2 == 0) ? vals_a : vals_b);
      xa.bags_out = last ? sorted_bag : ((ps % 2 == 0) ? bags_a : bags_b);
      xa.totals = reinterpret_cast<uint32_t*>(ws + L.totals) + ps * kMaxDigits;
      xa.prev_totals = ps > 0 ? reinterpret_cast<uint32_t*>(ws + L.totals) + (ps - 1) * kMaxDigits : nullptr;
      xa.status = reinterpret_cast<uint64_t*>(back + L.pass_status);
      xa.rows = reinterpret_cast<uint64_t*>(back + L.rows);
      xa.grp = reinterpret_cast<uint64_t*>(back + L.grp);
      xa.coresident = 0;
      xa.xcd_order = sort_tiles > kXcdOrderMinTiles;
      xa.prefix_mode = kPrefixGroups;
      xa.later = nullptr;
      xa.totals_all = reinterpret_cast<uint32_t*>(ws + L.totals);
      xa.npass = p.plan.passes;
      for (int i = 0; i < kMaxPasses; ++i) {
        xa.pass_shift[i] = p.plan.shift[i];
        xa.pass_bits[i] = p.plan.bits[i];
      }
      xa.search_bags = 0;
      xa.T = p.T;
      xa.uniq_status = reinterpret_cast<uint64_t*>(ws + L.uniq_status);
      xa.uniq_tiles = 0;  // the members' unique scans use their own words
      xa.hdr = ghdr;
      xa.N = N;
      xa.ntiles = sort_tiles;
      xa.shift = p.plan.shift[ps];
      xa.bits = p.plan.bits[ps];
      xa.pass = ps;
      xa.status_stride = status_stride;
      if (last) {
        // each member's values and bags straight to its own buffers
        xa.split_n = n;
        xa.split_bits = p.key_bits;
        for (int i = 0; i < n; ++i) {
          xa.split_P[i] = (int32_t)p.m[i].P;
          xa.split_N[i] = p.m[i].N;
          xa.split_perm[i] = p.m[i].sort_perm;
          xa.split_bag[i] = p.m[i].sorted_bag;
        }
      }
      CountArgs ca{};
      ca.keys = kin;
      ca.N = N;
      ca.shift = xa.shift;
      ca.bits = xa.bits;
      ca.stride = status_stride;
      ca.counts = counts;
      if (it == kSortItemsCore)
        hipLaunchKernelGGL(k_tile_counts<kSortItemsCore>, dim3((unsigned)sort_tiles), dim3(kSortThreads), 0, s, ca);
      else
        hipLaunchKernelGGL(k_tile_counts<kSortItemsWide>, dim3((unsigned)sort_tiles), dim3(kSortThreads), 0, s, ca);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      ColScanArgs sa{};
      sa.counts = counts;
      sa.totals = xa.totals;
      sa.tiles = sort_tiles;
      sa.nd = 1 << xa.bits;
      sa.stride = status_stride;
      hipLaunchKernelGGL(k_column_scan, dim3((unsigned)((sa.nd + kColDigits - 1) / kColDigits)),
                         dim3(kColDigits * kColChunks), 0, s, sa);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      xa.prefix = counts;
      e = it == kSortItemsCore ? launch_pass_bits<kSortItemsCore>(xa, sort_tiles, s)
                               : launch_pass_bits<kSortItemsWide>(xa, sort_tiles, s);
      if (e != hipSuccess) return e;
      kin = xa.keys_out;
      vin = xa.vals_out;
      bin = xa.bags_out;
    }
  }

  // each member's unique scan on its share
  UniqGroupArgs ua{};
  ua.n = n;
  ua.key_mask = p.key_bits >= 32 ? 0xffffffffu : ((1u << p.key_bits) - 1u);
  ua.skeys = sorted_keys;
  int tiles = 0;
  for (int i = 0; i < n; ++i) {
    const GroupMember& m = p.m[i];
    ua.first[i] = tiles;
    const int nt = (m.N + kUniqTile - 1) / kUniqTile;
    ua.b[i] = UniqMember{m.P, m.N, nt, (m.N + kChunk - 1) / kChunk, m.unique_keys, m.counts, m.seg_offsets,
                         m.num_unique, m.chunk_seg, m.uniq_words, m.totals, m.hdr};
    tiles += nt;
  }
  ua.first[n] = tiles;
  ua.ghdr = ghdr;
  ua.sorted = p.N > 0 ? 1 : 0;
  if (tiles > 0) {
    hipLaunchKernelGGL(k_uniq_counts_group, dim3((unsigned)tiles), dim3(kUniqThreads), 0, s, ua);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // every member's call generation (and an empty member's outputs), then
  // the scan of the unique counts
  hipLaunchKernelGGL(k_uniq_scan_group, dim3((unsigned)n), dim3(kUniqScanThreads), 0, s, ua);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k_unique_group, dim3((unsigned)tiles), dim3(kUniqThreads), 0, s, ua);
  return hipGetLastError();
}

}  // namespace emb
