// Backward segment-reduce and sparse optimizer step (gfx950).
//
//   g_u = sum over sorted positions k of segment u of scale_{m(k)} * G[m(k)]
//   W_r <- opt(W_r, g_u), r = unique_keys[u]
//
// A row of D fp32 values is held by a group of G lanes (float4 per lane per
// vector, NV vectors), so a wavefront works on 64/G rows at a time.
//  - Light segments (at most kChunk positions, the long tail of a skewed
//    batch): one lane group owns the whole segment, sums its gradient rows
//    and applies the optimizer to its table row.  Each row has exactly one
//    owner, so no atomics are needed.
//  - Heavy segments (the hot ids): their sorted positions are cut at the
//    aligned kChunk boundaries; one wavefront sums each piece into a partial
//    row, and the block that owns the segment's first chunk adds the partials
//    in chunk order and applies the optimizer.
// Every sum runs in a fixed order, so results are bitwise reproducible.
#include "emb_common.h"
#include "kernels.h"

namespace emb {

namespace {

struct Upd {
  void* W;
  float* state;
  int32_t D, opt, fuse;
  float lr, eps;
  int32_t rounding;  // bf16 stores: 0 nearest even, 1 stochastic
  uint64_t seed;
};

struct RArgs {
  const float* G;
  const int32_t* seg;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  const int32_t* sorted_bag;  // bag of every sorted position
  const int32_t* offsets;     // bag offsets (mean pooling scales by 1 / bag length)
  const int32_t* chunk_seg;
  float* grad_rows;
  float* partials;
  uint64_t* level2;     // [ncomb][2][D] tagged rows, cleared by the main kernel
  uint32_t* arrivals;   // [ncomb] arrival counters, cleared by the main kernel
  int32_t ncomb;        // combine blocks
  void* hdr;            // workspace header (error bits)
  int32_t N, D, pool, nchunks;
  Upd up;
};

template <typename TW>
struct Row4;

template <>
struct Row4<float> {
  __device__ __forceinline__ static void load(const float* p, float (&o)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    o[0] = v.x;
    o[1] = v.y;
    o[2] = v.z;
    o[3] = v.w;
  }
  __device__ __forceinline__ static void store(float* p, const float (&o)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(o[0], o[1], o[2], o[3]);
  }
};

template <>
struct Row4<uint16_t> {
  __device__ __forceinline__ static void load(const uint16_t* p, float (&o)[4]) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    o[0] = __uint_as_float(v.x << 16);
    o[1] = __uint_as_float(v.x & 0xffff0000u);
    o[2] = __uint_as_float(v.y << 16);
    o[3] = __uint_as_float(v.y & 0xffff0000u);
  }
  __device__ __forceinline__ static void store(uint16_t* p, const float (&o)[4]) {
    uint2 v;
    v.x = (uint32_t)f32_to_bf16_rne(o[0]) | ((uint32_t)f32_to_bf16_rne(o[1]) << 16);
    v.y = (uint32_t)f32_to_bf16_rne(o[2]) | ((uint32_t)f32_to_bf16_rne(o[3]) << 16);
    *reinterpret_cast<uint2*>(p) = v;
  }
};

// splitmix64 (Steele, Lea and Flood 2014): the output for generator state x
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// Row of four stored values with stochastic rounding to bf16: element e of
// counter c0 + e gets the top 16 bits of splitmix64(seed ^ splitmix64(c)),
// added to the 16 bits below the bf16 mantissa, which are then cut off (the
// magnitude rounds up with probability dropped / 2^16); non-finite values
// round to nearest even.
__device__ __forceinline__ void store_bf16_stochastic(uint16_t* p, const float (&o)[4], uint64_t seed, uint64_t c0) {
  uint16_t b[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t u = __float_as_uint(o[e]);
    const uint32_t r16 = (uint32_t)(splitmix64(seed ^ splitmix64(c0 + (uint64_t)e)) >> 48);
    b[e] = (u & 0x7f800000u) == 0x7f800000u ? f32_to_bf16_rne(o[e]) : (uint16_t)((u + r16) >> 16);
  }
  uint2 v;
  v.x = (uint32_t)b[0] | ((uint32_t)b[1] << 16);
  v.y = (uint32_t)b[2] | ((uint32_t)b[3] << 16);
  *reinterpret_cast<uint2*>(p) = v;
}

template <typename TW>
__device__ __forceinline__ void store_w(const Upd& up, TW* p, const float (&o)[4], uint64_t c0);
template <>
__device__ __forceinline__ void store_w<float>(const Upd&, float* p, const float (&o)[4], uint64_t) {
  Row4<float>::store(p, o);
}
template <>
__device__ __forceinline__ void store_w<uint16_t>(const Upd& up, uint16_t* p, const float (&o)[4], uint64_t c0) {
  if (up.rounding) store_bf16_stochastic(p, o, up.seed, c0);
  else Row4<uint16_t>::store(p, o);
}

template <int G, int NV>
__device__ __forceinline__ void zero(float (&acc)[NV][4]) {
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[v][e] = 0.f;
}

// acc += sc * src[0..D) (this lane's columns)
template <int G, int NV>
__device__ __forceinline__ void add_row(const float* src, float sc, int D, int sub, float (&acc)[NV][4]) {
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c0 = (v * G + sub) * 4;
    if (c0 < D) {
      float x[4];
      Row4<float>::load(src + c0, x);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[v][e] += sc * x[e];
    }
  }
}

// rows of up to 256 floats a lane group keeps in flight (fewer for wider rows)
constexpr int rows_in_flight(int nv) { return nv >= 4 ? 2 : (nv == 2 ? 4 : 8); }

// acc[j] += sc[q][j] * src[idx[q][j]] (this lane's columns) for every (q, j)
// with idx >= 0.  All loads are issued before the first is used, from
// in-bounds addresses (index 0 and column 0 stand in for the unused ones),
// and the unused values are dropped by a select, so no load waits for
// another.
template <int G, int NV, int Q, int S>
__device__ __forceinline__ void add_rows(const float* src, const int (&idx)[Q][S], const float (&sc)[Q][S], int D,
                                         int sub, float (&acc)[S][NV][4]) {
  float x[Q][S][NV][4];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const float* rp = src + (size_t)(idx[q][j] > 0 ? idx[q][j] : 0) * (size_t)D;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c0 = (v * G + sub) * 4;
        Row4<float>::load(rp + (c0 < D ? c0 : 0), x[q][j][v]);
      }
    }
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int j = 0; j < S; ++j)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const bool ok = idx[q][j] >= 0 && (v * G + sub) * 4 < D;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[j][v][e] += ok ? sc[q][j] * x[q][j][v][e] : 0.f;
      }
}

// The table row and optimizer state an update reads, loaded ahead of time.
template <int NV>
struct RowPre {
  float w[NV][4];
  float h;
};

template <typename TW, int G, int NV>
__device__ __forceinline__ void prefetch_row(const Upd& up, uint32_t r, int sub, RowPre<NV>& pre) {
  pre.h = 0.f;
  if (!up.fuse) return;
  if (up.opt == EMB_OPT_ADAGRAD_ROWWISE) pre.h = up.state[r];
  const TW* wp = reinterpret_cast<const TW*>(up.W) + (size_t)r * (size_t)up.D;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c0 = (v * G + sub) * 4;
    if (c0 < up.D) Row4<TW>::load(wp + c0, pre.w[v]);
  }
}

// Write g_u (if grad_rows) and apply the optimizer to row r (if fused) from
// the prefetched row.  Called by the G lanes of one group, all active.
template <typename TW, int G, int NV>
__device__ __forceinline__ void apply_row(const Upd& up, float* grad_rows, int64_t u, uint32_t r,
                                          const float (&acc)[NV][4], const RowPre<NV>& pre, int sub) {
  const int D = up.D;
  if (grad_rows) {
    float* gp = grad_rows + u * D;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c0 = (v * G + sub) * 4;
      if (c0 < D) Row4<float>::store(gp + c0, acc[v]);
    }
  }
  if (!up.fuse) return;
  float step = up.lr;
  if (up.opt == EMB_OPT_ADAGRAD_ROWWISE) {
    float sq = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) sq += acc[v][e] * acc[v][e];
#pragma unroll
    for (int o = 1; o < G; o <<= 1) sq += __shfl_xor(sq, o, kWave);
    const float h = pre.h + sq / (float)D;
    if (sub == 0) up.state[r] = h;
    step = up.lr / (sqrtf(h) + up.eps);
  }
  TW* wp = reinterpret_cast<TW*>(up.W) + (size_t)r * (size_t)D;
  if (up.opt == EMB_OPT_ADAGRAD_ELEMENTWISE) {
    // one accumulator per element, read here (row r has no other owner)
    float* hp = up.state + (size_t)r * (size_t)D;
    float hv[NV][4];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c0 = (v * G + sub) * 4;
      if (c0 < D) Row4<float>::load(hp + c0, hv[v]);
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c0 = (v * G + sub) * 4;
      if (c0 < D) {
        float w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hv[v][e] += acc[v][e] * acc[v][e];
          w[e] = pre.w[v][e] - up.lr * acc[v][e] / (sqrtf(hv[v][e]) + up.eps);
        }
        Row4<float>::store(hp + c0, hv[v]);
        store_w<TW>(up, wp + c0, w, (uint64_t)r * (uint64_t)D + (uint64_t)c0);
      }
    }
    return;
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c0 = (v * G + sub) * 4;
    if (c0 < D) {
      float w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pre.w[v][e] - step * acc[v][e];
      store_w<TW>(up, wp + c0, w, (uint64_t)r * (uint64_t)D + (uint64_t)c0);
    }
  }
}

template <typename TW, int G, int NV>
__device__ __forceinline__ void finalize(const Upd& up, float* grad_rows, int64_t u, uint32_t r,
                                         const float (&acc)[NV][4], int sub) {
  RowPre<NV> pre;
  prefetch_row<TW, G, NV>(up, r, sub, pre);
  apply_row<TW, G, NV>(up, grad_rows, u, r, acc, pre, sub);
}

// whether the dedup this reduce follows flagged an error: its unique scan made
// its generation the header's, so its error bits are those of that generation
__device__ __forceinline__ bool dedup_failed(const RArgs& a) {
  const WsHeader* h = reinterpret_cast<const WsHeader*>(a.hdr);
  return (call_errors(h, h->gen) & kDedupErrors) != 0u;
}

// 1 / bag length for mean pooling (a position's bag is never empty), else 1
__device__ __forceinline__ float bag_scale(const RArgs& a, int bag) {
  return a.pool == EMB_POOL_MEAN ? 1.0f / (float)(a.offsets[bag + 1] - a.offsets[bag]) : 1.0f;
}

// Metadata of one heavy-segment check: the pieces of heavy segments that
// lie in chunk c.  Slot 0: the segment holding the chunk's first position
// (if heavy); slot 1: a different heavy segment holding its last position.
struct ChunkPieces {
  int lo[2], hi[2];
  int u0, s0, e0;  // the segment holding the chunk's first position
  int u1, s1, e1;  // the segment holding the chunk's last position
};

__device__ __forceinline__ ChunkPieces chunk_pieces(const RArgs& a, int c, int U) {
  ChunkPieces r;
  const int p0 = c * kChunk, p1 = min(a.N, p0 + kChunk);
  const int u0 = a.chunk_seg[c], cs1 = a.chunk_seg[c + 1];
  // all needed offsets in one round of independent loads
  const int s0 = a.seg[u0], e0 = a.seg[u0 + 1];
  const int sc = a.seg[cs1];
  const int scm = cs1 > 0 ? a.seg[cs1 - 1] : 0;
  const int scp = cs1 < U ? a.seg[cs1 + 1] : a.N;
  if (sc == p1) {  // position p1 starts segment cs1: the chunk ends with segment cs1 - 1
    r.u1 = cs1 - 1;
    r.s1 = scm;
    r.e1 = sc;
  } else {
    r.u1 = cs1;
    r.s1 = sc;
    r.e1 = scp;
  }
  r.u0 = u0;
  r.s0 = s0;
  r.e0 = e0;
  r.lo[0] = r.hi[0] = r.lo[1] = r.hi[1] = 0;
  if (e0 - s0 > kChunk) {
    r.lo[0] = p0;
    r.hi[0] = min(p1, e0);
  }
  if (r.u1 != u0 && r.e1 - r.s1 > kChunk) {
    r.lo[1] = r.s1;
    r.hi[1] = p1;
  }
  return r;
}

// Sum of the scaled gradient rows of sorted positions [lo, hi) (at most 64)
// by all groups of the wavefront, every row load issued up front; the groups
// are reduced with a butterfly, the result is valid in every group.
// Within a segment the positions of one bag are consecutive (positions
// ascend and so do their bags), so each distinct bag's row is loaded once and
// weighted by its multiplicity: the runs of equal bags are found with a
// ballot and their heads packed to the low lanes with a lane permutation.
template <int G, int NV>
__device__ __forceinline__ void wave_piece_sum(const RArgs& a, int lo, int hi, int g, int sub, int lane,
                                               float (&acc)[NV][4]) {
  constexpr int RPI = kWave / G;
  constexpr int UN = rows_in_flight(NV);
  const int n = hi - lo;
  const int mbag = lane < n ? a.sorted_bag[lo + lane] : -1;
  const int up = __shfl_up(mbag, 1, kWave);
  const bool head = lane < n && (lane == 0 || up != mbag);
  const uint64_t H = __ballot(head);
  const int nh = __popcll(H);
  const uint64_t above = lane == kWave - 1 ? 0ull : (H >> (lane + 1));
  const int next = above ? lane + 1 + __builtin_ctzll(above) : n;
  const float wgt = head ? (float)(next - lane) * bag_scale(a, mbag) : 0.f;
  // heads go to lanes 0..nh-1 in order, the other lanes fill the rest
  const int dst = head ? (int)lanes_below(H) : nh + (int)lanes_below(~H);
  const int cbag = __builtin_amdgcn_ds_permute(dst << 2, mbag);
  const float cw = __int_as_float(__builtin_amdgcn_ds_permute(dst << 2, __float_as_int(wgt)));
  float acc1[1][NV][4];
  zero<G, NV>(acc1[0]);
  for (int i0 = 0; i0 < nh; i0 += RPI * UN) {
    int bag[UN][1];
    float sc[UN][1];
#pragma unroll
    for (int q = 0; q < UN; ++q) {
      const int k = i0 + q * RPI + g;
      bag[q][0] = __shfl(cbag, k & (kWave - 1), kWave);
      sc[q][0] = __shfl(cw, k & (kWave - 1), kWave);
      if (k >= nh) bag[q][0] = -1;
    }
    add_rows<G, NV, UN, 1>(a.G, bag, sc, a.D, sub, acc1);
  }
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[v][e] = acc1[0][v][e];
#pragma unroll
  for (int o = G; o < kWave; o <<= 1)
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);
}

template <int G, int NV>
__device__ __forceinline__ void store_row(float* dst, int D, int sub, const float (&acc)[NV][4]) {
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c0 = (v * G + sub) * 4;
    if (c0 < D) Row4<float>::store(dst + c0, acc[v]);
  }
}

// positions of every light slot whose rows are loaded together
constexpr int light_round(int nv) { return nv >= 4 ? 1 : 2; }
// slots per lane group: one lane of the wavefront reads each segment's offsets
constexpr int slots_for(int rpi) { return rpi * kSlots <= kWave ? kSlots : kWave / rpi; }
// register budget of the main kernel: 5 waves per SIMD for rows of up to 256 floats (no spills)
constexpr int reduce_waves(int nv) { return nv == 1 ? 5 : 4; }

// Light segments, kSlots per lane group: the segments of a batch are
// consecutive; their offsets and keys are read by one lane each, the bags of
// their positions by the group's lanes, then every slot's rows are summed
// with the loads of all slots in flight together.
template <typename TW, int G, int NV>
__device__ __forceinline__ void light_batch(const RArgs& a, int ubase, int U, int g, int sub, int lane) {
  constexpr int RPI = kWave / G;
  constexpr int S = slots_for(RPI);
  constexpr int LR = light_round(NV);
  int ms = 0, me = 0;
  uint32_t mk = 0;
  if (lane < RPI * S && ubase + lane < U) {
    ms = a.seg[ubase + lane];
    me = a.seg[ubase + lane + 1];
    mk = a.ukeys[ubase + lane];
  }
  int s[S], c[S];
  uint32_t r[S];
  int cmax = 0;
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int src = j * RPI + g;
    s[j] = __shfl(ms, src, kWave);
    c[j] = __shfl(me, src, kWave) - s[j];
    r[j] = (uint32_t)__shfl((int)mk, src, kWave);
    if (ubase + src >= U || c[j] > kTinySeg) c[j] = 0;  // absent, medium or heavy
    cmax = max(cmax, c[j]);
  }
  RowPre<NV> pre[S];
#pragma unroll
  for (int j = 0; j < S; ++j)
    if (c[j] > 0) prefetch_row<TW, G, NV>(a.up, r[j], sub, pre[j]);
  float acc[S][NV][4];
#pragma unroll
  for (int j = 0; j < S; ++j) zero<G, NV>(acc[j]);
  for (int i0 = 0; i0 < cmax; i0 += G) {
    int mb[S];
    float msc[S];
#pragma unroll
    for (int j = 0; j < S; ++j) {
      mb[j] = 0;
      msc[j] = 0.f;
      if (i0 + sub < c[j]) {
        mb[j] = a.sorted_bag[s[j] + i0 + sub];
        msc[j] = bag_scale(a, mb[j]);
      }
    }
    const int n = min(G, cmax - i0);
    for (int i = 0; i < n; i += LR) {
      // LR positions of every slot per round, their loads issued together
      int bag[LR][S];
      float sc[LR][S];
#pragma unroll
      for (int q = 0; q < LR; ++q)
#pragma unroll
        for (int j = 0; j < S; ++j) {
          const int src = g * G + ((i + q) & (G - 1));
          bag[q][j] = __shfl(mb[j], src, kWave);
          sc[q][j] = __shfl(msc[j], src, kWave);
          if (i + q >= n || i0 + i + q >= c[j]) bag[q][j] = -1;
        }
      add_rows<G, NV, LR, S>(a.G, bag, sc, a.D, sub, acc);
    }
  }
#pragma unroll
  for (int j = 0; j < S; ++j)
    if (c[j] > 0) apply_row<TW, G, NV>(a.up, a.grad_rows, ubase + j * RPI + g, r[j], acc[j], pre[j], sub);

  // medium segments of the batch (kTinySeg < count <= kChunk): the whole
  // wavefront sums each one with all its rows in flight, group 0 applies it
  const int cnt = me - ms;
  uint64_t medium = __ballot(lane < RPI * S && ubase + lane < U && cnt > kTinySeg && cnt <= kChunk);
  while (medium) {
    const int l = __builtin_ctzll(medium);
    medium &= medium - 1;
    const int lo = __shfl(ms, l, kWave), hi = __shfl(me, l, kWave);
    const uint32_t key = (uint32_t)__shfl((int)mk, l, kWave);
    RowPre<NV> pm;
    if (g == 0) prefetch_row<TW, G, NV>(a.up, key, sub, pm);
    float am[NV][4];
    wave_piece_sum<G, NV>(a, lo, hi, g, sub, lane, am);
    if (g == 0) apply_row<TW, G, NV>(a.up, a.grad_rows, ubase + l, key, am, pm, sub);
  }
}

template <typename TW, int G, int NV>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(reduce_waves(NV), reduce_waves(NV)))) void k_reduce_main(
    RArgs a) {
  constexpr int RPI = kWave / G;
  const int lane = threadIdx.x & (kWave - 1), g = lane / G, sub = lane % G;
  // the wavefront index is uniform: keep the work loops' bookkeeping scalar
  const int wave_id = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int nwaves = gridDim.x * 4;
  const int U = *a.num_unique;
  if (dedup_failed(a)) {
    // The dedup this reduce follows flagged an error: its outputs are
    // undefined, so no table row is written.  Unfused, the gradient rows of
    // the unique ids it reported are zeroed, so that the optimizer step
    // applied to them afterwards leaves every row as it is (for SGD, and for
    // Adagrad with eps > 0).
    if (a.grad_rows) {
      const int64_t n = (int64_t)min(max(U, 0), a.N) * a.D;
      for (int64_t i = (int64_t)wave_id * kWave + lane; i < n; i += (int64_t)nwaves * kWave) a.grad_rows[i] = 0.f;
    }
    return;
  }
  // the combine that follows starts from cleared level-2 rows and counters
  {
    const int nw = a.ncomb * 2 * a.D;
    for (int i = wave_id * kWave + lane; i < nw + a.ncomb; i += nwaves * kWave) {
      if (i < nw) a.level2[i] = 0;
      else a.arrivals[i - nw] = 0u;
    }
  }

  // even wavefronts: the heavy pieces of aligned chunks of sorted positions,
  // one chunk at a time; odd wavefronts: batches of light segments (the two
  // kinds of work interleave on the compute units instead of running one
  // after the other in every wavefront)
  const int half = nwaves / 2;
  const int hw = wave_id >> 1;
  if ((wave_id & 1) == 0) {
    for (int c = hw; c < a.nchunks; c += half) {
      const ChunkPieces cp = chunk_pieces(a, c, U);
#pragma unroll
      for (int slot = 0; slot < 2; ++slot) {
        if (cp.hi[slot] > cp.lo[slot]) {
          float acc[NV][4];
          wave_piece_sum<G, NV>(a, cp.lo[slot], cp.hi[slot], g, sub, lane, acc);
          if (g == 0) store_row<G, NV>(a.partials + ((size_t)c * 2 + slot) * a.D, a.D, sub, acc);
        }
      }
    }
    return;
  }
  // light segments: batches of RPI * slots consecutive segments per wavefront
  const int per_batch = RPI * slots_for(RPI);
  for (int ub = hw * per_batch; ub < U; ub += half * per_batch) light_batch<TW, G, NV>(a, ub, U, g, sub, lane);
}

// Heavy segments.  The block of a range of kCombineChunks chunks lists (one
// lane per chunk) the pieces of heavy segments in its range: the segments
// that start in it and the one that holds its first position, if that one
// started earlier.  One wavefront per piece sums the piece's chunk partials
// in chunk order.  A segment that lies in the range is finished at once; a
// segment that crosses ranges leaves one row per range (slot 1 in the range
// where it starts, slot 0 in the others) as tagged words, and the block
// that arrives last at the segment's counter adds those rows in range order
// and applies the optimizer.  The order of every sum is fixed, so the result
// does not depend on which block arrives last; no block ever waits for
// another to arrive.
constexpr uint32_t kLevel2Tag = 1u;  // rows and counters are cleared by the main kernel

// sum of this lane's columns of level-2 rows [g0, g1) (slot 1 of the first
// range, slot 0 of the others), rows split over the lane groups with the
// words of several rows loaded together; a word is polled until it carries
// the tag (bounded)
template <int G, int NV>
__device__ __forceinline__ void level2_sum(const RArgs& a, int g0, int g1, int g, int sub, WsHeader* h,
                                           float (&acc)[NV][4]) {
  constexpr int RPI = kWave / G;
  constexpr int RR = rows_in_flight(NV) / 2 > 0 ? rows_in_flight(NV) / 2 : 1;
  zero<G, NV>(acc);
  for (int r0 = g0 + g; r0 < g1; r0 += RPI * RR) {
    uint64_t x[RR][NV][4];
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int r = r0 + q * RPI;
      const uint64_t* src = a.level2 + ((size_t)(r < g1 ? r : g0) * 2 + (r == g0 ? 1 : 0)) * a.D;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c0 = (v * G + sub) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[q][v][e] = ld_relaxed_u64(src + (c0 < a.D ? c0 + e : e));
      }
    }
#pragma unroll
    for (int q = 0; q < RR; ++q) {
      const int r = r0 + q * RPI;
      if (r >= g1) continue;
      const uint64_t* src = a.level2 + ((size_t)r * 2 + (r == g0 ? 1 : 0)) * a.D;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c0 = (v * G + sub) * 4;
        if (c0 >= a.D) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t spins = 0;
          const uint64_t t0 = wait_clock();
          while ((uint32_t)(x[q][v][e] >> 32) != kLevel2Tag) {
            if (wait_over(h, h->gen, t0, ++spins)) {
              flag_timeout(h, h->gen, kSiteCombine, kCombineError);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
            x[q][v][e] = ld_relaxed_u64(src + c0 + e);
          }
          acc[v][e] += __uint_as_float((uint32_t)x[q][v][e]);
        }
      }
    }
  }
#pragma unroll
  for (int o = G; o < kWave; o <<= 1)
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);
}

template <typename TW, int G, int NV>
__global__ __launch_bounds__(kCombineThreads) void k_reduce_combine(RArgs a) {
  constexpr int RPI = kWave / G;
  constexpr int NWv = kCombineThreads / kWave;
  constexpr int CU = rows_in_flight(NV);  // chunk partials of a lane group loaded together
  __shared__ int4 s_piece[kCombineChunks + 1];  // (segment, first chunk in range, start, end)
  __shared__ int s_n;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), g = lane / G, sub = lane % G;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform across the wavefront
  const int U = *a.num_unique;
  if (dedup_failed(a)) return;  // as in k_reduce_main
  const int blk = blockIdx.x;
  const int c0 = blk * kCombineChunks, c1 = min(a.nchunks, c0 + kCombineChunks);
  if (tid == 0) s_n = 0;
  __syncthreads();
  if (tid < c1 - c0) {
    const int c = c0 + tid;
    const ChunkPieces cp = chunk_pieces(a, c, U);
    if (cp.e1 - cp.s1 > kChunk && cp.s1 >= c * kChunk) s_piece[atomicAdd(&s_n, 1)] = make_int4(cp.u1, c, cp.s1, cp.e1);
    if (c == c0 && cp.hi[0] > cp.lo[0] && cp.s0 < c * kChunk)
      s_piece[atomicAdd(&s_n, 1)] = make_int4(cp.u0, c, cp.s0, cp.e0);
  }
  __syncthreads();
  const int n = s_n;
  for (int k = w; k < n; k += NWv) {
    const int4 pc = s_piece[k];
    const int u = pc.x, cf = pc.y, st = pc.z, en = pc.w;
    const int cs = st / kChunk, ce = (en - 1) / kChunk;  // chunks of the whole segment
    const int cl = min(c1 - 1, ce);                      // last chunk of this piece
    const int np = cl - cf + 1;
    const uint32_t key = a.ukeys[u];
    RowPre<NV> pre;
    if (g == 0) prefetch_row<TW, G, NV>(a.up, key, sub, pre);
    float acc1[1][NV][4];
    zero<G, NV>(acc1[0]);
    for (int i0 = 0; i0 < np; i0 += RPI * CU) {
      int pidx[CU][1];
      float one[CU][1];
#pragma unroll
      for (int q = 0; q < CU; ++q) {
        const int i = i0 + q * RPI + g;
        const int c = cf + i;
        const int slot = (c == cs && st != c * kChunk) ? 1 : 0;
        pidx[q][0] = i < np ? c * 2 + slot : -1;
        one[q][0] = 1.0f;
      }
      add_rows<G, NV, CU, 1>(a.partials, pidx, one, a.D, sub, acc1);
    }
    float acc[NV][4];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[v][e] = acc1[0][v][e];
#pragma unroll
    for (int o = G; o < kWave; o <<= 1)
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);
    const int bs = cs / kCombineChunks, be = ce / kCombineChunks;  // combine blocks of the segment
    if (bs == be) {
      if (g == 0) apply_row<TW, G, NV>(a.up, a.grad_rows, u, key, acc, pre, sub);
      continue;
    }
    // publish this range's row, then arrive
    uint64_t* dst = a.level2 + ((size_t)blk * 2 + (blk == bs ? 1 : 0)) * a.D;
    if (g == 0) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int c0v = (v * G + sub) * 4;
        if (c0v < a.D)
#pragma unroll
          for (int e = 0; e < 4; ++e) st_u64(dst + c0v + e, ((uint64_t)kLevel2Tag << 32) | __float_as_uint(acc[v][e]));
      }
    }
    uint32_t old = 0;
    if (lane == 0) old = atomic_add_u32(&a.arrivals[bs], 1u);
    old = (uint32_t)__shfl((int)old, 0, kWave);
    if (old == (uint32_t)(be - bs)) {
      WsHeader* h = reinterpret_cast<WsHeader*>(a.hdr);
      level2_sum<G, NV>(a, bs, be + 1, g, sub, h, acc);
      if (g == 0) apply_row<TW, G, NV>(a.up, a.grad_rows, u, key, acc, pre, sub);
    }
  }
}

struct UArgs {
  const float* grad_rows;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  int32_t max_unique;
  uint32_t rows;
  Upd up;
};

template <typename TW, int G, int NV>
__global__ __launch_bounds__(256) void k_sparse_update(UArgs a) {
  constexpr int RPI = kWave / G;
  const int lane = threadIdx.x & (kWave - 1), g = lane / G, sub = lane % G;
  const int gid = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPI + g;
  const int ngroups = gridDim.x * 4 * RPI;
  const int U = min(*a.num_unique, a.max_unique);
  for (int u = gid; u < U; u += ngroups) {
    float acc[NV][4];
    zero<G, NV>(acc);
    const uint32_t key = a.ukeys[u];
    if (key >= a.rows) continue;  // not a row: keys of a failed dedup are never written through
    add_row<G, NV>(a.grad_rows + (size_t)u * a.up.D, 1.0f, a.up.D, sub, acc);
    finalize<TW, G, NV>(a.up, nullptr, u, key, acc, sub);
  }
}

template <typename TW, int G, int NV>
hipError_t launch_reduce_t(const RArgs& ra, int blocks_main, int blocks_comb, hipStream_t s) {
  hipLaunchKernelGGL((k_reduce_main<TW, G, NV>), dim3((unsigned)blocks_main), dim3(256), 0, s, ra);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_reduce_combine<TW, G, NV>), dim3((unsigned)blocks_comb), dim3(kCombineThreads), 0, s, ra);
  return hipGetLastError();
}

// Rows of 33 to 64 values are held two vectors per lane (half as many lanes
// per row, twice as many rows per wavefront): a wavefront then carries twice
// the light segments, which outweighs the lower occupancy (measured on rows
// of 64 fp32 values).  Narrower rows, and wider ones (128 bf16 values lost on
// small batches), keep one vector.
template <typename TW>
hipError_t launch_reduce_dt(const RArgs& ra, int bm, int bc, hipStream_t s) {
  const int vecs = (ra.D + 3) / 4;
  if (vecs <= 1) return launch_reduce_t<TW, 1, 1>(ra, bm, bc, s);
  if (vecs <= 2) return launch_reduce_t<TW, 2, 1>(ra, bm, bc, s);
  if (vecs <= 4) return launch_reduce_t<TW, 4, 1>(ra, bm, bc, s);
  if (vecs <= 8) return launch_reduce_t<TW, 8, 1>(ra, bm, bc, s);
  if (vecs <= 16) return launch_reduce_t<TW, 8, 2>(ra, bm, bc, s);
  if (vecs <= 32) return launch_reduce_t<TW, 32, 1>(ra, bm, bc, s);
  if (vecs <= 64) return launch_reduce_t<TW, 64, 1>(ra, bm, bc, s);
  if (vecs <= 128) return launch_reduce_t<TW, 64, 2>(ra, bm, bc, s);
  if (vecs <= 256) return launch_reduce_t<TW, 64, 4>(ra, bm, bc, s);
  return hipErrorInvalidValue;
}

template <typename TW, int G, int NV>
hipError_t launch_update_t(const UArgs& ua, int blocks, hipStream_t s) {
  hipLaunchKernelGGL((k_sparse_update<TW, G, NV>), dim3((unsigned)blocks), dim3(256), 0, s, ua);
  return hipGetLastError();
}

// the reduce's lane layout for every width, so that the row-wise Adagrad sum
// of squares runs in the same order and the unfused update equals the fused one
template <typename TW>
hipError_t launch_update_dt(const UArgs& ua, int blocks, hipStream_t s) {
  const int vecs = (ua.up.D + 3) / 4;
  if (vecs <= 1) return launch_update_t<TW, 1, 1>(ua, blocks, s);
  if (vecs <= 2) return launch_update_t<TW, 2, 1>(ua, blocks, s);
  if (vecs <= 4) return launch_update_t<TW, 4, 1>(ua, blocks, s);
  if (vecs <= 8) return launch_update_t<TW, 8, 1>(ua, blocks, s);
  if (vecs <= 16) return launch_update_t<TW, 8, 2>(ua, blocks, s);
  if (vecs <= 32) return launch_update_t<TW, 32, 1>(ua, blocks, s);
  if (vecs <= 64) return launch_update_t<TW, 64, 1>(ua, blocks, s);
  if (vecs <= 128) return launch_update_t<TW, 64, 2>(ua, blocks, s);
  if (vecs <= 256) return launch_update_t<TW, 64, 4>(ua, blocks, s);
  return hipErrorInvalidValue;
}

int clamp_blocks(int64_t want, int lo, int hi) {
  if (want < lo) return lo;
  if (want > hi) return hi;
  return (int)want;
}

}  // namespace

int reduce_max_dim() { return 1024; }

hipError_t launch_grad_reduce(const ReduceLaunch& p, hipStream_t s) {
  if (p.N == 0) return hipSuccess;
  char* ws = static_cast<char*>(p.ws);
  RArgs ra{};
  ra.G = p.grad_out;
  ra.seg = p.seg;
  ra.ukeys = p.ukeys;
  ra.num_unique = p.num_unique;
  ra.sorted_bag = reinterpret_cast<const int32_t*>(ws + p.lay.sorted_bag);
  ra.offsets = p.offsets;
  ra.chunk_seg = reinterpret_cast<const int32_t*>(ws + p.lay.chunk_seg);
  ra.grad_rows = p.grad_rows;
  ra.partials = reinterpret_cast<float*>(ws + p.lay.partials);
  ra.level2 = reinterpret_cast<uint64_t*>(ws + p.lay.level2);
  ra.arrivals = reinterpret_cast<uint32_t*>(ws + p.lay.arrivals);
  ra.nchunks = (p.N + kChunk - 1) / kChunk;
  ra.ncomb = (ra.nchunks + kCombineChunks - 1) / kCombineChunks;  // of this batch (the layout is the workspace's)
  ra.hdr = ws + p.lay.hdr;
  ra.N = p.N;
  ra.D = p.D;
  ra.pool = p.pool;
  ra.up.W = p.W;
  ra.up.state = p.state;
  ra.up.D = p.D;
  ra.up.opt = p.opt;
  ra.up.fuse = p.fuse;
  ra.up.lr = p.lr;
  ra.up.eps = p.eps;
  ra.up.rounding = p.rounding;
  ra.up.seed = p.seed;
  // main: two wavefronts per chunk of sorted positions (one for its heavy
  // pieces, one for a batch of light segments), up to two full devices
  const int bm = clamp_blocks(((int64_t)ra.nchunks + 1) / 2, 1, 4096);
  const int bc = clamp_blocks(ra.ncomb, 1, 1 << 20);
  return p.dtype == EMB_FP32 ? launch_reduce_dt<float>(ra, bm, bc, s) : launch_reduce_dt<uint16_t>(ra, bm, bc, s);
}

hipError_t launch_sparse_update(const UpdateLaunch& p, hipStream_t s) {
  if (p.max_unique <= 0) return hipSuccess;
  UArgs ua{};
  ua.grad_rows = p.grad_rows;
  ua.ukeys = p.ukeys;
  ua.num_unique = p.num_unique;
  ua.max_unique = (int32_t)p.max_unique;
  ua.rows = p.rows;
  ua.up.W = p.W;
  ua.up.state = p.state;
  ua.up.D = p.D;
  ua.up.opt = p.opt;
  ua.up.fuse = 1;
  ua.up.lr = p.lr;
  ua.up.eps = p.eps;
  ua.up.rounding = p.rounding;
  ua.up.seed = p.seed;
  const int blocks = clamp_blocks((p.max_unique + 15) / 16, 1, 2048);
  return p.dtype == EMB_FP32 ? launch_update_dt<float>(ua, blocks, s) : launch_update_dt<uint16_t>(ua, blocks, s);
}

}  // namespace emb
