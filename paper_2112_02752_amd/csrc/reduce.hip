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
};

struct RArgs {
  const float* G;
  const int32_t* perm;
  const int32_t* seg;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  const int32_t* bag_of;
  const int32_t* offsets;
  const int32_t* chunk_seg;
  float* grad_rows;
  float* partials;
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

// Write g_u (if grad_rows) and apply the optimizer to row r (if fused).
// Called by the G lanes of one group, all active.
template <typename TW, int G, int NV>
__device__ __forceinline__ void finalize(const Upd& up, float* grad_rows, int64_t u, uint32_t r,
                                         const float (&acc)[NV][4], int sub) {
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
    const float h = up.state[r] + sq / (float)D;
    if (sub == 0) up.state[r] = h;
    step = up.lr / (sqrtf(h) + up.eps);
  }
  TW* wp = reinterpret_cast<TW*>(up.W) + (size_t)r * (size_t)D;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c0 = (v * G + sub) * 4;
    if (c0 < D) {
      float w[4];
      Row4<TW>::load(wp + c0, w);
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = w[e] - step * acc[v][e];
      Row4<TW>::store(wp + c0, w);
    }
  }
}

__device__ __forceinline__ float bag_scale(const RArgs& a, int bag) {
  return a.pool == EMB_POOL_MEAN ? 1.0f / (float)(a.offsets[bag + 1] - a.offsets[bag]) : 1.0f;
}

// Sum the gradient rows of sorted positions [lo, hi) (hi - lo <= 64) with all
// groups of the wavefront, then reduce the groups.  Result valid in group 0.
template <int G, int NV>
__device__ __forceinline__ void wave_piece_sum(const RArgs& a, int lo, int hi, int g, int sub, int lane,
                                               float (&acc)[NV][4]) {
  constexpr int RPI = kWave / G;
  const int n = hi - lo;
  int mbag = 0;
  float msc = 0.f;
  if (lane < n) {
    mbag = a.bag_of[a.perm[lo + lane]];
    msc = bag_scale(a, mbag);
  }
  zero<G, NV>(acc);
  for (int i0 = 0; i0 < n; i0 += RPI * 4) {
    int bag[4];
    float sc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = i0 + q * RPI + g;
      bag[q] = __shfl(mbag, k & (kWave - 1), kWave);
      sc[q] = __shfl(msc, k & (kWave - 1), kWave);
      if (k >= n) sc[q] = 0.f, bag[q] = -1;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (bag[q] >= 0) add_row<G, NV>(a.G + (size_t)bag[q] * a.D, sc[q], a.D, sub, acc);
  }
#pragma unroll
  for (int o = G; o < kWave; o <<= 1)
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);
}

template <typename TW, int G, int NV>
__global__ __launch_bounds__(256) void k_reduce_main(RArgs a) {
  constexpr int RPI = kWave / G;
  const int lane = threadIdx.x & (kWave - 1), g = lane / G, sub = lane % G;
  const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nwaves = gridDim.x * 4;
  const int U = *a.num_unique;

  // heavy pieces: one wavefront per aligned chunk of sorted positions
  for (int c = wave_id; c < a.nchunks; c += nwaves) {
    const int p0 = c * kChunk, p1 = min(a.N, p0 + kChunk);
    const int u0 = a.chunk_seg[c];
    const int s0 = a.seg[u0], e0 = a.seg[u0 + 1];
    const int cs1 = a.chunk_seg[c + 1];
    const int u1 = (a.seg[cs1] == p1) ? cs1 - 1 : cs1;
    float acc[NV][4];
    if (e0 - s0 > kChunk) {
      wave_piece_sum<G, NV>(a, p0, min(p1, e0), g, sub, lane, acc);
      if (g == 0) {
        float* pp = a.partials + ((size_t)c * 2 + 0) * a.D;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int c0 = (v * G + sub) * 4;
          if (c0 < a.D) Row4<float>::store(pp + c0, acc[v]);
        }
      }
    }
    if (u1 != u0) {
      const int s1 = a.seg[u1], e1 = a.seg[u1 + 1];
      if (e1 - s1 > kChunk) {
        wave_piece_sum<G, NV>(a, s1, p1, g, sub, lane, acc);
        if (g == 0) {
          float* pp = a.partials + ((size_t)c * 2 + 1) * a.D;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const int c0 = (v * G + sub) * 4;
            if (c0 < a.D) Row4<float>::store(pp + c0, acc[v]);
          }
        }
      }
    }
  }

  // light segments: one lane group per segment
  for (int u = wave_id * RPI + g; u < U; u += nwaves * RPI) {
    const int s = a.seg[u], e = a.seg[u + 1];
    if (e - s > kChunk) continue;
    float acc[NV][4];
    zero<G, NV>(acc);
    for (int k0 = s; k0 < e; k0 += G) {
      const int my = k0 + sub;
      int mbag = 0;
      float msc = 0.f;
      if (my < e) {
        mbag = a.bag_of[a.perm[my]];
        msc = bag_scale(a, mbag);
      }
      const int n = min(G, e - k0);
      for (int i = 0; i < n; i += 4) {
        int bag[4];
        float sc[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int src = g * G + ((i + q) % G);
          bag[q] = __shfl(mbag, src, kWave);
          sc[q] = __shfl(msc, src, kWave);
          if (i + q >= n) bag[q] = -1;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (bag[q] >= 0) add_row<G, NV>(a.G + (size_t)bag[q] * a.D, sc[q], a.D, sub, acc);
      }
    }
    finalize<TW, G, NV>(a.up, a.grad_rows, u, a.ukeys[u], acc, sub);
  }
}

// Combine the partials of each heavy segment, in chunk order, by the block
// of the segment's first chunk.
template <typename TW, int G, int NV>
__global__ __launch_bounds__(256) void k_reduce_combine(RArgs a) {
  constexpr int RPI = kWave / G;
  constexpr int NG = 4 * RPI;
  __shared__ float s_red[4][G * NV * 4];
  const int lane = threadIdx.x & (kWave - 1), g = lane / G, sub = lane % G, w = threadIdx.x >> 6;
  for (int c = blockIdx.x; c < a.nchunks; c += gridDim.x) {
    const int p0 = c * kChunk, p1 = min(a.N, p0 + kChunk);
    const int cs1 = a.chunk_seg[c + 1];
    const int u1 = (a.seg[cs1] == p1) ? cs1 - 1 : cs1;
    const int s1 = a.seg[u1], e1 = a.seg[u1 + 1];
    if (s1 < p0 || e1 - s1 <= kChunk) continue;
    const int np = (e1 - 1) / kChunk - c + 1;
    float acc[NV][4];
    zero<G, NV>(acc);
    for (int i0 = w * RPI + g; i0 < np; i0 += NG * 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + q * NG;
        if (i < np) {
          const int slot = (i == 0 && s1 != p0) ? 1 : 0;
          add_row<G, NV>(a.partials + ((size_t)(c + i) * 2 + slot) * a.D, 1.0f, a.D, sub, acc);
        }
      }
    }
#pragma unroll
    for (int o = G; o < kWave; o <<= 1)
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);
    if (g == 0) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) s_red[w][(v * G + sub) * 4 + e] = acc[v][e];
    }
    __syncthreads();
    if (w == 0 && g == 0) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float t = s_red[0][(v * G + sub) * 4 + e];
#pragma unroll
          for (int ww = 1; ww < 4; ++ww) t += s_red[ww][(v * G + sub) * 4 + e];
          acc[v][e] = t;
        }
      finalize<TW, G, NV>(a.up, a.grad_rows, u1, a.ukeys[u1], acc, sub);
    }
    __syncthreads();
  }
}

struct UArgs {
  const float* grad_rows;
  const uint32_t* ukeys;
  const int32_t* num_unique;
  int32_t max_unique;
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
    add_row<G, NV>(a.grad_rows + (size_t)u * a.up.D, 1.0f, a.up.D, sub, acc);
    finalize<TW, G, NV>(a.up, nullptr, u, a.ukeys[u], acc, sub);
  }
}

template <typename TW, int G, int NV>
hipError_t launch_reduce_t(const RArgs& ra, int blocks_main, int blocks_comb, hipStream_t s) {
  hipLaunchKernelGGL((k_reduce_main<TW, G, NV>), dim3((unsigned)blocks_main), dim3(256), 0, s, ra);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_reduce_combine<TW, G, NV>), dim3((unsigned)blocks_comb), dim3(256), 0, s, ra);
  return hipGetLastError();
}

template <typename TW>
hipError_t launch_reduce_dt(const RArgs& ra, int bm, int bc, hipStream_t s) {
  const int vecs = (ra.D + 3) / 4;
  if (vecs <= 1) return launch_reduce_t<TW, 1, 1>(ra, bm, bc, s);
  if (vecs <= 2) return launch_reduce_t<TW, 2, 1>(ra, bm, bc, s);
  if (vecs <= 4) return launch_reduce_t<TW, 4, 1>(ra, bm, bc, s);
  if (vecs <= 8) return launch_reduce_t<TW, 8, 1>(ra, bm, bc, s);
  if (vecs <= 16) return launch_reduce_t<TW, 16, 1>(ra, bm, bc, s);
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

template <typename TW>
hipError_t launch_update_dt(const UArgs& ua, int blocks, hipStream_t s) {
  const int vecs = (ua.up.D + 3) / 4;
  if (vecs <= 1) return launch_update_t<TW, 1, 1>(ua, blocks, s);
  if (vecs <= 2) return launch_update_t<TW, 2, 1>(ua, blocks, s);
  if (vecs <= 4) return launch_update_t<TW, 4, 1>(ua, blocks, s);
  if (vecs <= 8) return launch_update_t<TW, 8, 1>(ua, blocks, s);
  if (vecs <= 16) return launch_update_t<TW, 16, 1>(ua, blocks, s);
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
  ra.perm = p.perm;
  ra.seg = p.seg;
  ra.ukeys = p.ukeys;
  ra.num_unique = p.num_unique;
  ra.bag_of = reinterpret_cast<const int32_t*>(ws + p.lay.bag_of);
  ra.offsets = p.offsets;
  ra.chunk_seg = reinterpret_cast<const int32_t*>(ws + p.lay.chunk_seg);
  ra.grad_rows = p.grad_rows;
  ra.partials = reinterpret_cast<float*>(ws + p.lay.partials);
  ra.N = p.N;
  ra.D = p.D;
  ra.pool = p.pool;
  ra.nchunks = (p.N + kChunk - 1) / kChunk;
  ra.up.W = p.W;
  ra.up.state = p.state;
  ra.up.D = p.D;
  ra.up.opt = p.opt;
  ra.up.fuse = p.fuse;
  ra.up.lr = p.lr;
  ra.up.eps = p.eps;
  // main: enough wavefronts to give every lane group a few segments
  const int groups_per_block = 4 * (64 / (((p.D + 3) / 4) >= 64 ? 64 : 1));
  (void)groups_per_block;
  const int bm = clamp_blocks(((int64_t)p.N + 63) / 64, 1, 2048);
  const int bc = clamp_blocks(ra.nchunks, 1, 1024);
  return p.dtype == EMB_FP32 ? launch_reduce_dt<float>(ra, bm, bc, s) : launch_reduce_dt<uint16_t>(ra, bm, bc, s);
}

hipError_t launch_sparse_update(const UpdateLaunch& p, hipStream_t s) {
  if (p.max_unique <= 0) return hipSuccess;
  UArgs ua{};
  ua.grad_rows = p.grad_rows;
  ua.ukeys = p.ukeys;
  ua.num_unique = p.num_unique;
  ua.max_unique = (int32_t)p.max_unique;
  ua.up.W = p.W;
  ua.up.state = p.state;
  ua.up.D = p.D;
  ua.up.opt = p.opt;
  ua.up.fuse = 1;
  ua.up.lr = p.lr;
  ua.up.eps = p.eps;
  const int blocks = clamp_blocks((p.max_unique + 15) / 16, 1, 2048);
  return p.dtype == EMB_FP32 ? launch_update_dt<float>(ua, blocks, s) : launch_update_dt<uint16_t>(ua, blocks, s);
}

}  // namespace emb
