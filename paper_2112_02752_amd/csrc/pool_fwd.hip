// Pooled embedding lookup, forward (gfx950).
//
//   out[m][d] = scale_m * sum_{j in bag m} W[row_offset[t(m)] + idx[j]][d]
//
// One wavefront per bag.  A row of D*sizeof(T) bytes is read as 16-byte
// vectors by a group of G lanes (G a power of two), so one wave instruction
// gathers 64/G rows; each group walks its share of the bag with UNROLL rows
// in flight, accumulating in fp32.  The groups are summed with a butterfly at
// the end and group 0 stores the pooled row.  Ids of the bag are read 64 at a
// time with one coalesced load; repeated ids of such a chunk are merged (one
// row load, added with its multiplicity) and the distinct ids are handed to
// the groups by lane shuffles.
#include "emb_common.h"
#include "kernels.h"

namespace emb {

namespace {

template <typename TW>
struct Vec;  // 16 bytes of table row, widened to fp32

// (loaded raw, widened where it is used, so that every load of a round is
// issued before the first one is waited for)
template <>
struct Vec<float> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static uint4 load(const float* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static void widen(const uint4& v, float (&o)[4]) {
    o[0] = __uint_as_float(v.x);
    o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z);
    o[3] = __uint_as_float(v.w);
  }
};

template <>
struct Vec<uint16_t> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static uint4 load(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static void widen(const uint4& v, float (&o)[8]) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};

constexpr int unroll_for(int rpi) { return rpi == 1 ? 8 : (rpi == 2 ? 8 : (rpi == 4 ? 8 : 4)); }

template <typename TW, int G, int NV, typename TI>
__global__ __launch_bounds__(256) void k_pool_fwd(const TW* __restrict__ W, const int32_t* __restrict__ offsets,
                                                  const TI* __restrict__ idx, TableOffsets ro, int32_t B,
                                                  int32_t M, int32_t D, int32_t pool, float* __restrict__ out) {
  constexpr int RPI = kWave / G;
  constexpr int E = Vec<TW>::kElems;
  constexpr int UN = unroll_for(RPI) / NV > 0 ? unroll_for(RPI) / NV : 1;  // rows in flight per lane group
  const int lane = threadIdx.x & (kWave - 1);
  // the bag is uniform across the wavefront: keep its bookkeeping scalar
  const int m = __builtin_amdgcn_readfirstlane(blockIdx.x * (256 / kWave) + (threadIdx.x >> 6));
  if (m >= M) return;
  const int g = lane / G, sub = lane % G;
  const uint32_t base = ro.off[m / B];
  const int start = offsets[m], end = offsets[m + 1];

  float acc[NV][E];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[v][e] = 0.f;

  for (int j0 = start; j0 < end; j0 += kWave) {
    const int n = min(kWave, end - j0);
    const bool valid = lane < n;
    const int my_id = valid ? (int)idx[j0 + lane] : 0;
    // Skewed ids repeat within a bag: each distinct id of the chunk is loaded
    // once and added with its multiplicity.  Lanes are classed by an 8-bit
    // hash of the id (one ballot per hash bit); a lane whose id equals the
    // lowest lane of its class is a duplicate of it, every other lane (the
    // lowest lane itself, or a hash collision) loads its own row.
    const uint32_t h = ((uint32_t)my_id * 0x9E3779B1u) >> 24;
    uint64_t cls = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (h >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      cls &= bit ? bb : ~bb;
    }
    const int lead = valid ? (int)__builtin_ctzll(cls) : lane;
    // (the shuffle runs on every lane: a lane switched off does not supply its value)
    const int lead_id = __shfl(my_id, lead, kWave);
    const bool dup = valid && lead != lane && lead_id == my_id;
    const uint64_t dups = __ballot(dup);
    const bool loader = valid && !dup;
    const uint64_t lm = __ballot(loader);
    const int nu = (int)__popcll(lm);
    // compact the loaders' (id, multiplicity) into lanes 0..nu-1
    const int dst = loader ? (int)lanes_below(lm) : nu + (int)lanes_below(~lm);
    const int mult = loader ? 1 + (int)__popcll(dups & cls) * (lead == lane) : 0;
    const int c_id = __builtin_amdgcn_ds_permute(dst * 4, my_id);
    const int c_mult = __builtin_amdgcn_ds_permute(dst * 4, mult);
    for (int i0 = 0; i0 < nu; i0 += RPI * UN) {
      // every row load of the round is issued before the first is used (the
      // raw 16 bytes are widened afterwards); unused slots load nothing and
      // are dropped by a select below
      uint4 raw[UN][NV];
      float wt[UN];  // multiplicity; 0 marks an unused slot
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int s = i0 + u * RPI + g;
        const int id = __shfl(c_id, s & (kWave - 1), kWave);
        const int mu = __shfl(c_mult, s & (kWave - 1), kWave);
        wt[u] = s < nu ? (float)mu : 0.f;
        const TW* rp = W + (size_t)(base + (uint32_t)id) * (size_t)D;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int c0 = (v * G + sub) * E;
          raw[u][v] = make_uint4(0u, 0u, 0u, 0u);
          if (s < nu && c0 < D) raw[u][v] = Vec<TW>::load(rp + c0);
        }
      }
      // a row of multiplicity 1 is added exactly as a plain sum would add it
#pragma unroll
      for (int u = 0; u < UN; ++u)
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const bool use = wt[u] != 0.f && (v * G + sub) * E < D;
          float x[E];
          Vec<TW>::widen(raw[u][v], x);
#pragma unroll
          for (int e = 0; e < E; ++e) acc[v][e] = use ? __builtin_fmaf(wt[u], x[e], acc[v][e]) : acc[v][e];
        }
    }
  }

  // sum the RPI groups (butterfly over the group index bits)
#pragma unroll
  for (int o = G; o < kWave; o <<= 1)
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < E; ++e) acc[v][e] += __shfl_xor(acc[v][e], o, kWave);

  if (g == 0) {
    const int L = end - start;
    const float scale = (pool == EMB_POOL_MEAN && L > 0) ? 1.0f / (float)L : 1.0f;
    float* op = out + (size_t)m * (size_t)D;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c0 = (v * G + sub) * E;
      if (c0 < D) {
#pragma unroll
        for (int e = 0; e < E; e += 4) {
          float4 w = make_float4(acc[v][e] * scale, acc[v][e + 1] * scale, acc[v][e + 2] * scale,
                                 acc[v][e + 3] * scale);
          *reinterpret_cast<float4*>(op + c0 + e) = w;
        }
      }
    }
  }
}

template <typename TW, int G, int NV>
hipError_t launch_t(const FwdLaunch& p, hipStream_t s) {
  dim3 grid((unsigned)((p.M + 3) / 4)), block(256);
  // the index type (int32 or int64) is a template argument: no per-load branch
  if (p.idx64)
    hipLaunchKernelGGL((k_pool_fwd<TW, G, NV, int64_t>), grid, block, 0, s, reinterpret_cast<const TW*>(p.W),
                       p.offsets, static_cast<const int64_t*>(p.idx), p.ro, p.B, p.M, p.D, p.pool, p.out);
  else
    hipLaunchKernelGGL((k_pool_fwd<TW, G, NV, int32_t>), grid, block, 0, s, reinterpret_cast<const TW*>(p.W),
                       p.offsets, static_cast<const int32_t*>(p.idx), p.ro, p.B, p.M, p.D, p.pool, p.out);
  return hipGetLastError();
}

template <typename TW>
hipError_t launch_dtype(const FwdLaunch& p, hipStream_t s) {
  const int vecs = p.D * (int)sizeof(TW) / 16;  // 16-byte vectors per row
  if (vecs <= 1) return launch_t<TW, 1, 1>(p, s);
  if (vecs <= 2) return launch_t<TW, 2, 1>(p, s);
  if (vecs <= 4) return launch_t<TW, 4, 1>(p, s);
  if (vecs <= 8) return launch_t<TW, 8, 1>(p, s);
  if (vecs <= 16) return launch_t<TW, 16, 1>(p, s);
  if (vecs <= 32) return launch_t<TW, 32, 1>(p, s);
  if (vecs <= 64) return launch_t<TW, 64, 1>(p, s);
  if (vecs <= 128) return launch_t<TW, 64, 2>(p, s);
  if (vecs <= 256) return launch_t<TW, 64, 4>(p, s);
  if (vecs <= 512) return launch_t<TW, 64, 8>(p, s);
  return hipErrorInvalidValue;
}

}  // namespace

int fwd_max_row_vectors() { return 512; }

hipError_t launch_pool_fwd(const FwdLaunch& p, hipStream_t s) {
  if (p.M == 0) return hipSuccess;
  return p.dtype == EMB_FP32 ? launch_dtype<float>(p, s) : launch_dtype<uint16_t>(p, s);
}

}  // namespace emb
