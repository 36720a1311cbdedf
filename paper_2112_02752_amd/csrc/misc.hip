// Batch validation, workspace clearing (off the timed path) and the
// residency query used to pick the sort's prefix scheme.
#include <map>
#include <mutex>
#include <utility>

#include "emb_common.h"
#include "kernels.h"

namespace emb {

namespace {

__global__ void k_fill_zero_u32(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// flag bits: 1 offsets[0] != 0, 2 decreasing offsets, 4 offsets[M] != N, 8 id out of range
__global__ void k_validate(const int32_t* offsets, const void* idx, int32_t idx64, TableOffsets ro, int32_t B,
                           int32_t M, int64_t N, int32_t* flag) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t bits = 0;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t0 == 0) {
    if (offsets[0] != 0) bits |= 1u;
    if ((int64_t)offsets[M] != N) bits |= 4u;
  }
  for (int64_t m = t0; m < M; m += stride) {
    const int32_t s = offsets[m], e = offsets[m + 1];
    if (e < s) {
      bits |= 2u;
      continue;
    }
    const int t = (int)(m / B);
    const int64_t rows = (int64_t)ro.off[t + 1] - (int64_t)ro.off[t];
    const int32_t lo = s < 0 ? 0 : s;
    const int64_t hi = (int64_t)e < N ? (int64_t)e : N;
    for (int64_t j = lo; j < hi; ++j) {
      const int64_t id = idx64 ? static_cast<const int64_t*>(idx)[j] : (int64_t) static_cast<const int32_t*>(idx)[j];
      if (id < 0 || id >= rows) bits |= 8u;
    }
  }
  if (bits) atomicOr(reinterpret_cast<uint32_t*>(flag), bits);
}

// status of the last dedup call on a workspace (emb_workspace_status)
__global__ void k_workspace_status(const WsHeader* h, int32_t* status) {
  if (threadIdx.x == 0) {
    status[0] = (int32_t)call_errors(h, h->gen);
    status[1] = (int32_t)h->timeout_site;
    status[2] = (int32_t)h->timeout_block;
    status[3] = (int32_t)h->timeouts;
  }
}

}  // namespace

hipError_t launch_workspace_status(const void* ws, int32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(k_workspace_status, dim3(1), dim3(64), 0, s, static_cast<const WsHeader*>(ws), status);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(void* p, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_zero_u32, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint32_t*>(p), n);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateLaunch& p, hipStream_t s) {
  hipError_t e = launch_zero_bytes(p.flag, 4, s);
  if (e != hipSuccess) return e;
  int64_t blocks = ((int64_t)p.M + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_validate, dim3((unsigned)blocks), dim3(256), 0, s, p.offsets, p.idx, p.idx64, p.ro, p.B, p.M,
                     p.N,
                     p.flag);
  return hipGetLastError();
}

int resident_blocks(const void* kernel, int threads) {
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(mu);
  auto key = std::make_pair(dev, kernel);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) per_cu = 0;
  const int n = cus * per_cu;
  cache[key] = n;
  return n;
}

int coresident_limit(const void* kernel, int threads) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return resident_blocks(kernel, threads) >= cus ? cus : 0;
}

}  // namespace emb
