// Device-side fill of a table's initial values with the same counter-based
// draw as the host generator (splitmix64 chain, top 24 bits -> fp32 grid),
// so a multi-gigabyte table is produced in HBM without a host copy.  The
// host generator regenerates any row bit-identically for checking.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9e3779b97f4a7c15ULL;

__device__ __forceinline__ uint64_t sm64(uint64_t x) {
  uint64_t z = x + kGolden;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

uint64_t sm64_host(uint64_t x) {
  uint64_t z = x + kGolden;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

// stream key of the weight quantity (tag 4, coordinates 0, 0)
uint64_t weight_stream(uint64_t seed) {
  return sm64_host(sm64_host(sm64_host(seed ^ (4ULL << 48)) ^ 0ULL) ^ 0ULL);
}

__device__ __forceinline__ float weight_value(uint64_t stream, uint64_t e) {
  const float step = (float)(0.01 / 8388608.0);
  uint64_t h = sm64(stream ^ sm64(e));
  int32_t q = (int32_t)(h >> 40) - 8388608;
  return (float)q * step;
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// element e = r*D + d of the stacked table, elements [e0, e0 + n)
__global__ void fill_f32(float* __restrict__ out, uint64_t stream, uint64_t e0, uint64_t n) {
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) out[i] = weight_value(stream, e0 + i);
}

__global__ void fill_bf16(uint16_t* __restrict__ out, uint64_t stream, uint64_t e0, uint64_t n) {
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) out[i] = bf16_rne(weight_value(stream, e0 + i));
}

__global__ void fill_zero_f32(float* __restrict__ out, uint64_t n) {
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) out[i] = 0.0f;
}

}  // namespace

// Fill rows [0, rows) x D of a device table (dtype 0 fp32, 1 bf16) with the
// initial values of global rows [row0, row0 + rows).  Returns a hipError_t.
extern "C" int synth_dev_fill_weights(void* dev, int32_t dtype, uint64_t seed, uint64_t row0, uint64_t rows,
                                      int32_t D, void* stream) {
  if (dev == nullptr || D <= 0 || (dtype != 0 && dtype != 1)) return (int)hipErrorInvalidValue;
  uint64_t n = rows * (uint64_t)D, e0 = row0 * (uint64_t)D;
  if (n == 0) return 0;
  uint64_t st = weight_stream(seed);
  hipStream_t s = (hipStream_t)stream;
  dim3 grid(4096), block(256);
  if (dtype == 0)
    hipLaunchKernelGGL(fill_f32, grid, block, 0, s, (float*)dev, st, e0, n);
  else
    hipLaunchKernelGGL(fill_bf16, grid, block, 0, s, (uint16_t*)dev, st, e0, n);
  return (int)hipGetLastError();
}

// Zero-fill n floats (optimizer state) without a memset node.
extern "C" int synth_dev_zero_f32(void* dev, uint64_t n, void* stream) {
  if (dev == nullptr) return (int)hipErrorInvalidValue;
  if (n == 0) return 0;
  hipLaunchKernelGGL(fill_zero_f32, dim3(4096), dim3(256), 0, (hipStream_t)stream, (float*)dev, n);
  return (int)hipGetLastError();
}
