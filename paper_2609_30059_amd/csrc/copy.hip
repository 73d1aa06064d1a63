// Calibration copy: the achievable HBM bandwidth of a plain streaming kernel
// on this device (16-byte loads and stores, grid-stride), and the reference
// against which hardware byte counters are scaled.
#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_COPY_UNROLL
#define FS_COPY_UNROLL 1
#endif
#ifndef FS_COPY_BLOCKS_PER_CU
#define FS_COPY_BLOCKS_PER_CU 64
#endif

namespace fs {
namespace {

__global__ __launch_bounds__(256) void copy128_kernel(const u32x4* __restrict__ src,
                                                       u32x4* __restrict__ dst, int64_t n) {
  constexpr int U = FS_COPY_UNROLL;
  const int64_t stride = int64_t(gridDim.x) * 256;
  int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  for (; i + (U - 1) * stride < n; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = ld128<true>(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) st128<true>(dst + i + u * stride, v[u]);
  }
  for (; i < n; i += stride) st128<true>(dst + i, ld128<true>(src + i));
}

__global__ __launch_bounds__(256) void copy8_kernel(const uint8_t* __restrict__ src,
                                                     uint8_t* __restrict__ dst, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
    dst[i] = src[i];
}

}  // namespace

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int cus, hipStream_t s) {
  const bool vec = (reinterpret_cast<uintptr_t>(src) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(dst) % 16 == 0) && (bytes % 16 == 0);
  const int64_t n = vec ? bytes / 16 : bytes;
  int64_t grid = (n + 255) / 256;
  const int64_t cap = int64_t(cus) * FS_COPY_BLOCKS_PER_CU;
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  if (vec)
    hipLaunchKernelGGL(copy128_kernel, dim3(unsigned(grid)), dim3(256), 0, s,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), n);
  else
    hipLaunchKernelGGL(copy8_kernel, dim3(unsigned(grid)), dim3(256), 0, s,
                       static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), n);
  return hipGetLastError();
}

}  // namespace fs
