// Engine-clock probe for the benchmark's clock-transient mode (not a
// sub-kernel; nothing in libfusedsub calls it).  One launch keeps every CU's
// SIMDs issuing fp32 FMAs for a few microseconds and records, for its first
// wave, the shader clock counter and the 100 MHz real-time counter elapsed
// over that work: their ratio is the engine clock at that moment of a
// workload, when the probe is enqueued between the workload's kernels.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kChains = 8, kUnroll = 4, kBlock = 256;

__global__ __launch_bounds__(kBlock) void clock_probe_kernel(unsigned long long* out, int idx,
                                                             int iters) {
  float a[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) a[j] = 0.5f + threadIdx.x * 1e-7f + j * 0.01f;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int j = 0; j < kChains; ++j) a[j] = fmaf(a[j], 0.999f, 0.001f);
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kChains; ++j) s += a[j];
  if (s == 1234.5f) out[2 * idx] = 0;          // keeps the chains live
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    out[2 * idx] = t1 - t0;
    out[2 * idx + 1] = r1 - r0;
  }
}

}  // namespace

// out: device array of 2 * slots counters; idx in [0, slots): the launch
// writes (shader clocks, real-time ticks) of its first wave to out[2 idx],
// out[2 idx + 1].  blocks: grid size (4 waves each); iters: trips of 32 FMAs
// per thread.  Returns 0, or a negative value for arguments out of range
// (nothing launched), or the HIP error of the launch.
extern "C" __attribute__((visibility("default"))) int fsx_clock_probe(
    unsigned long long* out, int idx, int slots, int blocks, int iters, hipStream_t stream) {
  if (!out || idx < 0 || idx >= slots || blocks < 1 || iters < 0) return -1;
  hipLaunchKernelGGL(clock_probe_kernel, dim3(blocks), dim3(kBlock), 0, stream, out, idx, iters);
  return int(hipGetLastError());
}
