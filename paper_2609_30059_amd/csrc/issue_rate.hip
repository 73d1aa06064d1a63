// Issue-rate calibration for the bottleneck-tier classifier (tiers.py):
// SIMD cycles per wave64 instruction of an fp32 FMA, v_exp_f32 and
// v_rcp_f32 on this device.  Every thread runs 8 independent chains of one
// instruction at 8 waves per SIMD, so the SIMDs issue back to back; the
// engine clock is read from the shader clock counter against the 100 MHz
// real-time counter inside the kernel.  Prints one line per instruction.
//
//   ./issue_rate            (built next to the libraries by build.py)
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 1;                                                               \
    }                                                                         \
  } while (0)

namespace {

constexpr int kChains = 8, kUnroll = 4, kBlock = 256;

template <int OP>
__global__ __launch_bounds__(kBlock) void chains(float* sink, int iters, float seed,
                                                  unsigned long long* clocks) {
  float a[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) a[j] = seed + threadIdx.x * 1e-7f + j * 0.01f;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int j = 0; j < kChains; ++j) {
        if constexpr (OP == 0) a[j] = fmaf(a[j], 0.999f, 0.001f);
        else if constexpr (OP == 1) a[j] = __builtin_amdgcn_exp2f(a[j]);
        else a[j] = __builtin_amdgcn_rcpf(a[j]);
      }
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kChains; ++j) s += a[j];
  if (s == 1234.5f) sink[threadIdx.x] = s;     // keeps the chains live
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    clocks[0] = t1 - t0;
    clocks[1] = r1 - r0;
  }
}

template <int OP>
int run(const char* name, float* sink, unsigned long long* clocks, int cus) {
  const int grid = cus * 8, iters = 4000;           // 8 blocks of 4 waves per CU
  hipLaunchKernelGGL(chains<OP>, dim3(grid), dim3(kBlock), 0, 0, sink, 16, 0.5f, clocks);
  CHECK(hipDeviceSynchronize());
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  CHECK(hipEventRecord(e0, 0));
  hipLaunchKernelGGL(chains<OP>, dim3(grid), dim3(kBlock), 0, 0, sink, iters, 0.5f, clocks);
  CHECK(hipEventRecord(e1, 0));
  CHECK(hipEventSynchronize(e1));
  CHECK(hipGetLastError());
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  unsigned long long c[2];
  CHECK(hipMemcpy(c, clocks, sizeof(c), hipMemcpyDeviceToHost));
  const double hz = double(c[0]) / (double(c[1]) / 100e6);
  const double wave_insts = double(grid) * (kBlock / 64) * iters * kUnroll * kChains;
  const double simds = 4.0 * cus;
  const double cycles = ms * 1e-3 * hz * simds / wave_insts;
  std::printf("%-9s %8.3f ms  engine clock %5.0f MHz  %.2f SIMD cycles per wave64 instruction\n",
              name, ms, hz / 1e6, cycles);
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return 0;
}

}  // namespace

int main() {
  int dev = 0, cus = 0;
  CHECK(hipGetDevice(&dev));
  CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  float* sink = nullptr;
  unsigned long long* clocks = nullptr;
  CHECK(hipMalloc(&sink, kBlock * sizeof(float)));
  CHECK(hipMalloc(&clocks, 2 * sizeof(unsigned long long)));
  std::printf("compute units: %d\n", cus);
  if (run<0>("v_fma_f32", sink, clocks, cus)) return 1;
  if (run<1>("v_exp_f32", sink, clocks, cus)) return 1;
  if (run<2>("v_rcp_f32", sink, clocks, cus)) return 1;
  CHECK(hipFree(sink));
  CHECK(hipFree(clocks));
  return 0;
}
