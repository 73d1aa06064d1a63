// LayerNorm fused with the residual add.
//
// h = x + residual; y = (h - mean) / sqrt(var + eps) * gamma + beta;
// residual_out = h -- KernelOPT Appendix A (Fusion Agent: normalisation
// fusion, residual + norm in one memory pass; Codegen prompt: single-pass
// LayerNorm).
//
// Design (gfx950): one row per group of W wave64s, EPT elements per thread
// held in registers: x and residual are read from HBM once, residual_out and
// y written once.  The statistics are exact two-pass values per thread (mean
// of the thread's elements, then the sum of squared deviations from it) and
// one all-reduce merges the (count, mean, M2) triples with the pairwise
// update of Chan, Golub and LeVeque (1979):
//     n = na + nb, mean = (na*ma + nb*mb) / n, M2 = M2a + M2b + (mb-ma)^2 na nb / n
// written so that combine(a, b) and combine(b, a) round identically, so every
// lane ends with the same statistics.  No E[h^2] - mean^2 cancellation.
#include "device_common.hpp"
#include "launch.hpp"

namespace fs {
namespace {

struct MeanM2P {
  float n, mean, m2;
  __device__ __forceinline__ static MeanM2P combine(const MeanM2P& a, const MeanM2P& b) {
    if (a.n == 0.f) return b;
    if (b.n == 0.f) return a;
    const float n = a.n + b.n;
    const float mean = (a.n * a.mean + b.n * b.mean) / n;
    const float d = b.mean - a.mean;
    return {n, mean, (a.m2 + b.m2) + d * d * ((a.n * b.n) / n)};
  }
  template <class F> __device__ __forceinline__ static MeanM2P map(const MeanM2P& a, F f) {
    return {f(a.n), f(a.mean), f(a.m2)};
  }
};

template <typename T, int W, int EPT, bool VEC, int G>
__global__ __launch_bounds__(64 * W * G) void layernorm_kernel(
    const T* __restrict__ x, int64_t ld_x, const T* __restrict__ res, int64_t ld_r,
    const T* __restrict__ gamma, const T* __restrict__ beta, T* y, int64_t ld_y, T* res_out,
    int64_t ld_ro, int64_t rows, int cols, float eps) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  constexpr int NV = EPT / V;
  static_assert(EPT % V == 0, "EPT must be a multiple of the vector width");
  __shared__ MeanM2P lds[2][W];

  const int tid = threadIdx.x % kThreads;
  const int wave = tid / 64, lane = tid % 64;
  const int g = threadIdx.x / kThreads;
  int parity = 0;

  // columns this thread owns and how many are inside the row
  int n_local = 0;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c0 = (k * kThreads + tid) * V;
    n_local += (c0 < cols) ? V : 0;
  }

  for (int64_t row = int64_t(blockIdx.x) * G + g; row < rows; row += int64_t(gridDim.x) * G) {
    const T* xr = x + row * ld_x;
    const T* rr = res ? res + row * ld_r : nullptr;
    float h[EPT];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c0 = (k * kThreads + tid) * V;
      if (c0 < cols) {
        ldv<T, V>(xr + c0, h + k * V);
        if (rr) {
          float rv[V];
          ldv<T, V>(rr + c0, rv);
#pragma unroll
          for (int i = 0; i < V; ++i) h[k * V + i] += rv[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) h[k * V + i] = 0.f;
      }
    }
    if (res_out) {
      T* ro = res_out + row * ld_ro;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = (k * kThreads + tid) * V;
        if (c0 < cols) {
          if constexpr (VEC) st128<true>(ro + c0, Elem<T>::pack(h + k * V));
          else Elem<T>::store1(ro + c0, h[k]);
        }
      }
    }

    // per-thread exact two-pass statistics over the owned columns
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < EPT; ++i) s += h[i];     // out-of-row slots hold 0
    const float nl = float(n_local);
    const float mean_l = n_local ? s / nl : 0.f;
    float m2 = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c0 = (k * kThreads + tid) * V;
      if (c0 < cols) {
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const float d = h[k * V + i] - mean_l;
          m2 = fmaf(d, d, m2);
        }
      }
    }
    const MeanM2P st = group_allreduce<W>(MeanM2P{nl, mean_l, m2}, lds[parity], wave, lane);
    parity ^= 1;
    const float rstd = rsqrtf(st.m2 / st.n + eps);
    const float mean = st.mean;

    T* yr = y + row * ld_y;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c0 = (k * kThreads + tid) * V;
      if (c0 < cols) {
        float gv[V], bv[V];
        if (gamma) ldv<T, V, false>(gamma + c0, gv);
        else {
#pragma unroll
          for (int i = 0; i < V; ++i) gv[i] = 1.f;
        }
        if (beta) ldv<T, V, false>(beta + c0, bv);
        else {
#pragma unroll
          for (int i = 0; i < V; ++i) bv[i] = 0.f;
        }
        float o[V];
#pragma unroll
        for (int i = 0; i < V; ++i) o[i] = fmaf((h[k * V + i] - mean) * rstd, gv[i], bv[i]);
        if constexpr (VEC) st128<true>(yr + c0, Elem<T>::pack(o));
        else Elem<T>::store1(yr + c0, o[0]);
      }
    }
  }
}

template <typename T, bool VEC>
hipError_t dispatch(const LayerNormArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  const int64_t c = a.cols;
  auto launch = [&](auto kern, int threads, int rows_per_block, int blocks_per_cu) {
    int64_t want = (a.rows + rows_per_block - 1) / rows_per_block;
    int64_t cap = int64_t(cus) * blocks_per_cu;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s, static_cast<const T*>(a.x), a.ld_x,
                       static_cast<const T*>(a.res), a.ld_r, static_cast<const T*>(a.gamma),
                       static_cast<const T*>(a.beta), static_cast<T*>(a.y), a.ld_y,
                       static_cast<T*>(a.res_out), a.ld_ro, a.rows, int(a.cols), a.eps);
    return hipGetLastError();
  };
#define FS_LN(Wv, E, Gv, BPC)                                                   \
  if (c <= int64_t(64) * Wv * E)                                                 \
    return launch(layernorm_kernel<T, Wv, E, VEC, Gv>, 64 * Wv * Gv, Gv, BPC);
  if constexpr (V <= 1) { FS_LN(1, 1, 4, 64) }
  if constexpr (V <= 2) { FS_LN(1, 2, 4, 64) }
  if constexpr (V <= 4) { FS_LN(1, 4, 4, 64) }
  FS_LN(1, 8, 4, 64)
  FS_LN(1, 16, 4, 64)
  FS_LN(1, 32, 4, 32)
  FS_LN(1, 64, 4, 16)
  FS_LN(2, 64, 1, 32)
  FS_LN(4, 64, 1, 16)
  FS_LN(8, 64, 1, 8)
  FS_LN(16, 64, 1, 4)
#undef FS_LN
  return hipErrorInvalidValue;   // unreachable: the host checks cols
}

}  // namespace

hipError_t launch_layernorm(const LayerNormArgs& a, int cus, hipStream_t s) {
  if (a.dtype == FS_BF16)
    return a.vec ? dispatch<uint16_t, true>(a, cus, s) : dispatch<uint16_t, false>(a, cus, s);
  return a.vec ? dispatch<float, true>(a, cus, s) : dispatch<float, false>(a, cus, s);
}

}  // namespace fs
