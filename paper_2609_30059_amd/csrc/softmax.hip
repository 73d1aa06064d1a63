// Fused row softmax with pre-scale, additive mask and causal masking.
//
// y[r, :] = softmax(x[r, :] * scale + mask[r, :]) -- KernelOPT Appendix A
// (Planner item 9, fused softmax; Codegen prompt, online softmax).
//
// Design (gfx950): one row per group of W wave64s; each thread holds EPT
// elements of the row in registers, so HBM is read once and written once.
// Per thread the logits are turned into base-2 exponents
// a = (x * scale + mask) * log2(e), the local max m and the local sum d of
// exp2(a - m) are formed with the exponentials kept in registers, and a
// single all-reduce combines the (m, d) pairs:
//     (m1, d1) + (m2, d2) = (M, d1 * 2^(m1 - M) + d2 * 2^(m2 - M)),  M = max
// with m = -inf acting as the identity (never evaluating -inf - -inf).  The
// output is the stored exponential times 2^(m - M) / D: one exp2 per element.
#include "device_common.hpp"
#include "launch.hpp"

namespace fs {
namespace {

struct MaxSumP {
  float m, d;
  __device__ __forceinline__ static MaxSumP combine(const MaxSumP& a, const MaxSumP& b) {
    const float M = fmaxf(a.m, b.m);
    if (M == -INFINITY) return {-INFINITY, 0.f};
    // symmetric in (a, b): both products are formed the same way
    return {M, a.d * __builtin_amdgcn_exp2f(a.m - M) + b.d * __builtin_amdgcn_exp2f(b.m - M)};
  }
  template <class F> __device__ __forceinline__ static MaxSumP map(const MaxSumP& a, F f) {
    return {f(a.m), f(a.d)};
  }
};

// T: storage type of x and y; MT: storage type of the mask.
// W waves per row; EPT elements per thread; VEC: 16-byte vector path.
// G rows per block (W == 1 only).
template <typename T, typename MT, int W, int EPT, bool VEC, int G>
__global__ __launch_bounds__(64 * W * G) void softmax_kernel(
    const T* __restrict__ x, int64_t ld_x, const MT* __restrict__ mask, int64_t ld_m,
    T* y, int64_t ld_y, int64_t rows, int cols, float scale, int64_t q_len) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  constexpr int NV = EPT / V;                       // vectors per thread
  static_assert(EPT % V == 0, "EPT must be a multiple of the vector width");
  __shared__ MaxSumP lds[2][W];

  const int tid = threadIdx.x % kThreads;
  const int wave = tid / 64, lane = tid % 64;
  const int g = threadIdx.x / kThreads;
  const bool has_mask = mask != nullptr;
  const float scale_log2e = scale * kLog2e;
  int parity = 0;

  for (int64_t row = int64_t(blockIdx.x) * G + g; row < rows; row += int64_t(gridDim.x) * G) {
    const T* xr = x + row * ld_x;
    const MT* mr = has_mask ? mask + row * ld_m : nullptr;
    // last unmasked column (inclusive) under the causal rule
    const int64_t limit = q_len > 0 ? (row % q_len) + (cols - q_len) : int64_t(cols) - 1;
    const int lim = int(limit < int64_t(cols) - 1 ? limit : int64_t(cols) - 1);

    // a = (x * scale + mask) * log2(e): base-2 exponents
    float a[EPT];
    if constexpr (VEC) {
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = (k * kThreads + tid) * V;
        float xv[V];
        if (c0 <= lim) {
          ldv<T, V>(xr + c0, xv);
          if (has_mask) {
            float mv[V];
            ldv<MT, V>(mr + c0, mv);
#pragma unroll
            for (int i = 0; i < V; ++i) xv[i] = fmaf(xv[i], scale, mv[i]) * kLog2e;
          } else {
#pragma unroll
            for (int i = 0; i < V; ++i) xv[i] *= scale_log2e;
          }
#pragma unroll
          for (int i = 0; i < V; ++i) a[k * V + i] = (c0 + i <= lim) ? xv[i] : -INFINITY;
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i) a[k * V + i] = -INFINITY;
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int c = k * kThreads + tid;
        float v = -INFINITY;
        if (c <= lim) {
          const float xv = Elem<T>::load1(xr + c);
          v = has_mask ? fmaf(xv, scale, Elem<MT>::load1(mr + c)) * kLog2e : xv * scale_log2e;
        }
        a[k] = v;
      }
    }

    // local (m, d), exponentials kept in a[]
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < EPT; ++i) m = fmaxf(m, a[i]);
    const float m_safe = (m == -INFINITY) ? 0.f : m;
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      a[i] = __builtin_amdgcn_exp2f(a[i] - m_safe);   // exp2(-inf) = 0
      d += a[i];
    }

    MaxSumP p = group_allreduce<W>(MaxSumP{m, d}, lds[parity], wave, lane);
    parity ^= 1;
    // fully masked row: p.m = -inf, every a[i] = 0 -> output 0
    const float f = (p.m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_safe - p.m) / p.d;

    T* yr = y + row * ld_y;
    if constexpr (VEC) {
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = (k * kThreads + tid) * V;
        if (c0 < cols) {
          float o[V];
#pragma unroll
          for (int i = 0; i < V; ++i) o[i] = a[k * V + i] * f;
          st128<true>(yr + c0, Elem<T>::pack(o));
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int c = k * kThreads + tid;
        if (c < cols) Elem<T>::store1(yr + c, a[k] * f);
      }
    }
  }
}


template <typename T, typename MT, bool VEC>
hipError_t dispatch(const SoftmaxArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  // smallest capacity >= cols; the vector path needs EPT >= V
  const int64_t c = a.cols;
  auto launch = [&](auto kern, int threads, int rows_per_block, int blocks_per_cu) {
    int64_t want = (a.rows + rows_per_block - 1) / rows_per_block;
    int64_t cap = int64_t(cus) * blocks_per_cu;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s,
                       static_cast<const T*>(a.x), a.ld_x, static_cast<const MT*>(a.mask),
                       a.ld_mask, static_cast<T*>(a.y), a.ld_y, a.rows, int(a.cols),
                       a.scale, a.causal_q_len);
    return hipGetLastError();
  };
#define FS_SM(Wv, E, Gv, BPC)                                                      \
  if (c <= int64_t(64) * Wv * E)                                                    \
    return launch(softmax_kernel<T, MT, Wv, E, VEC, Gv>, 64 * Wv * Gv, Gv, BPC);
  if constexpr (V <= 1) { FS_SM(1, 1, 4, 64) }
  if constexpr (V <= 2) { FS_SM(1, 2, 4, 64) }
  if constexpr (V <= 4) { FS_SM(1, 4, 4, 64) }
  FS_SM(1, 8, 4, 64)
  FS_SM(1, 16, 4, 64)
  FS_SM(1, 32, 4, 32)
  FS_SM(1, 64, 4, 16)
  FS_SM(2, 64, 1, 32)
  FS_SM(4, 64, 1, 16)
  FS_SM(8, 64, 1, 8)
  FS_SM(16, 64, 1, 4)
#undef FS_SM
  return hipErrorInvalidValue;   // unreachable: the host checks cols
}

}  // namespace

hipError_t launch_softmax(const SoftmaxArgs& a, int cus, hipStream_t s) {
  const bool bf16 = a.dtype == FS_BF16;
  const bool mbf16 = a.mask_dtype == FS_BF16;
  if (bf16) {
    if (mbf16) return a.vec ? dispatch<uint16_t, uint16_t, true>(a, cus, s)
                            : dispatch<uint16_t, uint16_t, false>(a, cus, s);
    return a.vec ? dispatch<uint16_t, float, true>(a, cus, s)
                 : dispatch<uint16_t, float, false>(a, cus, s);
  }
  if (mbf16) return a.vec ? dispatch<float, uint16_t, true>(a, cus, s)
                          : dispatch<float, uint16_t, false>(a, cus, s);
  return a.vec ? dispatch<float, float, true>(a, cus, s) : dispatch<float, float, false>(a, cus, s);
}

}  // namespace fs
