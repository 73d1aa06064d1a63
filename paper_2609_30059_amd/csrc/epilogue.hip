// GEMM epilogue with a row reduction, applied to a library GEMM's output C:
//
//   out[i] = reduce_j act((C[i, j] + bias[j]) * col_scale[j])
//
// KernelOPT Appendix A (Codegen prompt: keep the matmul a library call and
// fuse only its epilogue; Fusion Agent: reduction + pointwise).
//
// Design (gfx950): a block of W wave64s owns ALL columns of the matrix and
// walks down the rows (grid-stride).  Each thread owns NV 16-byte column
// vectors and keeps their epilogue coefficients in registers for the whole
// kernel, so C is the only HBM stream; bias and scale are read once per
// block.  (C + b) * s is evaluated as C * s + b * s (one FMA); for the
// sigmoid the factor -log2(e) is folded into both coefficients so that
// sigmoid = 1 / (1 + 2^u) costs one v_exp_f32 and one v_rcp_f32.  R rows are
// processed per trip; their W per-wave partial sums meet in LDS
// (double-buffered, one barrier per trip) and R threads finish them.
#include "device_common.hpp"
#include "launch.hpp"

namespace fs {
namespace {

template <int ACT>
__device__ __forceinline__ float epi_act(float u) {
  if constexpr (ACT == FS_ACT_SIGMOID) {
    return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(u));   // u = -t*log2(e)
  } else if constexpr (ACT == FS_ACT_GELU_ERF) {
    return 0.5f * u * (1.f + erff(u * 0.70710678118654752f));
  } else if constexpr (ACT == FS_ACT_RELU) {
    return u > 0.f ? u : 0.f;
  } else {
    return u;
  }
}

template <int R>
struct RowSums {
  float s[R];
  __device__ __forceinline__ static RowSums combine(const RowSums& a, const RowSums& b) {
    RowSums o;
#pragma unroll
    for (int r = 0; r < R; ++r) o.s[r] = a.s[r] + b.s[r];
    return o;
  }
  template <class F> __device__ __forceinline__ static RowSums map(const RowSums& a, F f) {
    RowSums o;
#pragma unroll
    for (int r = 0; r < R; ++r) o.s[r] = f(a.s[r]);
    return o;
  }
};

template <typename CT, typename BT, int ACT, int W, int NV, int R, bool VEC>
__global__ __launch_bounds__(64 * W) void epilogue_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ col_scale, float* __restrict__ out, int64_t rows, int cols,
    int mean) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC ? Elem<CT>::kVec : 1;
  __shared__ float lds[2][R][W];
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;

  // per-column coefficients: u = C * sc + bs
  float sc[NV][V], bs[NV][V];
  const float sgn = (ACT == FS_ACT_SIGMOID) ? -kLog2e : 1.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c0 = (k * kThreads + tid) * V;
#pragma unroll
    for (int i = 0; i < V; ++i) {
      const int col = c0 + i;
      float s = 0.f, b = 0.f;
      if (col < cols) {
        s = col_scale ? col_scale[col] : 1.f;
        b = bias ? Elem<BT>::load1(bias + col) : 0.f;
      }
      sc[k][i] = s * sgn;
      bs[k][i] = b * s * sgn;
    }
  }

  int parity = 0;
  for (int64_t r0 = int64_t(blockIdx.x) * R; r0 < rows; r0 += int64_t(gridDim.x) * R) {
    float cv[R][NV][V];
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = (k * kThreads + tid) * V;
        if (r0 + r < rows && c0 < cols) {
          ldv<CT, V>(c + (r0 + r) * ld_c + c0, cv[r][k]);
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i) cv[r][k][i] = 0.f;
        }
      }
    }
    RowSums<R> ps;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = (k * kThreads + tid) * V;
        if (c0 < cols) {
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const float v = epi_act<ACT>(fmaf(cv[r][k][i], sc[k][i], bs[k][i]));
            if (VEC || c0 + i < cols) acc += v;
          }
        }
      }
      ps.s[r] = acc;
    }
    ps = wave_allreduce(ps);
    if constexpr (W == 1) {
      // every lane holds the R sums; lane r stores row r0 + r
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (lane == r && r0 + r < rows) out[r0 + r] = mean ? ps.s[r] / float(cols) : ps.s[r];
      }
    } else {
      if (lane == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r) lds[parity][r][wave] = ps.s[r];
      }
      __syncthreads();
      if (tid < R && r0 + tid < rows) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < W; ++w) t += lds[parity][tid][w];
        out[r0 + tid] = mean ? t / float(cols) : t;
      }
      parity ^= 1;
    }
  }
}

// Rows longer than the register-resident capacity: one block per row, the
// coefficients read through the cache for every element.
template <typename CT, typename BT, int ACT>
__global__ __launch_bounds__(256) void epilogue_wide_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ col_scale, float* __restrict__ out, int64_t rows, int64_t cols,
    int mean) {
  __shared__ SumP lds[2][4];
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const float sgn = (ACT == FS_ACT_SIGMOID) ? -kLog2e : 1.f;
  int parity = 0;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const CT* cr = c + row * ld_c;
    float acc = 0.f;
    for (int64_t j = tid; j < cols; j += 256) {
      const float s = (col_scale ? col_scale[j] : 1.f) * sgn;
      const float b = bias ? Elem<BT>::load1(bias + j) : 0.f;
      acc += epi_act<ACT>(fmaf(Elem<CT>::load1(cr + j), s, b * s));
    }
    const SumP t = group_allreduce<4>(SumP{acc}, lds[parity], wave, lane);
    parity ^= 1;
    if (tid == 0) out[row] = mean ? t.s / float(cols) : t.s;
  }
}

template <typename CT, typename BT, int ACT, bool VEC>
hipError_t dispatch(const EpilogueArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<CT>::kVec : 1;
  constexpr int R = 2;
  const int64_t c = a.cols;
  const int mean = a.reduce == FS_REDUCE_MEAN;
  auto launch = [&](auto kern, int threads, int blocks_per_cu) {
    int64_t want = (a.rows + R - 1) / R;
    int64_t cap = int64_t(cus) * blocks_per_cu;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s, static_cast<const CT*>(a.c), a.ld_c,
                       static_cast<const BT*>(a.bias), a.col_scale, a.out, a.rows, int(a.cols),
                       mean);
    return hipGetLastError();
  };
#define FS_EP(Wv, NVv, BPC)                                                           \
  if (c <= int64_t(64) * Wv * NVv * V)                                                 \
    return launch(epilogue_kernel<CT, BT, ACT, Wv, NVv, R, VEC>, 64 * Wv, BPC);
  if constexpr (VEC) {
    FS_EP(1, 1, 16)
    FS_EP(1, 2, 16)
    FS_EP(2, 2, 8)
    FS_EP(4, 2, 4)
    FS_EP(4, 4, 4)
    FS_EP(8, 4, 2)
  } else {
    FS_EP(1, 1, 16)
    FS_EP(1, 4, 16)
    FS_EP(4, 4, 4)
    FS_EP(4, 16, 4)
    FS_EP(16, 16, 1)
  }
#undef FS_EP
  int64_t grid = a.rows < int64_t(cus) * 8 ? a.rows : int64_t(cus) * 8;
  hipLaunchKernelGGL((epilogue_wide_kernel<CT, BT, ACT>), dim3(unsigned(grid)), dim3(256), 0, s,
                     static_cast<const CT*>(a.c), a.ld_c, static_cast<const BT*>(a.bias),
                     a.col_scale, a.out, a.rows, a.cols, mean);
  return hipGetLastError();
}

template <typename CT, typename BT, bool VEC>
hipError_t by_act(const EpilogueArgs& a, int cus, hipStream_t s) {
  switch (a.act) {
    case FS_ACT_SIGMOID: return dispatch<CT, BT, FS_ACT_SIGMOID, VEC>(a, cus, s);
    case FS_ACT_GELU_ERF: return dispatch<CT, BT, FS_ACT_GELU_ERF, VEC>(a, cus, s);
    case FS_ACT_RELU: return dispatch<CT, BT, FS_ACT_RELU, VEC>(a, cus, s);
    default: return dispatch<CT, BT, FS_ACT_NONE, VEC>(a, cus, s);
  }
}

template <typename CT>
hipError_t by_bias(const EpilogueArgs& a, int cus, hipStream_t s) {
  if (a.bias_dtype == FS_BF16)
    return a.vec ? by_act<CT, uint16_t, true>(a, cus, s) : by_act<CT, uint16_t, false>(a, cus, s);
  return a.vec ? by_act<CT, float, true>(a, cus, s) : by_act<CT, float, false>(a, cus, s);
}

}  // namespace

hipError_t launch_epilogue(const EpilogueArgs& a, int cus, hipStream_t s) {
  return a.c_dtype == FS_BF16 ? by_bias<uint16_t>(a, cus, s) : by_bias<float>(a, cus, s);
}

}  // namespace fs
