// GEMM epilogue with a row max or log-sum-exp:
//   out[i] = max_j act((C[i, j] + bias[j]) * col_scale[j])            (FS_REDUCE_MAX)
//          = log sum_j exp(act((C[i, j] + bias[j]) * col_scale[j]))   (FS_REDUCE_LOGSUMEXP)
//
// The reductions KernelOPT's level-2 case study chains after a linear layer
// (sum, max, mean, log-sum-exp), fused with the epilogue as its Appendix A
// prompts ask (keep the matmul a library call, fuse reduction + pointwise).
// The sum and mean run in epilogue.hip; these two reductions merge (max) and
// (max, sum of exp(v - max)) pairs instead of sums.
//
// Design (gfx950): one row per 256-thread block at a time (grid-stride over
// rows), the row streamed in trips of 4 16-byte vectors of C per lane, every
// load of a trip issued before any use, one pair per lane merged per vector,
// then a block all-reduce of the pairs.  Rows of one trip (up to 8192 bf16
// columns) keep each lane's column coefficients in registers for all its
// rows; longer rows load them per trip from the cache.  A vector's
// values are first reduced among themselves (their maximum, then the sum of
// exp(v - that maximum) as independent terms), so the dependent merge runs
// once per vector.
#include <type_traits>

#include "device_common.hpp"
#include "launch.hpp"

namespace fs {
namespace {

constexpr int kRowsBlock = 256;

struct EMaxP {   // NaN-propagating maximum
  float m;
  __device__ __forceinline__ static EMaxP combine(const EMaxP& a, const EMaxP& b) {
    return {__builtin_elementwise_maximum(a.m, b.m)};
  }
  template <class F> __device__ __forceinline__ static EMaxP map(const EMaxP& a, F f) {
    return {f(a.m)};
  }
};

// (m, s): the largest value and the sum of exp(v - m); a part whose maximum
// equals the merged one keeps its sum (no inf - inf), NaN propagates.
struct ELseP {
  float m, s;
  __device__ __forceinline__ static float scaled(float s, float m, float M) {
    const float ms = M == -INFINITY ? 0.f : M;
    return m == M ? s : s * __builtin_amdgcn_exp2f((m - ms) * kLog2e);
  }
  __device__ __forceinline__ static ELseP combine(const ELseP& a, const ELseP& b) {
    const float M = __builtin_elementwise_maximum(a.m, b.m);
    return {M, scaled(a.s, a.m, M) + scaled(b.s, b.m, M)};
  }
  template <class F> __device__ __forceinline__ static ELseP map(const ELseP& a, F f) {
    return {f(a.m), f(a.s)};
  }
};

template <int ACT>
__device__ __forceinline__ float act_of(float t) {
  if constexpr (ACT == FS_ACT_GELU_ERF) return gelu_erf(t);
  else if constexpr (ACT == FS_ACT_SIGMOID) return sigmoid(t);
  else if constexpr (ACT == FS_ACT_RELU) return t < 0.f ? 0.f : t;   // a NaN stays NaN
  else return t;
}

// RES: every row fits one trip (cols <= 256 * V * U), so each lane's columns
// are the same in every row and their (s, b * s) stay in registers for all
// the rows it processes; otherwise the coefficients are loaded per trip
// (cache-resident).  (c + b) * s is evaluated as fma(c, s, b * s).
template <typename CT, typename BT, int ACT, bool LSE, bool VEC, bool RES>
__global__ __launch_bounds__(kRowsBlock) void epilogue_rows_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ scale, float* __restrict__ out, int64_t rows, int cols) {
  constexpr int V = VEC ? Elem<CT>::kVec : 1;
  constexpr int W = kRowsBlock / 64;
  constexpr int U = 4;                         // vectors per lane per trip
  using P = typename std::conditional<LSE, ELseP, EMaxP>::type;
  __shared__ P lds[2][W];
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int clast = cols - V;                  // start of a row's last vector
  const int trips = RES ? 1 : (cols + kRowsBlock * V * U - 1) / (kRowsBlock * V * U);
  int parity = 0;

  // (s, b * s) of the lane's vectors of trip t
  float sc[U][V], bs[U][V];
  auto coefs = [&](int t) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c0 = ((t * U + u) * kRowsBlock + tid) * V;
      const int cl = c0 < cols ? c0 : clast;
      float bv[V];
      if (bias) {
        Raw<BT, V> rb;
        rb.template load<false>(bias + cl);
        rb.unpack(bv);
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) bv[i] = 0.f;
      }
      if (scale) {
        Raw<float, V> rs;
        rs.template load<false>(scale + cl);
        rs.unpack(sc[u]);
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) sc[u][i] = 1.f;
      }
#pragma unroll
      for (int i = 0; i < V; ++i) bs[u][i] = bv[i] * sc[u][i];
    }
  };
  if constexpr (RES) coefs(0);

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const CT* cr = c + row * ld_c;
    P acc;
    if constexpr (LSE) acc = ELseP{-INFINITY, 0.f};
    else acc = EMaxP{-INFINITY};
    for (int t = 0; t < trips; ++t) {
      // the trip's C loads first (vectors past the row end re-read its last
      // vector, in bounds, and count nothing)
      Raw<CT, V> rc[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = ((t * U + u) * kRowsBlock + tid) * V;
        rc[u].load(cr + (c0 < cols ? c0 : clast));
      }
      if constexpr (!RES) coefs(t);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = ((t * U + u) * kRowsBlock + tid) * V;
        float z[V];
        rc[u].unpack(z);
        float vm = -INFINITY;
#pragma unroll
        for (int i = 0; i < V; ++i) {
          z[i] = act_of<ACT>(fmaf(z[i], sc[u][i], bs[u][i]));
          vm = __builtin_elementwise_maximum(vm, z[i]);
        }
        if (c0 >= cols) continue;
        if constexpr (LSE) {
          // sum of exp(z - vm) as exp2((z - vm) log2e): the difference first,
          // exact near the maximum at any magnitude (the one-fma form
          // z log2e - round(vm log2e) carries that rounding, which past
          // |vm| ~ 1e9 overflows the exponent); a vector whose maximum is
          // +inf counts its +inf values without forming inf - inf
          float vs = 0.f;
          if (vm == INFINITY) {
#pragma unroll
            for (int i = 0; i < V; ++i) vs += z[i] == vm ? 1.f : 0.f;
          } else {
            const float ms = vm == -INFINITY ? 0.f : vm;
#pragma unroll
            for (int i = 0; i < V; ++i) vs += __builtin_amdgcn_exp2f((z[i] - ms) * kLog2e);
          }
          acc = ELseP::combine(acc, ELseP{vm, vs});
        } else {
          acc = EMaxP::combine(acc, EMaxP{vm});
        }
      }
    }
    const P tot = group_allreduce<W>(acc, lds[parity], wave, lane);
    parity ^= 1;
    if (tid == 0) {
      if constexpr (LSE) out[row] = tot.m + logf(tot.s);   // -inf + -inf, inf + log s
      else out[row] = tot.m;
    }
  }
}

template <typename CT, typename BT, int ACT>
hipError_t dispatch(const EpilogueArgs& a, int cus, hipStream_t s) {
  const bool lse = a.reduce == FS_REDUCE_LOGSUMEXP;
  const int64_t cap = int64_t(cus) * 8;
  const unsigned grid = unsigned(a.rows < cap ? a.rows : cap);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kRowsBlock), 0, s, static_cast<const CT*>(a.c),
                       a.ld_c, static_cast<const BT*>(a.bias), a.col_scale, a.out, a.rows,
                       int(a.cols));
    return hipGetLastError();
  };
  // the vector path also loads bias and col_scale 16 bytes at a time
  if (a.vec && a.coef_vec) {
    constexpr int V = Elem<CT>::kVec;
    if (a.cols <= int64_t(kRowsBlock) * V * 4)
      return lse ? go(epilogue_rows_kernel<CT, BT, ACT, true, true, true>)
                 : go(epilogue_rows_kernel<CT, BT, ACT, false, true, true>);
    return lse ? go(epilogue_rows_kernel<CT, BT, ACT, true, true, false>)
               : go(epilogue_rows_kernel<CT, BT, ACT, false, true, false>);
  }
  return lse ? go(epilogue_rows_kernel<CT, BT, ACT, true, false, false>)
             : go(epilogue_rows_kernel<CT, BT, ACT, false, false, false>);
}

template <typename CT, typename BT>
hipError_t by_act(const EpilogueArgs& a, int cus, hipStream_t s) {
  switch (a.act) {
    case FS_ACT_GELU_ERF: return dispatch<CT, BT, FS_ACT_GELU_ERF>(a, cus, s);
    case FS_ACT_SIGMOID: return dispatch<CT, BT, FS_ACT_SIGMOID>(a, cus, s);
    case FS_ACT_RELU: return dispatch<CT, BT, FS_ACT_RELU>(a, cus, s);
    default: return dispatch<CT, BT, FS_ACT_NONE>(a, cus, s);
  }
}

}  // namespace

hipError_t launch_epilogue_maxlse(const EpilogueArgs& a, int cus, hipStream_t s) {
  const bool bias_bf16 = a.bias != nullptr && a.bias_dtype == FS_BF16;
  if (a.c_dtype == FS_BF16)
    return bias_bf16 ? by_act<uint16_t, uint16_t>(a, cus, s) : by_act<uint16_t, float>(a, cus, s);
  return bias_bf16 ? by_act<float, uint16_t>(a, cus, s) : by_act<float, float>(a, cus, s);
}

}  // namespace fs
