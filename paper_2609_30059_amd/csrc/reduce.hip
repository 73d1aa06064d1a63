// Plain row reductions: sum, mean, max, log-sum-exp (fp32 out) and bit-exact
// argmax (int64 out, lowest index on ties, first NaN wins).
//
// KernelOPT Section 6 counts sum/mean reductions among the optimised
// sub-kernel classes; Appendix A (Executor prompt) asks for fp32 accumulation.
//
// Design (gfx950): a group of W wave64s per row; the row is streamed in trips
// of U 16-byte vectors per lane, all U loads issued before any use, with a
// trip count that is uniform across the group (lanes past the row end re-read
// the row's last vector and mask it).  Rows of any length are supported; the
// per-lane partials meet in one wave all-reduce (plus an LDS fold when W > 1).
#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_RED_UNROLL
#define FS_RED_UNROLL 4
#endif

namespace fs {
namespace {

struct MaxP {   // NaN-propagating maximum
  float m;
  __device__ __forceinline__ static MaxP combine(const MaxP& a, const MaxP& b) {
    if (a.m != a.m) return a;
    if (b.m != b.m) return b;
    return {fmaxf(a.m, b.m)};
  }
  template <class F> __device__ __forceinline__ static MaxP map(const MaxP& a, F f) {
    return {f(a.m)};
  }
};

// (value, index): larger value wins, NaN above every number, lowest index on
// a tie (between two NaNs too).  combine(a, b) == combine(b, a).
struct ArgP {
  float v;
  int i;
  // written with selects only: early returns of the struct kept it in
  // scratch memory
  __device__ __forceinline__ static ArgP combine(const ArgP& a, const ArgP& b) {
    const bool an = a.v != a.v, bn = b.v != b.v;
    const bool a_wins = an ? (!bn || a.i < b.i)
                           : (!bn && (a.v > b.v || (a.v == b.v && a.i < b.i)));
    return {a_wins ? a.v : b.v, a_wins ? a.i : b.i};
  }
  template <class F> __device__ __forceinline__ static ArgP map(const ArgP& a, F f) {
    return {f(a.v), __float_as_int(f(__int_as_float(a.i)))};
  }
};

// (m, s): the largest value seen and the sum of exp(v - m) over the values
// seen, for a log-sum-exp.  Merging rescales the sum of the smaller maximum
// by exp(m - M); a part whose maximum equals M keeps its sum as it is, so
// infinite maxima merge without inf - inf.  NaN propagates through M.
struct LseP {
  float m, s;
  __device__ __forceinline__ static float scaled(float s, float m, float M) {
    const float ms = M == -INFINITY ? 0.f : M;   // all -inf: every sum is 0
    return m == M ? s : s * __builtin_amdgcn_exp2f((m - ms) * kLog2e);
  }
  __device__ __forceinline__ static LseP combine(const LseP& a, const LseP& b) {
    const float M = __builtin_elementwise_maximum(a.m, b.m);
    return {M, scaled(a.s, a.m, M) + scaled(b.s, b.m, M)};
  }
  template <class F> __device__ __forceinline__ static LseP map(const LseP& a, F f) {
    return {f(a.m), f(a.s)};
  }
};

constexpr int kOpSum = 0, kOpMax = 2, kOpArg = 3, kOpLse = 4;   // MEAN runs as SUM

template <int OP> struct AccOf;
template <> struct AccOf<kOpSum> { using type = SumP; };
template <> struct AccOf<kOpMax> { using type = MaxP; };
template <> struct AccOf<kOpArg> { using type = ArgP; };
template <> struct AccOf<kOpLse> { using type = LseP; };

template <int OP>
__device__ __forceinline__ typename AccOf<OP>::type identity() {
  if constexpr (OP == kOpSum) return SumP{0.f};
  else if constexpr (OP == kOpMax) return MaxP{-INFINITY};
  else if constexpr (OP == kOpLse) return LseP{-INFINITY, 0.f};
  else return ArgP{-INFINITY, 0x7fffffff};
}

// One step of an accumulator that sees its columns in increasing order.
// Argmax keeps the first of equal values and the first NaN: it moves only to
// a strictly larger value, or to a NaN while it holds none (`first` takes the
// accumulator's first element whatever it is, -inf and NaN included).  Max
// propagates NaN (v_maximum3_f32 on gfx950).
template <int OP>
__device__ __forceinline__ void accumulate(typename AccOf<OP>::type& acc, float v, int col,
                                           bool first) {
  if constexpr (OP == kOpSum) {
    acc.s += v;
  } else if constexpr (OP == kOpMax) {
    acc.m = __builtin_elementwise_maximum(acc.m, v);
  } else if constexpr (OP == kOpLse) {
    acc = LseP::combine(acc, LseP{v, 1.f});
  } else {
    const bool upd = first || (!(v <= acc.v) && acc.v == acc.v);
    acc.v = upd ? v : acc.v;
    acc.i = upd ? col : acc.i;
  }
}

// SHIFT (element-aligned rows that are not whole 16-byte vectors): 16-byte
// loads over each row's aligned body [h, bend) and one extra element per
// lane for the first h + (cols - bend) lanes (the head and the tail, at most
// 2 V - 2), merged with the symmetric combine, which keeps argmax exact.
template <typename T, int OP, int W, int G, bool VEC, bool SHIFT>
__global__ __launch_bounds__(64 * W * G) void reduce_kernel(
    const T* __restrict__ x, int64_t ld_x, float* __restrict__ out_f,
    int64_t* __restrict__ out_i, int64_t rows, int cols, int trips, float post_scale) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC || SHIFT ? Elem<T>::kVec : 1;
  constexpr int U = FS_RED_UNROLL;
  // one LDS fold area and one barrier sequence per block: rows wider than a
  // wave take the whole block (the row loop is then uniform across it)
  static_assert(W == 1 || G == 1, "multi-wave rows use one row group per block");
  using P = typename AccOf<OP>::type;
  __shared__ P lds[2][W];
  const int tid = threadIdx.x % kThreads;
  const int wave = tid / 64, lane = tid % 64;
  const int g = __builtin_amdgcn_readfirstlane(threadIdx.x / kThreads);   // wave-uniform
  const int clast = cols - V;     // start of the row's last vector
  int parity = 0;

  for (int64_t row = int64_t(blockIdx.x) * G + g; row < rows; row += int64_t(gridDim.x) * G) {
    const T* xr = x + row * ld_x;
    int h = 0, bend = cols;   // the row's 16-byte-aligned body (SHIFT)
    if constexpr (SHIFT) {
      const int phase = int(reinterpret_cast<uintptr_t>(xr) & 15) / int(sizeof(T));
      h = (V - phase) % V;
      bend = h + ((cols - h) / V) * V;
    }
    const int blast = bend - V;   // start of the body's last vector
    // V independent accumulators, one per slot of a vector: each sees its
    // columns in increasing order, and their chains run side by side (one
    // chain through all of a lane's elements made max and argmax
    // latency-bound, ten times slower than the sum)
    P acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = identity<OP>();
    for (int t = 0; t < trips; ++t) {
      Raw<T, V> rv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = h + ((t * U + u) * kThreads + tid) * V;
        rv[u].load(xr + (c0 < bend ? c0 : (SHIFT ? blast : clast)));
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (OP == kOpLse) {
        // the trip's values at once: their maximum tm, the sum of
        // exp(v - tm) over them (independent terms), then one merge into the
        // running pair -- about one exponential per value and one dependent
        // merge per trip; vectors past the row end count nothing.
        float vals[U][V];
        float tm = -INFINITY;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c0 = h + ((t * U + u) * kThreads + tid) * V;
          rv[u].unpack(vals[u]);
#pragma unroll
          for (int i = 0; i < V; ++i)
            tm = c0 < bend ? __builtin_elementwise_maximum(tm, vals[u][i]) : tm;
        }
        // exp(v - tm) as exp2((v - tm) log2e): the difference first, exact
        // near the maximum at any magnitude (the one-fma form carries the
        // rounding of tm log2e, which past |tm| ~ 1e9 overflows the
        // exponent); a trip whose maximum is +inf counts its +inf values
        // without inf - inf
        float ts = 0.f;
        if (tm == INFINITY) {
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int c0 = h + ((t * U + u) * kThreads + tid) * V;
#pragma unroll
            for (int i = 0; i < V; ++i) ts += c0 < bend && vals[u][i] == tm ? 1.f : 0.f;
          }
        } else {
          const float tms = tm == -INFINITY ? 0.f : tm;
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int c0 = h + ((t * U + u) * kThreads + tid) * V;
#pragma unroll
            for (int i = 0; i < V; ++i) {
              const float e = __builtin_amdgcn_exp2f((vals[u][i] - tms) * kLog2e);
              ts += c0 < bend ? e : 0.f;
            }
          }
        }
        acc[0] = LseP::combine(acc[0], LseP{tm, ts});
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int c0 = h + ((t * U + u) * kThreads + tid) * V;
          // the lane's first vector holds its lowest columns; if it lies past
          // the row end, so do all the lane's vectors
          const bool first = t == 0 && u == 0;
          float v[V];
          rv[u].unpack(v);
          if (c0 < bend) {   // the whole vector is in the row (or body)
#pragma unroll
            for (int i = 0; i < V; ++i) accumulate<OP>(acc[i], v[i], c0 + i, first);
          }
        }
      }
    }
    P lane_acc = acc[0];
#pragma unroll
    for (int i = 1; i < V; ++i) lane_acc = P::combine(lane_acc, acc[i]);
    if constexpr (SHIFT) {
      const int nx = h + (cols - bend);
      const bool has = tid < nx;
      const int ce = has ? (tid < h ? tid : bend + (tid - h)) : 0;
      P ax = identity<OP>();
      const float v = Elem<T>::load1(xr + ce);
      if (has) accumulate<OP>(ax, v, ce, true);
      lane_acc = P::combine(lane_acc, ax);
    }
    const P tot = group_allreduce<W>(lane_acc, lds[parity], wave, lane);
    parity ^= 1;
    if (tid == 0) {
      if constexpr (OP == kOpArg) out_i[row] = tot.i;
      else if constexpr (OP == kOpSum) out_f[row] = tot.s * post_scale;
      else if constexpr (OP == kOpLse) out_f[row] = tot.m + logf(tot.s);   // -inf + -inf, inf + log s
      else out_f[row] = tot.m;
    }
  }
}

template <typename T, int OP, bool VEC, bool SHIFT>
hipError_t dispatch(const ReduceArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC || SHIFT ? Elem<T>::kVec : 1;
  constexpr int U = FS_RED_UNROLL;
  // waves per row: enough that a trip covers about half the row, at most 8
  const int64_t per_wave_trip = int64_t(64) * V * U;
  const int64_t want_w = (a.cols + 2 * per_wave_trip - 1) / (2 * per_wave_trip);
  const float post = (a.op == FS_ROW_MEAN && a.cols > 0) ? 1.f / float(a.cols) : 1.f;
  auto launch = [&](auto kern, int w, int g) {
    const int trips = int((a.cols + int64_t(64) * w * V * U - 1) / (int64_t(64) * w * V * U));
    int64_t want = (a.rows + g - 1) / g;
    int64_t cap = int64_t(cus) * (32 / (w * g) > 0 ? 32 / (w * g) : 1) * 4;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * w * g), 0, s, static_cast<const T*>(a.x),
                       a.ld_x, a.out_f, a.out_i, a.rows, int(a.cols), trips, post);
    return hipGetLastError();
  };
  if (want_w <= 1) return launch(reduce_kernel<T, OP, 1, 4, VEC, SHIFT>, 1, 4);
  if (want_w <= 2) return launch(reduce_kernel<T, OP, 2, 1, VEC, SHIFT>, 2, 1);
  if (want_w <= 4) return launch(reduce_kernel<T, OP, 4, 1, VEC, SHIFT>, 4, 1);
  return launch(reduce_kernel<T, OP, 8, 1, VEC, SHIFT>, 8, 1);
}

template <typename T, int OP>
hipError_t by_path(const ReduceArgs& a, int cus, hipStream_t s) {
  if (a.vec) return dispatch<T, OP, true, false>(a, cus, s);
  if (a.shifted) return dispatch<T, OP, false, true>(a, cus, s);
  return dispatch<T, OP, false, false>(a, cus, s);
}

template <typename T>
hipError_t by_op(const ReduceArgs& a, bool argmax, int cus, hipStream_t s) {
  if (argmax) return by_path<T, kOpArg>(a, cus, s);
  if (a.op == FS_ROW_MAX) return by_path<T, kOpMax>(a, cus, s);
  if (a.op == FS_ROW_LOGSUMEXP) return by_path<T, kOpLse>(a, cus, s);
  return by_path<T, kOpSum>(a, cus, s);
}

}  // namespace

hipError_t launch_reduce(const ReduceArgs& a, int cus, hipStream_t s) {
  const bool argmax = a.out_i != nullptr;
  return a.dtype == FS_BF16 ? by_op<uint16_t>(a, argmax, cus, s) : by_op<float>(a, argmax, cus, s);
}

}  // namespace fs
