// Fused pointwise chain y = act(x * scale + bias[col]) + residual.
//
// KernelOPT Appendix A (Fusion Agent: pointwise + pointwise and activation +
// bias fusion -- load every input once, apply the whole chain in registers,
// store once).  Its Section 6 speedup analysis attributes the largest
// pointwise gains to removing the HBM round trips between separately
// launched elementwise kernels; here the whole chain is one pass.
//
// Design (gfx950): a block of 256 threads owns a slab of 256 column vectors
// (16 bytes each) and walks down the rows; the bias of its columns is loaded
// once into registers.  Each trip handles U rows so that 2U independent
// 128-bit loads are in flight per thread.  The grid is sized to a few blocks
// per compute unit and strides over the rows.
#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_PW_ROWS_PER_TRIP
#define FS_PW_ROWS_PER_TRIP 4
#endif
#ifndef FS_PW_BLOCKS_PER_CU
#define FS_PW_BLOCKS_PER_CU 16
#endif
#ifndef FS_PW_FLAT
#define FS_PW_FLAT 1            // dense rows without a bias walk one flat run of vectors
#endif
#ifndef FS_PW_FLAT_CHUNK
#define FS_PW_FLAT_CHUNK 4      // vectors per lane per wave chunk of the flat walk
#endif
#ifndef FS_PW_FLAT_BPC
#define FS_PW_FLAT_BPC 4        // its 256-thread blocks per compute unit
#endif

namespace fs {
namespace {

constexpr int kBlock = 256;

template <int ACT>
__device__ __forceinline__ float act_fn(float z) {
  if constexpr (ACT == FS_ACT_GELU_ERF) {
    return gelu_erf(z);
  } else if constexpr (ACT == FS_ACT_SIGMOID) {
    return sigmoid(z);
  } else if constexpr (ACT == FS_ACT_RELU) {
    return z < 0.f ? 0.f : z;   // a NaN stays NaN
  } else {
    return z;
  }
}

template <typename T, int ACT, bool HAS_RES, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void pointwise_kernel(
    const T* x, int64_t ld_x, const T* __restrict__ bias, const T* res, int64_t ld_r, T* y,
    int64_t ld_y, int64_t rows, int cols, float scale, int col_blocks) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  const int cb = blockIdx.x % col_blocks;
  const int64_t rg = blockIdx.x / col_blocks;
  const int64_t nrg = gridDim.x / col_blocks;
  const int c0 = (cb * kBlock + threadIdx.x) * V;
  if (c0 >= cols) return;               // no barriers below: early exit is safe

  float b[V];
  if (bias) {
    Raw<T, V> rb;
    rb.template load<false>(bias + c0);
    rb.unpack(b);
  } else {
#pragma unroll
    for (int i = 0; i < V; ++i) b[i] = 0.f;
  }

  for (int64_t r0 = rg * U; r0 < rows; r0 += nrg * U) {
    // all 2U loads of the trip are issued before any use; rows past the end
    // re-read the last row (in bounds) and are not stored
    Raw<T, V> rx[U], rr[HAS_RES ? U : 1];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = r0 + u < rows ? r0 + u : rows - 1;
      rx[u].load(x + r * ld_x + c0);
      if constexpr (HAS_RES) rr[u].load(res + r * ld_r + c0);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float xv[V], o[V];
      rx[u].unpack(xv);
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] = act_fn<ACT>(fmaf(xv[i], scale, b[i]));
      if constexpr (HAS_RES) {
        float rv[V];
        rr[u].unpack(rv);
#pragma unroll
        for (int i = 0; i < V; ++i) o[i] += rv[i];
      }
      if (r0 + u < rows) stv<T, V>(y + (r0 + u) * ld_y + c0, o);
    }
  }
}

// Dense rows without a bias (x, residual and y all with row stride == cols):
// the tensor is one contiguous run of n vectors, walked in chunks of 64 U
// vectors per wave (4 KiB of bf16 or fp32 for U = 4) with a grid stride.
// The U loads of a wave cover one contiguous span of every input, where the
// row-slab kernel reads U rows' 1 KiB slices; a short launch (the block's
// 96 MiB residual add) starts streaming sooner.  Vectors past the last whole
// chunk go one per thread.  Same arithmetic as pointwise_kernel.
template <typename T, int ACT, bool HAS_RES, int U>
__global__ __launch_bounds__(kBlock) void pointwise_flat_kernel(const T* x, const T* res, T* y,
                                                                int64_t n, float scale) {
  constexpr int V = Elem<T>::kVec;
  const int lane = threadIdx.x % 64;
  const int64_t wave = int64_t(blockIdx.x) * (kBlock / 64) + threadIdx.x / 64;
  const int64_t waves = int64_t(gridDim.x) * (kBlock / 64);
  const int64_t nch = n / (64 * U);
  auto chain = [](const Raw<T, V>& rx, const Raw<T, V>& rr, float scale, float* o) {
    float xv[V];
    rx.unpack(xv);
#pragma unroll
    for (int i = 0; i < V; ++i) o[i] = act_fn<ACT>(fmaf(xv[i], scale, 0.f));
    if constexpr (HAS_RES) {
      float rv[V];
      rr.unpack(rv);
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] += rv[i];
    }
  };
  for (int64_t c = wave; c < nch; c += waves) {
    const int64_t base = (c * 64 * U + lane) * V;
    Raw<T, V> rx[U], rr[HAS_RES ? U : 1];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      rx[k].load(x + base + k * 64 * V);
      if constexpr (HAS_RES) rr[k].load(res + base + k * 64 * V);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      float o[V];
      chain(rx[k], rr[HAS_RES ? k : 0], scale, o);
      stv<T, V>(y + base + k * 64 * V, o);
    }
  }
  for (int64_t v = nch * 64 * U + int64_t(blockIdx.x) * kBlock + threadIdx.x; v < n;
       v += int64_t(gridDim.x) * kBlock) {
    Raw<T, V> rx, rr;
    rx.load(x + v * V);
    if constexpr (HAS_RES) rr.load(res + v * V);
    float o[V];
    chain(rx, rr, scale, o);
    stv<T, V>(y + v * V, o);
  }
}

// Rows that are not whole 16-byte vectors (odd widths, odd row offsets) but
// whose x, residual and y start every row at one offset within a 16-byte
// unit: each row's aligned body, from its first 16-byte boundary to its last,
// is read and written 16 bytes at a time; thread t of column block cb owns
// body vector cb*kBlock + t of every row.  A row starting h columns before a
// 16-byte boundary puts element e of body vector v at column h + v*V + e, so
// the block stages the bias of its columns in LDS in V planes (column j at
// plane j % V, index j / V): element e reads plane (h+e) % V at index
// t + (h+e) / V, consecutive across the lanes whatever h is.  The head and
// tail of each row (at most V-1 elements each) go one per lane to wave 0 of
// column block 0, whose loads are issued with the body's.
template <typename T, int ACT, bool HAS_RES, int U>
__global__ __launch_bounds__(kBlock) void pointwise_shift_kernel(
    const T* x, int64_t ld_x, const T* __restrict__ bias, const T* res, int64_t ld_r, T* y,
    int64_t ld_y, int64_t rows, int cols, float scale, int col_blocks) {
  constexpr int V = Elem<T>::kVec;
  constexpr int Q = kBlock + 1;          // the block's vectors, plus the carry
  __shared__ float bpl[V * Q];
  const int cb = blockIdx.x % col_blocks;
  const int64_t rg = blockIdx.x / col_blocks;
  const int64_t nrg = gridDim.x / col_blocks;
  const int tid = threadIdx.x;
  const int v = cb * kBlock + tid;       // the thread's body vector
  // every staging load is issued before the first is used (a stand-in
  // pointer when there is no bias keeps them unconditional)
  constexpr int NS = (V * Q + kBlock - 1) / kBlock;
  const T* bsrc = bias != nullptr ? bias : x;
  float bst[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int i = tid + k * kBlock, pl = i / Q, q = i % Q;
    const int j = (cb * kBlock + q) * V + pl;
    bst[k] = Elem<T>::load1(bsrc + (i < V * Q && j < cols ? j : 0));
  }
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int i = tid + k * kBlock, pl = i / Q, q = i % Q;
    const int j = (cb * kBlock + q) * V + pl;
    if (i < V * Q) bpl[i] = bias != nullptr && j < cols ? bst[k] : 0.f;
  }
  __syncthreads();
  const bool edge = cb == 0 && tid < 64;   // uniform per wave
  if (v >= cols / V && !edge) return;      // no barriers below

  auto head_of = [&](int64_t r) {
    const int phase = int(reinterpret_cast<uintptr_t>(x + r * ld_x) & 15) / int(sizeof(T));
    return (V - phase) & (V - 1);
  };
  for (int64_t r0 = rg * U; r0 < rows; r0 += nrg * U) {
    Raw<T, V> rx[U], rr[HAS_RES ? U : 1];
    int hh[U], nb[U];
    T ex[U], er[U];
    float eb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = r0 + u < rows ? r0 + u : rows - 1;
      hh[u] = head_of(r);
      nb[u] = (cols - hh[u]) / V;          // >= 1: rows span at least two vectors
      const int vc = v < nb[u] ? v : nb[u] - 1;
      rx[u].load(x + r * ld_x + hh[u] + vc * V);
      if constexpr (HAS_RES) rr[u].load(res + r * ld_r + hh[u] + vc * V);
    }
    if (edge) {
      // lanes below h take the head, the next ones the tail (column
      // nb*V + lane); lanes past them re-read column 0 and store nothing
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t r = r0 + u < rows ? r0 + u : rows - 1;
        const int nx = cols - nb[u] * V;
        const int ce = tid < nx ? (tid < hh[u] ? tid : nb[u] * V + tid) : 0;
        ex[u] = x[r * ld_x + ce];
        if constexpr (HAS_RES) er[u] = res[r * ld_r + ce];
        eb[u] = Elem<T>::load1(bsrc + ce);   // zeroed at use when there is no bias
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float xv[V], o[V];
      rx[u].unpack(xv);
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const int he = hh[u] + e;
        const float b = bpl[(he & (V - 1)) * Q + (he >= V ? 1 : 0) + tid];
        o[e] = act_fn<ACT>(fmaf(xv[e], scale, b));
      }
      if constexpr (HAS_RES) {
        float rv[V];
        rr[u].unpack(rv);
#pragma unroll
        for (int e = 0; e < V; ++e) o[e] += rv[e];
      }
      if (r0 + u < rows && v < nb[u]) stv<T, V>(y + (r0 + u) * ld_y + hh[u] + v * V, o);
    }
    if (edge) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int nx = cols - nb[u] * V;
        if (r0 + u < rows && tid < nx) {
          const int ce = tid < hh[u] ? tid : nb[u] * V + tid;
          float o = act_fn<ACT>(fmaf(raw_f32(ex[u]), scale, bias != nullptr ? eb[u] : 0.f));
          if constexpr (HAS_RES) o += raw_f32(er[u]);
          Elem<T>::store1(y + (r0 + u) * ld_y + ce, o);
        }
      }
    }
  }
}

template <typename T, int ACT, bool HAS_RES, bool VEC>
hipError_t dispatch(const PointwiseArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  if constexpr (VEC) {
    // dense rows without a bias, large enough that every wave of the flat
    // grid gets at least one chunk
    constexpr int UF = FS_PW_FLAT_CHUNK;
    const bool dense = a.rows == 1 || (a.ld_x == a.cols && a.ld_y == a.cols &&
                                       (a.res == nullptr || a.ld_r == a.cols));
    const int64_t n = a.rows * (a.cols / V);
    const int64_t grid = int64_t(cus) * FS_PW_FLAT_BPC;
    if (FS_PW_FLAT && a.bias == nullptr && dense && n / (64 * UF) >= grid * (kBlock / 64)) {
      hipLaunchKernelGGL((pointwise_flat_kernel<T, ACT, HAS_RES, UF>), dim3(unsigned(grid)),
                         dim3(kBlock), 0, s, static_cast<const T*>(a.x),
                         static_cast<const T*>(a.res), static_cast<T*>(a.y), n, a.scale);
      return hipGetLastError();
    }
  }
  const int64_t vecs = (a.cols + V - 1) / V;
  const int col_blocks = int((vecs + kBlock - 1) / kBlock);
  // U rows per trip; fewer when the problem is too small to fill the chip
  constexpr int U = FS_PW_ROWS_PER_TRIP;
  const int64_t row_groups_needed = (a.rows + U - 1) / U;
  const int64_t target_blocks = int64_t(cus) * FS_PW_BLOCKS_PER_CU;
  int64_t rg = target_blocks / col_blocks;
  if (rg < 1) rg = 1;
  if (row_groups_needed < int64_t(cus) * 2) {
    // small problem: one row per trip, as many blocks as rows
    int64_t r1 = a.rows < target_blocks ? a.rows : target_blocks;
    int64_t grid = r1 * col_blocks;
    hipLaunchKernelGGL((pointwise_kernel<T, ACT, HAS_RES, VEC, 1>), dim3(unsigned(grid)), dim3(kBlock), 0,
                       s, static_cast<const T*>(a.x), a.ld_x, static_cast<const T*>(a.bias),
                       static_cast<const T*>(a.res), a.ld_r, static_cast<T*>(a.y), a.ld_y, a.rows,
                       int(a.cols), a.scale, col_blocks);
    return hipGetLastError();
  }
  if (rg > row_groups_needed) rg = row_groups_needed;
  const int64_t grid = rg * col_blocks;
  hipLaunchKernelGGL((pointwise_kernel<T, ACT, HAS_RES, VEC, U>), dim3(unsigned(grid)), dim3(kBlock), 0, s,
                     static_cast<const T*>(a.x), a.ld_x, static_cast<const T*>(a.bias),
                     static_cast<const T*>(a.res), a.ld_r, static_cast<T*>(a.y), a.ld_y, a.rows,
                     int(a.cols), a.scale, col_blocks);
  return hipGetLastError();
}

template <typename T, bool HAS_RES, bool VEC>
hipError_t by_act(const PointwiseArgs& a, int cus, hipStream_t s) {
  switch (a.act) {
    case FS_ACT_GELU_ERF: return dispatch<T, FS_ACT_GELU_ERF, HAS_RES, VEC>(a, cus, s);
    case FS_ACT_SIGMOID: return dispatch<T, FS_ACT_SIGMOID, HAS_RES, VEC>(a, cus, s);
    case FS_ACT_RELU: return dispatch<T, FS_ACT_RELU, HAS_RES, VEC>(a, cus, s);
    default: return dispatch<T, FS_ACT_NONE, HAS_RES, VEC>(a, cus, s);
  }
}

template <typename T, int ACT, bool HAS_RES>
hipError_t dispatch_shift(const PointwiseArgs& a, int cus, hipStream_t s) {
  constexpr int V = Elem<T>::kVec;
  const int64_t vecs = a.cols / V;     // the most body vectors a row can hold
  const int col_blocks = int((vecs + kBlock - 1) / kBlock);
  constexpr int U = FS_PW_ROWS_PER_TRIP;
  const int64_t row_groups_needed = (a.rows + U - 1) / U;
  const int64_t target_blocks = int64_t(cus) * FS_PW_BLOCKS_PER_CU;
  auto go = [&](auto kern, int64_t grid) {
    hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(kBlock), 0, s,
                       static_cast<const T*>(a.x), a.ld_x, static_cast<const T*>(a.bias),
                       static_cast<const T*>(a.res), a.ld_r, static_cast<T*>(a.y), a.ld_y,
                       a.rows, int(a.cols), a.scale, col_blocks);
    return hipGetLastError();
  };
  if (row_groups_needed < int64_t(cus) * 2) {
    const int64_t r1 = a.rows < target_blocks ? a.rows : target_blocks;
    return go(pointwise_shift_kernel<T, ACT, HAS_RES, 1>, r1 * col_blocks);
  }
  int64_t rg = target_blocks / col_blocks;
  if (rg < 1) rg = 1;
  if (rg > row_groups_needed) rg = row_groups_needed;
  return go(pointwise_shift_kernel<T, ACT, HAS_RES, U>, rg * col_blocks);
}

template <typename T, bool HAS_RES>
hipError_t by_act_shift(const PointwiseArgs& a, int cus, hipStream_t s) {
  switch (a.act) {
    case FS_ACT_GELU_ERF: return dispatch_shift<T, FS_ACT_GELU_ERF, HAS_RES>(a, cus, s);
    case FS_ACT_SIGMOID: return dispatch_shift<T, FS_ACT_SIGMOID, HAS_RES>(a, cus, s);
    case FS_ACT_RELU: return dispatch_shift<T, FS_ACT_RELU, HAS_RES>(a, cus, s);
    default: return dispatch_shift<T, FS_ACT_NONE, HAS_RES>(a, cus, s);
  }
}

template <typename T>
hipError_t by_res(const PointwiseArgs& a, int cus, hipStream_t s) {
  if (a.shifted)
    return a.res == nullptr ? by_act_shift<T, false>(a, cus, s) : by_act_shift<T, true>(a, cus, s);
  if (a.res == nullptr)
    return a.vec ? by_act<T, false, true>(a, cus, s) : by_act<T, false, false>(a, cus, s);
  return a.vec ? by_act<T, true, true>(a, cus, s) : by_act<T, true, false>(a, cus, s);
}

}  // namespace

hipError_t launch_pointwise(const PointwiseArgs& a, int cus, hipStream_t s) {
  return a.dtype == FS_BF16 ? by_res<uint16_t>(a, cus, s) : by_res<float>(a, cus, s);
}

}  // namespace fs
