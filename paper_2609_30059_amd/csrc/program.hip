// Fused pointwise program: y = op_n(... op_1(x) ...), the operations of
// fs_op_code applied in fp32 registers, one load of every input and one
// store of y.
//
// KernelOPT merges adjacent fusible elementwise kernels of a compiled graph
// into one (Section 3; its example group is a multiply, a hardtanh and a
// GELU after a linear layer) and fuses pointwise chains and activations
// with their bias (Appendix A, Fusion Agent).  The fixed chain of
// pointwise.hip covers act(x * s + b) + r; this kernel takes the group as
// data, so one compiled kernel serves every such group.
//
// Design (gfx950): the launch shape of the pointwise chain -- a block of 256
// threads owns a slab of 256 column vectors (16 bytes each) and walks down
// the rows, U rows per trip with all their loads issued before any use; the
// column vectors (bias, col) stay in registers.  The program sits in the
// kernel's argument block and is read with scalar loads: the operation loop
// is uniform across the wave and runs once per group of rows of the trip
// holding 16 values per lane (only they are live across it, which keeps the
// register count low), so each operation costs a scalar load, a few compares
// and branches per 16 values, and their arithmetic.
#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_PROG_ROWS_PER_TRIP
#define FS_PROG_ROWS_PER_TRIP 4
#endif
#ifndef FS_PROG_BLOCKS_PER_CU
#define FS_PROG_BLOCKS_PER_CU 16
#endif

namespace fs {
namespace {

constexpr int kBlock = 256;

// tanh(v) = sign(v) (1 - e) / (1 + e) with e = exp(-2 |v|) in (0, 1]: no
// overflow for any v, +-1 at +-inf, NaN for NaN; absolute error a few units
// of 2^-24 (relative error larger only where |tanh v| is below about 1e-3)
__device__ __forceinline__ float tanh_fn(float v) {
  const float e = __builtin_amdgcn_exp2f(-2.f * kLog2e * fabsf(v));
  return copysignf((1.f - e) * __builtin_amdgcn_rcpf(1.f + e), v);
}

// Applies the program to the values v[G][W] in place, in order.  bias_at,
// col_at and res_at give the bias, column and residual operand of value
// (g, i); residual operations are compiled in only when HAS_RES (the C ABI
// passes no residual to a program without them).
template <bool HAS_RES, int G, int W, typename FB, typename FC, typename FR>
__device__ __forceinline__ void run_program(const Program& prog, float (&v)[G][W], FB bias_at,
                                            FC col_at, FR res_at) {
  for (int k = 0; k < prog.n; ++k) {
    const int code = prog.code[k];
    const float pa = prog.a[k], pb = prog.b[k];
#define FS_EACH(expr)                               \
  _Pragma("unroll") for (int g = 0; g < G; ++g)     \
    _Pragma("unroll") for (int i = 0; i < W; ++i) { \
      const float t = v[g][i];                      \
      v[g][i] = (expr);                             \
    }
    switch (code) {
      case FS_OP_SCALE: FS_EACH(t * pa) break;
      case FS_OP_SHIFT: FS_EACH(t + pa) break;
      case FS_OP_ADD_BIAS: FS_EACH(t + bias_at(g, i)) break;
      case FS_OP_MUL_COLUMN: FS_EACH(t * col_at(g, i)) break;
      case FS_OP_ADD_RESIDUAL:
        if constexpr (HAS_RES) { FS_EACH(t + res_at(g, i)) }
        break;
      case FS_OP_MUL_RESIDUAL:
        if constexpr (HAS_RES) { FS_EACH(t * res_at(g, i)) }
        break;
      // clamp and ReLU by comparisons, so that a NaN stays NaN (fminf and
      // fmaxf would return the other operand)
      case FS_OP_CLAMP: FS_EACH(t < pa ? pa : (t > pb ? pb : t)) break;
      case FS_OP_GELU_ERF: FS_EACH(gelu_erf(t)) break;
      case FS_OP_SIGMOID: FS_EACH(sigmoid(t)) break;
      case FS_OP_RELU: FS_EACH(t < 0.f ? 0.f : t) break;
      case FS_OP_TANH: FS_EACH(tanh_fn(t)) break;
      case FS_OP_SILU: FS_EACH(t * sigmoid(t)) break;
      default: FS_EACH(t >= 0.f ? t : pa * t) break;   // FS_OP_LEAKY_RELU
    }
#undef FS_EACH
  }
}

template <typename T, bool HAS_RES, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void program_kernel(
    const T* x, int64_t ld_x, const T* __restrict__ bias, const T* __restrict__ col, const T* res,
    int64_t ld_r, T* y, int64_t ld_y, int64_t rows, int cols, int col_blocks, Program prog) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  constexpr int RG = 16 / V < U ? (16 / V > 0 ? 16 / V : 1) : U;   // rows per operation dispatch
  static_assert(U % RG == 0, "row groups split the trip");
  const int cb = blockIdx.x % col_blocks;
  const int64_t rg = blockIdx.x / col_blocks;
  const int64_t nrg = gridDim.x / col_blocks;
  const int c0 = (cb * kBlock + threadIdx.x) * V;
  if (c0 >= cols) return;               // no barriers below: early exit is safe

  float bv[V], cv[V];
#pragma unroll
  for (int i = 0; i < V; ++i) bv[i] = cv[i] = 0.f;
  if (bias) {
    Raw<T, V> rb;
    rb.template load<false>(bias + c0);
    rb.unpack(bv);
  }
  if (col) {
    Raw<T, V> rc;
    rc.template load<false>(col + c0);
    rc.unpack(cv);
  }

  for (int64_t r0 = rg * U; r0 < rows; r0 += nrg * U) {
    // all loads of the trip first; rows past the end re-read the last row
    // (in bounds) and are not stored
    Raw<T, V> rx[U], rr[HAS_RES ? U : 1];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = r0 + u < rows ? r0 + u : rows - 1;
      rx[u].load(x + r * ld_x + c0);
      if constexpr (HAS_RES) rr[u].load(res + r * ld_r + c0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // the trip's rows go through the program in groups of RG rows, RG x V =
    // 16 values per lane (2 bf16 rows, 4 fp32 rows): each operation's
    // dispatch is shared by 16 values while only those stay live across the
    // operation loop
#pragma unroll
    for (int u0 = 0; u0 < U; u0 += RG) {
      float v[RG][V], rv[HAS_RES ? RG : 1][V];
#pragma unroll
      for (int g = 0; g < RG; ++g) {
        rx[u0 + g].unpack(v[g]);
        if constexpr (HAS_RES) rr[u0 + g].unpack(rv[g]);
      }
      run_program<HAS_RES>(
          prog, v, [&](int, int i) { return bv[i]; }, [&](int, int i) { return cv[i]; },
          [&](int g, int i) { return rv[HAS_RES ? g : 0][i]; });
#pragma unroll
      for (int g = 0; g < RG; ++g)
        if (r0 + u0 + g < rows) stv<T, V>(y + (r0 + u0 + g) * ld_y + c0, v[g]);
    }
  }
}

// Rows that are not whole 16-byte vectors but whose x, residual and y start
// every row at one offset within a 16-byte unit: each row's aligned body,
// from its first 16-byte boundary to its last, moves 16 bytes at a time, and
// thread t of column block cb owns body vector cb*kBlock + t of every row.
// A row starting h columns before a 16-byte boundary puts element e of body
// vector v at column h + v*V + e, so the block stages the bias and the
// column vector of its columns in LDS in V planes each (column j at plane
// j % V, index j / V, one spare index for the vector that crosses into the
// next block's columns): element e reads plane (h+e) % V at index
// t + (h+e) / V, consecutive across the lanes whatever h is, and only where
// the program reads it.  The head and tail of each row (at most V-1
// elements each) go one per lane to wave 0 of column block 0, whose loads
// are issued with the body's and whose operands come from global memory.
template <typename T, bool HAS_RES, int U>
__global__ __launch_bounds__(kBlock) void program_shift_kernel(
    const T* x, int64_t ld_x, const T* __restrict__ bias, const T* __restrict__ col, const T* res,
    int64_t ld_r, T* y, int64_t ld_y, int64_t rows, int cols, int col_blocks, Program prog) {
  constexpr int V = Elem<T>::kVec;
  constexpr int RG = 16 / V < U ? 16 / V : U;   // rows per operation dispatch
  static_assert(U % RG == 0, "row groups split the trip");
  constexpr int Q = kBlock + 1;                 // the block's vectors, plus the carry
  extern __shared__ float tab[];                // [bias planes][column planes], each V x Q
  float* const tb = tab;
  float* const tc = tab + (bias != nullptr ? V * Q : 0);
  const int cb = blockIdx.x % col_blocks;
  const int64_t rg = blockIdx.x / col_blocks;
  const int64_t nrg = gridDim.x / col_blocks;
  const int tid = threadIdx.x;
  const int v = cb * kBlock + tid;              // the thread's body vector
  constexpr int NS = (V * Q + kBlock - 1) / kBlock;
  auto stage = [&](const T* src, float* dst) {
    // every staging load issued before the first is used
    float st[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int i = tid + k * kBlock, pl = i / Q, q = i % Q;
      const int j = (cb * kBlock + q) * V + pl;
      st[k] = Elem<T>::load1(src + (i < V * Q && j < cols ? j : 0));
    }
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int i = tid + k * kBlock, pl = i / Q, q = i % Q;
      const int j = (cb * kBlock + q) * V + pl;
      if (i < V * Q) dst[i] = j < cols ? st[k] : 0.f;
    }
  };
  if (bias != nullptr) stage(bias, tb);         // uniform over the block
  if (col != nullptr) stage(col, tc);
  __syncthreads();
  const bool edge = cb == 0 && tid < 64;        // uniform per wave
  if (v >= cols / V && !edge) return;           // no barriers below

  for (int64_t r0 = rg * U; r0 < rows; r0 += nrg * U) {
    Raw<T, V> rx[U], rr[HAS_RES ? U : 1];
    int hh[U], nb[U];
    T ex[U], er[HAS_RES ? U : 1];
    float eb[U], ec[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // rows past the end re-read the last row (in bounds) and are not stored
      const int64_t r = r0 + u < rows ? r0 + u : rows - 1;
      const int phase = int(reinterpret_cast<uintptr_t>(x + r * ld_x) & 15) / int(sizeof(T));
      hh[u] = (V - phase) & (V - 1);
      nb[u] = (cols - hh[u]) / V;               // >= 1: rows span at least two vectors
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
        eb[u] = bias != nullptr ? Elem<T>::load1(bias + ce) : 0.f;
        ec[u] = col != nullptr ? Elem<T>::load1(col + ce) : 0.f;
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u0 = 0; u0 < U; u0 += RG) {
      float w[RG][V], rv[HAS_RES ? RG : 1][V];
#pragma unroll
      for (int g = 0; g < RG; ++g) {
        rx[u0 + g].unpack(w[g]);
        if constexpr (HAS_RES) rr[u0 + g].unpack(rv[g]);
      }
      // element i of row u0 + g's body vector sits in plane (h+i) % V at
      // index tid + (h+i) / V: lo + i*Q while h+i < V, hi + i*Q from there
      // (i*Q folds into the LDS read's offset)
      int lo[RG], hi[RG], cut[RG];
#pragma unroll
      for (int g = 0; g < RG; ++g) {
        lo[g] = hh[u0 + g] * Q + tid;
        hi[g] = lo[g] - (V * Q - 1);
        cut[g] = V - hh[u0 + g];
      }
      auto at = [&](int g, int i) { return (i < cut[g] ? lo[g] : hi[g]) + i * Q; };
      run_program<HAS_RES>(
          prog, w, [&](int g, int i) { return tb[at(g, i)]; },
          [&](int g, int i) { return tc[at(g, i)]; },
          [&](int g, int i) { return rv[HAS_RES ? g : 0][i]; });
#pragma unroll
      for (int g = 0; g < RG; ++g)
        if (r0 + u0 + g < rows && v < nb[u0 + g])
          stv<T, V>(y + (r0 + u0 + g) * ld_y + hh[u0 + g] + v * V, w[g]);
    }
    if (edge) {
      float e[U][1];
#pragma unroll
      for (int u = 0; u < U; ++u) e[u][0] = raw_f32(ex[u]);
      run_program<HAS_RES>(
          prog, e, [&](int g, int) { return eb[g]; }, [&](int g, int) { return ec[g]; },
          [&](int g, int) { return HAS_RES ? raw_f32(er[HAS_RES ? g : 0]) : 0.f; });
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int nx = cols - nb[u] * V;
        if (r0 + u < rows && tid < nx) {
          const int ce = tid < hh[u] ? tid : nb[u] * V + tid;
          Elem<T>::store1(y + (r0 + u) * ld_y + ce, e[u][0]);
        }
      }
    }
  }
}

template <typename T, bool HAS_RES, bool VEC>
hipError_t dispatch(const ProgramArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  const int64_t vecs = (a.cols + V - 1) / V;
  const int col_blocks = int((vecs + kBlock - 1) / kBlock);
  const int64_t target_blocks = int64_t(cus) * FS_PROG_BLOCKS_PER_CU;
  auto go = [&](auto kern, int64_t grid) {
    hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(kBlock), 0, s, static_cast<const T*>(a.x),
                       a.ld_x, static_cast<const T*>(a.bias), static_cast<const T*>(a.col),
                       static_cast<const T*>(a.res), a.ld_r, static_cast<T*>(a.y), a.ld_y, a.rows,
                       int(a.cols), col_blocks, a.prog);
    return hipGetLastError();
  };
  constexpr int U = FS_PROG_ROWS_PER_TRIP;
  const int64_t row_groups_needed = (a.rows + U - 1) / U;
  if (row_groups_needed < int64_t(cus) * 2) {
    // small problem: one row per trip, as many blocks as rows (up to the target)
    const int64_t r1 = a.rows < target_blocks ? a.rows : target_blocks;
    return go(program_kernel<T, HAS_RES, VEC, 1>, r1 * col_blocks);
  }
  int64_t rg = target_blocks / col_blocks;
  if (rg < 1) rg = 1;
  if (rg > row_groups_needed) rg = row_groups_needed;
  return go(program_kernel<T, HAS_RES, VEC, U>, rg * col_blocks);
}

template <typename T, bool HAS_RES>
hipError_t dispatch_shift(const ProgramArgs& a, int cus, hipStream_t s) {
  constexpr int V = Elem<T>::kVec;
  const int64_t vecs = a.cols / V;     // the most body vectors a row can hold
  const int col_blocks = int((vecs + kBlock - 1) / kBlock);
  const int64_t target_blocks = int64_t(cus) * FS_PROG_BLOCKS_PER_CU;
  const size_t lds = size_t((a.bias ? 1 : 0) + (a.col ? 1 : 0)) * V * (kBlock + 1) * sizeof(float);
  auto go = [&](auto kern, int64_t grid) {
    hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(kBlock), lds, s,
                       static_cast<const T*>(a.x), a.ld_x, static_cast<const T*>(a.bias),
                       static_cast<const T*>(a.col), static_cast<const T*>(a.res), a.ld_r,
                       static_cast<T*>(a.y), a.ld_y, a.rows, int(a.cols), col_blocks, a.prog);
    return hipGetLastError();
  };
  constexpr int U = FS_PROG_ROWS_PER_TRIP;
  const int64_t row_groups_needed = (a.rows + U - 1) / U;
  if (row_groups_needed < int64_t(cus) * 2) {
    const int64_t r1 = a.rows < target_blocks ? a.rows : target_blocks;
    return go(program_shift_kernel<T, HAS_RES, 1>, r1 * col_blocks);
  }
  int64_t rg = target_blocks / col_blocks;
  if (rg < 1) rg = 1;
  if (rg > row_groups_needed) rg = row_groups_needed;
  return go(program_shift_kernel<T, HAS_RES, U>, rg * col_blocks);
}

template <typename T>
hipError_t by_res(const ProgramArgs& a, int cus, hipStream_t s) {
  if (a.shifted)
    return a.res ? dispatch_shift<T, true>(a, cus, s) : dispatch_shift<T, false>(a, cus, s);
  if (a.res)
    return a.vec ? dispatch<T, true, true>(a, cus, s) : dispatch<T, true, false>(a, cus, s);
  return a.vec ? dispatch<T, false, true>(a, cus, s) : dispatch<T, false, false>(a, cus, s);
}

}  // namespace

hipError_t launch_program(const ProgramArgs& a, int cus, hipStream_t s) {
  return a.dtype == FS_BF16 ? by_res<uint16_t>(a, cus, s) : by_res<float>(a, cus, s);
}

}  // namespace fs
