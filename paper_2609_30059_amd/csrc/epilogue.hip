// GEMM epilogue with a row reduction, applied to a library GEMM's output C:
//
//   out[i] = reduce_j act((C[i, j] + bias[j]) * col_scale[j])
//
// KernelOPT Appendix A (Codegen prompt: keep the matmul a library call and
// fuse only its epilogue; Fusion Agent: reduction + pointwise).
//
// Design (gfx950).  (C + b) * s is evaluated as C * s + b * s (one FMA per
// element); for the sigmoid the factor -log2(e) is folded into both
// coefficients so that sigmoid = 1 / (1 + 2^u) costs one v_exp_f32, and the
// row kernels sum four sigmoids as one fraction with a single v_rcp_f32
// (epi_sum4): the transcendentals are quarter-rate, and inside a streaming
// workload that keeps the clock below its peak they, not HBM, would set the
// pace.  The per-column coefficients (s, b*s) are staged once per block
// in LDS; then every wave reduces whole rows on its own -- no block barrier
// in the row loop.  A wave reads its row in chunks of CH 16-byte vectors per
// lane and software-pipelines them: the loads of the next chunk (of this row
// or of its next row) are in flight while the current chunk is evaluated, so
// HBM traffic and the transcendental work overlap inside every wave.  Row r
// starts at chunk r mod (chunks per row), so waves running side by side read
// different offsets of their rows; blocks of 16 waves at 8 waves per SIMD
// keep 32 waves per CU.
//
// LDS layout: vector v = k*64 + lane of a row holds V columns; its V scale
// factors are H = V/4 float4s at index (k*H + h)*64 + lane, so each
// ds_read_b128 of a wave touches 64 consecutive float4s (no bank conflicts).
// The biases times scale use the same layout in a second array.
//
// Rows wider than the LDS staging capacity, or C that is not 16-byte
// aligned, take a block-per-row kernel that reads the coefficients through
// the cache.
#include <type_traits>

#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_EPI_ROTATE
#define FS_EPI_ROTATE 1
#endif
#ifndef FS_EPI_WPE
#define FS_EPI_WPE 8
#endif
#ifndef FS_EPI_NBUF
#define FS_EPI_NBUF 2   // chunk buffers of the staged kernel (prefetch depth + 1)
#endif
#ifndef FS_EPI_SIG4
#define FS_EPI_SIG4 1
#endif
#if FS_EPI_WPE > 0
#define FS_EPI_OCC __attribute__((amdgpu_waves_per_eu(FS_EPI_WPE, FS_EPI_WPE)))
#else
#define FS_EPI_OCC
#endif

namespace fs {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int ACT>
__device__ __forceinline__ float epi_act(float u) {
  if constexpr (ACT == FS_ACT_SIGMOID) {
    return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(u));   // u = -t*log2(e)
  } else if constexpr (ACT == FS_ACT_GELU_ERF) {
    return gelu_erf(u);
  } else if constexpr (ACT == FS_ACT_RELU) {
    return u < 0.f ? 0.f : u;   // a NaN stays NaN
  } else {
    return u;
  }
}

// act over four columns, summed.  For the sigmoid, with p = 1 + 2^u:
//   1/p0 + 1/p1 + 1/p2 + 1/p3 = n/d,  d = p0 p1 p2 p3,
// built one factor at a time (n' = n p + d, d' = d p), so four terms take
// one reciprocal instead of four.  u is capped at 31 so that d stays below
// 2^125 (a capped term counts 1/(1 + 2^31) < 4.7e-10 instead of its smaller
// exact value); the cap is a NaN-propagating minimum, so a NaN in C still
// reaches the row's result.
constexpr float kSigmoidCap = 31.f;

template <int ACT>
__device__ __forceinline__ float epi_sum4(const float* x, const f32x4& s4, const f32x4& b4) {
  if constexpr (ACT == FS_ACT_SIGMOID && FS_EPI_SIG4) {
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float u = __builtin_elementwise_minimum(fmaf(x[e], s4[e], b4[e]), kSigmoidCap);
      p[e] = 1.f + __builtin_amdgcn_exp2f(u);
    }
    float n = p[0] + p[1], d = p[0] * p[1];
    n = fmaf(n, p[2], d);
    d *= p[2];
    n = fmaf(n, p[3], d);
    d *= p[3];
    return n * __builtin_amdgcn_rcpf(d);
  } else {
    float t = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) t += epi_act<ACT>(fmaf(x[e], s4[e], b4[e]));
    return t;
  }
}

template <int ACT>
__device__ __forceinline__ float coef_sign() {
  return ACT == FS_ACT_SIGMOID ? -kLog2e : 1.f;
}

// Coefficients of the NVEC*64 vectors of a row into LDS (zeros past the row).
template <typename BT, int V, int H, int NVEC, int W, bool HB, bool HS>
__device__ __forceinline__ void fill_coef(f32x4* sc, f32x4* bs, const BT* __restrict__ bias,
                                          const float* __restrict__ col_scale, int nvec,
                                          float sgn) {
  // i enumerates (vector, half): vector vi = i / H, half h = i % H.  Every
  // load is issued before the first is used.
  constexpr int N = NVEC * 64 * H, NS = (N + 64 * W - 1) / (64 * W);
  float sv[NS][4], bv[NS][4];
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    const int i = threadIdx.x + t * 64 * W;
    const int vi = i / H, h = i % H;
    const int c0 = (i < N && vi < nvec ? vi : nvec - 1) * V + h * 4;   // clamped: in bounds
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sv[t][e] = HS ? col_scale[c0 + e] : 1.f;
      bv[t][e] = HB ? Elem<BT>::load1(bias + c0 + e) : 0.f;
    }
  }
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    const int i = threadIdx.x + t * 64 * W;
    const int vi = i / H, h = i % H;
    const int k = vi / 64, ln = vi % 64;
    const bool live = vi < nvec;
    f32x4 s4, b4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float s = sv[t][e] * sgn;
      s4[e] = live ? s : 0.f;
      b4[e] = live ? bv[t][e] * s : 0.f;
    }
    if (i < N) {
      sc[(k * H + h) * 64 + ln] = s4;
      bs[(k * H + h) * 64 + ln] = b4;
    }
  }
}

// NVEC: 16-byte vectors per lane per row (compile-time ceiling); CHMAX:
// vectors per pipelined chunk (at most NVEC); W: waves per block.
// FULL: the row fills every lane's NVEC slots (no clamps, no masks).
template <typename CT, typename BT, int ACT, int NVEC, int CHMAX, int W, bool FULL>
__global__ __launch_bounds__(64 * W) FS_EPI_OCC void epilogue_lds_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ col_scale, float* __restrict__ out, int64_t rows, int cols,
    int mean) {
  constexpr int V = Elem<CT>::kVec;    // columns per vector
  constexpr int H = V / 4;             // float4s of coefficients per vector
  constexpr int CH = CHMAX < NVEC ? CHMAX : NVEC;
  constexpr int NCH = NVEC / CH;
  static_assert(NVEC % CH == 0, "NVEC must be a multiple of CH");
  static_assert((NCH & (NCH - 1)) == 0, "the chunk count must be a power of two");
  extern __shared__ f32x4 lds_coef[];
  f32x4* sc = lds_coef;                       // [NVEC * H * 64]
  f32x4* bs = lds_coef + NVEC * H * 64;       // [NVEC * H * 64]

  const int nvec = cols / V;                  // vectors in a row
  const float sgn = coef_sign<ACT>();
  // the wave index is uniform: row and chunk arithmetic stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lane = threadIdx.x % 64;
  const int64_t stride = int64_t(gridDim.x) * W;
  int64_t row = int64_t(blockIdx.x) * W + wave;

  // raw chunks: CH vectors of 4 dwords each, in NB buffers: while chunk j is
  // evaluated, chunks j+1 .. j+NB-1 are in flight.  Loads are unconditional
  // (a lane past the row end re-reads the row's last vector, FULL rows have
  // none).  NB > 2 needs NCH % NB == 0, so that chunk j of every row sits in
  // buffer j % NB.
  constexpr int NB = (FS_EPI_NBUF > 2 && NCH % FS_EPI_NBUF == 0) ? FS_EPI_NBUF : 2;
  u32x4 buf[NB][CH];
  auto load_chunk = [&](u32x4 (&dst)[CH], int64_t r, int j, auto full) {
    const CT* cr = c + r * ld_c;
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int vi = (j * CH + q) * 64 + lane;
      dst[q] = ld128<true>(cr + (decltype(full)::value || vi < nvec ? vi : nvec - 1) * V);
    }
  };
  // Row r is walked starting at chunk r mod NCH (FS_EPI_ROTATE): waves that
  // run side by side then read different offsets of their rows instead of
  // the same offset of rows a fixed stride apart (which measured up to 1.6x
  // slower with one row per wave).
  auto rot_of = [&](int64_t r) { return FS_EPI_ROTATE ? int(r & (NCH - 1)) : 0; };
  int rot = rot_of(row);
  // the first NB-1 chunks are in flight while the coefficients are staged (a
  // wave without a row reads the last row and exits after the barrier)
#pragma unroll
  for (int i = 0; i + 1 < NB; ++i)
    load_chunk(buf[i], row < rows ? row : rows - 1, (rot + i) & (NCH - 1), std::false_type{});

  // stage (s, b*s): the null checks sit outside the loop so that each body is
  // branch-free and its loads are issued together
  if (bias) {
    if (col_scale) fill_coef<BT, V, H, NVEC, W, true, true>(sc, bs, bias, col_scale, nvec, sgn);
    else fill_coef<BT, V, H, NVEC, W, true, false>(sc, bs, bias, col_scale, nvec, sgn);
  } else {
    if (col_scale) fill_coef<BT, V, H, NVEC, W, false, true>(sc, bs, bias, col_scale, nvec, sgn);
    else fill_coef<BT, V, H, NVEC, W, false, false>(sc, bs, bias, col_scale, nvec, sgn);
  }
  __syncthreads();
  if (row >= rows) return;            // no barrier after this point

  const auto full = std::integral_constant<bool, FULL>{};
  {
    while (true) {
      float acc = 0.f;
      const int64_t next = row + stride;
      // the coefficients are re-read from LDS for every row: the opaque copy
      // of the lane index stops the compiler from hoisting 2*NVEC*H float4s
      // of loop-invariant LDS reads into registers (which would spill)
      int li = lane;
      asm volatile("" : "+v"(li));
      // the last NB-1 chunks prefetch the first chunks of the wave's next row;
      // on its last row every wave re-reads row 0 instead, which keeps the
      // loads free of branches and costs HBM traffic once per cache (a wave's
      // own streamed chunk is not kept in the cache: re-reading it measured
      // 3 % more traffic)
      const int64_t pre_row = next < rows ? next : 0;
      const int pre_chunk = next < rows ? rot_of(next) : 0;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int jp = j + NB - 1;                 // the chunk loaded now
        if (jp < NCH) load_chunk(buf[jp % NB], row, (jp + rot) & (NCH - 1), full);
        else load_chunk(buf[jp % NB], pre_row, (jp - NCH + pre_chunk) & (NCH - 1), full);
        const int pj = (j + rot) & (NCH - 1);
#pragma unroll
        for (int q = 0; q < CH; ++q) {
          const int vi = (pj * CH + q) * 64 + lane;
          float v[V];
          Elem<CT>::unpack(buf[j % NB][q], v);
          const int kq = pj * CH + q;
          float part = 0.f;
#pragma unroll
          for (int h = 0; h < H; ++h) {
            const f32x4 s4 = sc[(kq * H + h) * 64 + li];
            const f32x4 b4 = bs[(kq * H + h) * 64 + li];
            part += epi_sum4<ACT>(v + h * 4, s4, b4);
          }
          acc += (FULL || vi < nvec) ? part : 0.f;
        }
      }
      const SumP t = wave_allreduce(SumP{acc});
      if (lane == 0) out[row] = mean ? t.s / float(cols) : t.s;
      if (next >= rows) break;
      row = next;
      rot = rot_of(row);
      if constexpr (NB == 2 && NCH % 2 == 1) {
        // with an odd chunk count the next row's chunk 0 landed in buf[1]
#pragma unroll
        for (int q = 0; q < CH; ++q) buf[0][q] = buf[1][q];
      }
    }
  }
}

typedef float f32x2 __attribute__((ext_vector_type(2)));

// (s, b*s) pairs of every column into V planes: column j at plane j % V,
// index j / V (Q pairs per plane, zeros past the row).
template <typename BT, int V, int Q, int W, bool HB, bool HS>
__device__ __forceinline__ void fill_planes(f32x2* pl, const BT* __restrict__ bias,
                                            const float* __restrict__ col_scale, int cols,
                                            float sgn) {
  // every load is issued before the first is used
  constexpr int NS = (V * Q + 64 * W - 1) / (64 * W);
  float sv[NS], bv[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int i = threadIdx.x + k * 64 * W, r = i / Q, q = i % Q;
    const int j = q * V + r;
    const int jc = i < V * Q && j < cols ? j : cols - 1;   // clamped: always in bounds
    sv[k] = HS ? col_scale[jc] : 1.f;
    bv[k] = HB ? Elem<BT>::load1(bias + jc) : 0.f;
  }
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int i = threadIdx.x + k * 64 * W, r = i / Q, q = i % Q;
    const bool live = q * V + r < cols;
    const float sc = sv[k] * sgn;
    f32x2 pr;
    pr[0] = live ? sc : 0.f;
    pr[1] = live ? bv[k] * sc : 0.f;
    if (i < V * Q) pl[i] = pr;
  }
}

// Rows that are not whole 16-byte vectors (odd widths, odd row offsets) but
// span at least two, up to the staged widths: each row's aligned body, from
// its first 16-byte boundary to its last, is read 16 bytes at a time with the
// pipelining of epilogue_lds_kernel; its head and tail (at most V-1 elements
// each) go one per lane to the first lanes.  The body of a row starting h
// columns before a 16-byte boundary holds columns h + v*V + e, so element e
// of every lane's vector v lies in coefficient plane (h+e) % V at index
// v + (h+e) / V: 64 lanes read 64 consecutive pairs, whatever the row's h.
// WPE: waves per SIMD the register budget is sized for: 4 (one block per
// compute unit) where 8 would spill, i.e. from 16 bf16 vectors per lane.
template <typename CT, typename BT, int ACT, int NVEC, int CHMAX, int W, int WPE>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(WPE, WPE))) void
epilogue_shift_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ col_scale, float* __restrict__ out, int64_t rows, int cols,
    int mean) {
  constexpr int V = Elem<CT>::kVec;
  constexpr int Q = NVEC * 64 + 1;       // body vectors of a row, plus the carry
  constexpr int CH = CHMAX < NVEC ? CHMAX : NVEC;
  constexpr int NCH = NVEC / CH;
  static_assert(NVEC % CH == 0, "NVEC must be a multiple of CH");
  static_assert((NCH & (NCH - 1)) == 0, "the chunk count must be a power of two");
  extern __shared__ f32x2 lds_pl[];      // [V][Q]

  const float sgn = coef_sign<ACT>();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lane = threadIdx.x % 64;
  const int64_t stride = int64_t(gridDim.x) * W;
  int64_t row = int64_t(blockIdx.x) * W + wave;

  // h: columns before the row's first 16-byte boundary; nb: whole vectors
  // after it (>= 1 since cols >= 2V); the rest, cols - nb*V, are extras
  auto head_of = [&](int64_t r) {
    const int phase = int(reinterpret_cast<uintptr_t>(c + r * ld_c) & 15) / int(sizeof(CT));
    return (V - phase) & (V - 1);
  };
  u32x4 buf[2][CH];
  // ln: the lane index (per row, a copy the compiler cannot see through, so
  // that no per-lane offset is hoisted out of the row loop and kept live)
  auto load_chunk = [&](u32x4 (&dst)[CH], int64_t r, int hh, int nbb, int j, int ln) {
    const CT* cb = c + r * ld_c + hh;
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int vi = (j * CH + q) * 64 + ln;
      dst[q] = ld128<true>(cb + (vi < nbb ? vi : nbb - 1) * V);
    }
  };
  // a lane's extra column: lanes below h take the head, the next ones the
  // tail (column nb*V + lane); lanes past the extras re-read column 0
  auto extra_col = [&](int hh, int nbb, int ln) {
    const int nx = cols - nbb * V;
    return ln < nx ? (ln < hh ? ln : nbb * V + ln) : 0;
  };
  auto rot_of = [&](int64_t r) { return FS_EPI_ROTATE ? int(r & (NCH - 1)) : 0; };

  const int64_t first = row < rows ? row : rows - 1;
  int h = head_of(first);
  int nb = (cols - h) / V;
  int rot = rot_of(row);
  load_chunk(buf[0], first, h, nb, rot, lane);
  CT xraw = c[first * ld_c + extra_col(h, nb, lane)];

  if (bias) {
    if (col_scale) fill_planes<BT, V, Q, W, true, true>(lds_pl, bias, col_scale, cols, sgn);
    else fill_planes<BT, V, Q, W, true, false>(lds_pl, bias, col_scale, cols, sgn);
  } else {
    if (col_scale) fill_planes<BT, V, Q, W, false, true>(lds_pl, bias, col_scale, cols, sgn);
    else fill_planes<BT, V, Q, W, false, false>(lds_pl, bias, col_scale, cols, sgn);
  }
  __syncthreads();
  if (row >= rows) return;            // no barrier after this point

  while (true) {
    float acc = 0.f;
    const int64_t next = row + stride;
    int li = lane;
    asm volatile("" : "+v"(li));
    // element e of this row's vectors: plane (h+e) % V, index + (h+e) / V
    // (uniform offsets; the lane's addresses are formed again in every chunk
    // rather than kept live through the row)
    int off[V];
#pragma unroll
    for (int e = 0; e < V; ++e) off[e] = ((h + e) & (V - 1)) * Q + ((h + e) >= V ? 1 : 0);
    const int64_t pre_row = next < rows ? next : 0;
    const int ph = head_of(pre_row);
    const int pnb = (cols - ph) / V;
    const int pre_chunk = next < rows ? rot_of(next) : 0;
    CT xnext;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      if (j + 1 < NCH) {
        load_chunk(buf[(j + 1) & 1], row, h, nb, (j + 1 + rot) & (NCH - 1), li);
      } else {
        load_chunk(buf[(j + 1) & 1], pre_row, ph, pnb, pre_chunk, li);
        xnext = c[pre_row * ld_c + extra_col(ph, pnb, li)];
      }
      const int pj = (j + rot) & (NCH - 1);
      int lj = li;
      asm volatile("" : "+v"(lj));
#pragma unroll
      for (int q = 0; q < CH; ++q) {
        const int kq = (pj * CH + q) * 64;
        float v[V];
        Elem<CT>::unpack(buf[j & 1][q], v);
        float part = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) {
          const f32x2 pr = lds_pl[off[e] + lj + kq];
          part += epi_act<ACT>(fmaf(v[e], pr[0], pr[1]));
        }
        acc += kq + li < nb ? part : 0.f;
      }
    }
    {
      const int ce = extra_col(h, nb, li);
      const f32x2 pr = lds_pl[(ce & (V - 1)) * Q + ce / V];
      const float part = epi_act<ACT>(fmaf(raw_f32(xraw), pr[0], pr[1]));
      acc += li < cols - nb * V ? part : 0.f;
    }
    const SumP t = wave_allreduce(SumP{acc});
    if (lane == 0) out[row] = mean ? t.s / float(cols) : t.s;
    if (next >= rows) break;
    row = next;
    rot = rot_of(row);
    h = ph;
    nb = pnb;
    xraw = xnext;
    if constexpr (NCH % 2 == 1) {
#pragma unroll
      for (int q = 0; q < CH; ++q) buf[0][q] = buf[1][q];
    }
  }
}

// Rows the staged kernel does not take (wider than 16384 columns, or not
// whole 16-byte vectors): one block of 4 waves per row, coefficients through
// the cache.  Each thread keeps U vectors of the row in flight per trip
// (clamped loads, issued together) with one accumulator per vector slot;
// with VEC and coef_vec the coefficients are read as vectors too.
template <typename CT, typename BT, int ACT, bool VEC>
__global__ __launch_bounds__(256) void epilogue_wide_kernel(
    const CT* __restrict__ c, int64_t ld_c, const BT* __restrict__ bias,
    const float* __restrict__ col_scale, float* __restrict__ out, int64_t rows, int64_t cols,
    int mean, int coef_vec) {
  constexpr int V = VEC ? Elem<CT>::kVec : 1;
  constexpr int U = VEC ? 4 : 8;
  __shared__ SumP lds[2][4];
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const float sgn = coef_sign<ACT>();
  const int64_t nv = (cols + V - 1) / V;   // VEC rows are whole vectors
  int parity = 0;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const CT* cr = c + row * ld_c;
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = 0.f;
    for (int64_t v0 = tid; v0 < nv; v0 += 256 * U) {
      Raw<CT, V> rc[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t v = v0 + u * 256;
        rc[u].load(cr + (v < nv ? v : nv - 1) * V);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t v = v0 + u * 256;
        const int64_t j0 = (v < nv ? v : nv - 1) * V;
        float cv[V], sv[V], bv[V];
        rc[u].unpack(cv);
        if (col_scale) {
          if (VEC && coef_vec) {
            ldv<float, V, false>(col_scale + j0, sv);
          } else {
#pragma unroll
            for (int i = 0; i < V; ++i) sv[i] = col_scale[j0 + i];
          }
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i) sv[i] = 1.f;
        }
        if (bias) {
          if (VEC && coef_vec) {
            ldv<BT, V, false>(bias + j0, bv);
          } else {
#pragma unroll
            for (int i = 0; i < V; ++i) bv[i] = Elem<BT>::load1(bias + j0 + i);
          }
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i) bv[i] = 0.f;
        }
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const float s = sv[i] * sgn;
          part += epi_act<ACT>(fmaf(cv[i], s, bv[i] * s));
        }
        acc[u] += v < nv ? part : 0.f;
      }
    }
    float tot = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) tot += acc[u];
    const SumP t = group_allreduce<4>(SumP{tot}, lds[parity], wave, lane);
    parity ^= 1;
    if (tid == 0) out[row] = mean ? t.s / float(cols) : t.s;
  }
}

#ifndef FS_EPI_WAVES
#define FS_EPI_WAVES 16
#endif
#ifndef FS_EPI_CHUNK
#define FS_EPI_CHUNK 2   // vectors per pipelined chunk
#endif
#ifndef FS_EPI_CHUNK_FULL
#define FS_EPI_CHUNK_FULL 4   // the same for rows that fill 2..16 vectors per lane
#endif
#ifndef FS_EPI_BLOCKS_PER_CU
#define FS_EPI_BLOCKS_PER_CU 2
#endif
constexpr int kLdsW = FS_EPI_WAVES;    // waves per block of the staged kernel
constexpr int kLdsCH = FS_EPI_CHUNK;   // vectors per pipelined chunk
// Full rows of up to 16 vectors per lane read 4-vector chunks: twice the
// bytes in flight per wave.  Between other bandwidth-bound kernels the
// 2-vector form of the 8192-column epilogue ran either at 22 us or, in many
// runs for most of its launches, at 28 us with its waves resident longer at
// an unchanged clock; the 4-vector form stays near 23 us.  Wider or partial
// rows keep 2-vector chunks (4 would spill at 64 VGPRs).
template <int NV>
constexpr int kLdsChFull = NV <= 16 ? FS_EPI_CHUNK_FULL : FS_EPI_CHUNK;

template <typename CT, typename BT, int ACT>
hipError_t dispatch(const EpilogueArgs& a, int cus, hipStream_t s) {
  constexpr int V = Elem<CT>::kVec;
  const int mean = a.reduce == FS_REDUCE_MEAN;
  const int64_t per_lane = (a.cols / V + 63) / 64;
  auto staged = [&](auto kern, int nvec) {
    const size_t lds = size_t(2) * nvec * (V / 4) * 64 * 16;
    int64_t want = (a.rows + kLdsW - 1) / kLdsW;
    // tables above 80 KiB leave room for one block per compute unit
    int64_t cap = int64_t(cus) * (lds > 80 * 1024 ? 1 : FS_EPI_BLOCKS_PER_CU);
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * kLdsW), lds, s, static_cast<const CT*>(a.c),
                       a.ld_c, static_cast<const BT*>(a.bias), a.col_scale, a.out, a.rows,
                       int(a.cols), mean);
    return hipGetLastError();
  };
  if (a.vec && a.cols > 0) {
    const int64_t nvec = a.cols / V;
#define FS_EPI_RUNG(NV)                                                                 \
  if (per_lane <= NV)                                                                    \
    return nvec == int64_t(NV) * 64                                                      \
               ? staged(epilogue_lds_kernel<CT, BT, ACT, NV, kLdsChFull<NV>, kLdsW, true>, NV) \
               : staged(epilogue_lds_kernel<CT, BT, ACT, NV, kLdsCH, kLdsW, false>, NV);
    FS_EPI_RUNG(2)
    FS_EPI_RUNG(4)
    FS_EPI_RUNG(8)
    FS_EPI_RUNG(16)
    FS_EPI_RUNG(32)
    if constexpr (V == 4) { FS_EPI_RUNG(64) }
#undef FS_EPI_RUNG
  }
  if (a.shifted) {
    const int64_t body = a.cols / V;   // at most this many vectors in a row's body
    auto shift = [&](auto kern, int nvec, int wpe) {
      const size_t lds = size_t(V) * (nvec * 64 + 1) * 8;
      int64_t want = (a.rows + kLdsW - 1) / kLdsW;
      int64_t cap = int64_t(cus) * (wpe == 4 ? 1 : FS_EPI_BLOCKS_PER_CU);
      int grid = int(want < cap ? want : cap);
      if (grid < 1) grid = 1;
      hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * kLdsW), lds, s, static_cast<const CT*>(a.c),
                         a.ld_c, static_cast<const BT*>(a.bias), a.col_scale, a.out, a.rows,
                         int(a.cols), mean);
      return hipGetLastError();
    };
#define FS_EPI_SHIFT_RUNG(NV)                                                                   \
  if (body <= int64_t(NV) * 64) {                                                          \
    constexpr int wpe = V * NV >= 128 ? 4 : 8;                                             \
    return shift(epilogue_shift_kernel<CT, BT, ACT, NV, kLdsCH, kLdsW, wpe>, NV, wpe);     \
  }
    FS_EPI_SHIFT_RUNG(2)
    FS_EPI_SHIFT_RUNG(4)
    FS_EPI_SHIFT_RUNG(8)
    FS_EPI_SHIFT_RUNG(16)
    FS_EPI_SHIFT_RUNG(32)
    if constexpr (V == 4) { FS_EPI_SHIFT_RUNG(64) }
#undef FS_EPI_SHIFT_RUNG
  }
  int64_t grid = a.rows < int64_t(cus) * 8 ? a.rows : int64_t(cus) * 8;
  if (grid < 1) grid = 1;
  auto wide = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(256), 0, s, static_cast<const CT*>(a.c),
                       a.ld_c, static_cast<const BT*>(a.bias), a.col_scale, a.out, a.rows, a.cols,
                       mean, int(a.coef_vec));
    return hipGetLastError();
  };
  return a.vec && a.cols > 0 ? wide(epilogue_wide_kernel<CT, BT, ACT, true>)
                             : wide(epilogue_wide_kernel<CT, BT, ACT, false>);
}

template <typename CT, typename BT>
hipError_t by_act(const EpilogueArgs& a, int cus, hipStream_t s) {
  switch (a.act) {
    case FS_ACT_SIGMOID: return dispatch<CT, BT, FS_ACT_SIGMOID>(a, cus, s);
    case FS_ACT_GELU_ERF: return dispatch<CT, BT, FS_ACT_GELU_ERF>(a, cus, s);
    case FS_ACT_RELU: return dispatch<CT, BT, FS_ACT_RELU>(a, cus, s);
    default: return dispatch<CT, BT, FS_ACT_NONE>(a, cus, s);
  }
}

template <typename CT>
hipError_t by_bias(const EpilogueArgs& a, int cus, hipStream_t s) {
  return a.bias_dtype == FS_BF16 ? by_act<CT, uint16_t>(a, cus, s) : by_act<CT, float>(a, cus, s);
}

}  // namespace

hipError_t launch_epilogue(const EpilogueArgs& a, int cus, hipStream_t s) {
  return a.c_dtype == FS_BF16 ? by_bias<uint16_t>(a, cus, s) : by_bias<float>(a, cus, s);
}

}  // namespace fs
