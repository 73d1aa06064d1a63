// LayerNorm (and RMSNorm) fused with the residual add.
//
// h = x + residual; y = (h - mean) / sqrt(var + eps) * gamma + beta;
// residual_out = h -- KernelOPT Appendix A (Fusion Agent: normalisation
// fusion, residual + norm in one memory pass; Codegen prompt: single-pass
// LayerNorm).
//
// Design (gfx950): one row per group of W wave64s, EPT elements per thread
// held in registers: x and residual are read from HBM once, residual_out and
// y written once.  The statistics are exact two-pass values over the
// register-resident row -- an all-reduce of sum(h) gives the mean, then an
// all-reduce of sum((h - mean)^2) the biased variance -- so there is no
// E[h^2] - mean^2 cancellation and no second HBM pass.  Both all-reduces are
// plain sums, which fold into DPP adds.  RMSNorm (y = h / sqrt(mean(h^2) +
// eps) * gamma, the RMS form of the same normalisation fusion) shares the
// kernel with a single all-reduce of sum(h^2) and no mean.
#include "device_common.hpp"
#include "launch.hpp"

// Build-time tuning: rows of at least FS_LN_SPLIT_COLS columns use at least
// FS_LN_MIN_WAVES waves per row; one-wave rows are batched to about
// FS_LN_BATCH_ELEMS elements per lane per trip; the grid holds at most
// FS_LN_GRID_SCALE/4 times the per-variant blocks-per-CU figure.
#ifndef FS_LN_WAVE_PATH
#define FS_LN_WAVE_PATH 1   // lean one-wave kernel for rows that fill a wave's slots exactly
#endif
#ifndef FS_LN_FULL_PATH
#define FS_LN_FULL_PATH 1   // mask-free code for rows that fill every lane's slots
#endif
#ifndef FS_LN_MIN_WAVES
#define FS_LN_MIN_WAVES 2
#endif
#ifndef FS_LN_SPLIT_COLS
#define FS_LN_SPLIT_COLS 2048
#endif
#ifndef FS_LN_BATCH_ELEMS
#define FS_LN_BATCH_ELEMS 16
#endif
#ifndef FS_LN_CACHE_REGS
#define FS_LN_CACHE_REGS 32   // row-cache elements per lane held in registers
#endif
#ifndef FS_LN_CACHE_GB_AHEAD
#define FS_LN_CACHE_GB_AHEAD 1   // slots of gamma/beta loads in flight ahead in the row cache's pass 2
#endif
#ifndef FS_LN_ELEMENTWISE_REG_COLS
#define FS_LN_ELEMENTWISE_REG_COLS 8192   // widest element-wise row on the register rungs
#endif
#ifndef FS_LN_ELEMENTWISE_CACHE_COLS
#define FS_LN_ELEMENTWISE_CACHE_COLS 32768   // element-wise rows take the row cache past this
#endif
#ifndef FS_LN_CACHE_ELEMENTWISE
#define FS_LN_CACHE_ELEMENTWISE 1   // row cache also for rows of element-wise loads
#endif
#ifndef FS_LN_CACHE_AHEAD
#define FS_LN_CACHE_AHEAD 3   // slot groups of loads in flight ahead in the row cache's pass 1
#endif
#ifndef FS_LN_CACHE_GROUP_WORDS
#define FS_LN_CACHE_GROUP_WORDS 8   // raw load registers per slot group of the row cache
#endif
#ifndef FS_LN_STREAM_WAVES
#define FS_LN_STREAM_WAVES 8   // waves per row of the streamed kernel
#endif
#ifndef FS_LN_STREAM_BPC
#define FS_LN_STREAM_BPC 4     // its blocks per compute unit
#endif
#ifndef FS_LN_GRID_SCALE
#define FS_LN_GRID_SCALE 16
#endif

// rows that share a 16-byte phase take the register rungs up to this many
// columns (their LDS table of (gamma, beta) pairs grows with the rung)
#ifndef FS_LN_SHIFT_REG_COLS
#define FS_LN_SHIFT_REG_COLS 16384
#endif

namespace fs {
namespace {

// (gamma, beta) of one column as staged in LDS: two bf16 bit patterns in one
// dword (exact), or two floats
template <typename T> struct AffinePair;
template <> struct AffinePair<uint16_t> {
  using type = uint32_t;
  __device__ __forceinline__ static type make(uint16_t g, uint16_t b) { return uint32_t(g) | (uint32_t(b) << 16); }
  __device__ __forceinline__ static float gamma(type p) { return __uint_as_float(p << 16); }
  __device__ __forceinline__ static float beta(type p) { return __uint_as_float(p & 0xffff0000u); }
};
template <> struct AffinePair<float> {
  typedef float type __attribute__((ext_vector_type(2)));
  __device__ __forceinline__ static type make(float g, float b) { type p; p[0] = g; p[1] = b; return p; }
  __device__ __forceinline__ static float gamma(type p) { return p[0]; }
  __device__ __forceinline__ static float beta(type p) { return p[1]; }
};

// W waves per row, EPT elements per thread, G row groups per block (W == 1
// only), R rows per group per trip: narrow rows are batched so that a wave
// keeps R rows of loads in flight and reduces them with one shuffle sequence.
// SHIFT: rows that are not whole 16-byte vectors but whose x, residual, y and
// residual_out start every row at one offset within a 16-byte unit.  The
// threads' vectors tile each row's aligned body, from its first 16-byte
// boundary (h columns in) to its last; the head and tail (at most V-1 columns
// each) are one extra element for each of the group's first lanes.  gamma and
// beta are staged once per block in LDS as (gamma, beta) pairs in V planes,
// column j at plane j % V, index j / V: element e of body vector v (column
// h + v*V + e) reads plane (h+e) % V at index v + (h+e) / V, consecutive
// across the lanes whatever h is.
template <typename T, bool HAS_RES, bool RMS, int W, int EPT, bool VEC, bool SHIFT, int G, int R>
__global__ __launch_bounds__(64 * W * G) void layernorm_kernel(
    const T* __restrict__ x, int64_t ld_x, const T* __restrict__ res, int64_t ld_r,
    const T* __restrict__ gamma, const T* __restrict__ beta, T* y, int64_t ld_y, T* res_out,
    int64_t ld_ro, int64_t rows, int cols, float eps) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC || SHIFT ? Elem<T>::kVec : 1;
  constexpr int NV = EPT / V;
  using AP = AffinePair<T>;
  using Pair = typename AP::type;
  constexpr int Q = NV * kThreads + 1;     // SHIFT: pairs per plane
  // gamma and beta stay in registers for the whole kernel when they fit
  // (element-wise loads hold one value per register, so only small rungs
  // keep them); wider rows re-read them (cache-resident) after each trip's
  // statistics
  constexpr bool kAffineResident = !SHIFT && (VEC ? EPT <= 32 : EPT <= 8);
  static_assert(EPT % V == 0, "EPT must be a multiple of the vector width");
  // one LDS fold area and one barrier sequence per block: rows wider than a
  // wave take the whole block (the row loop is then uniform across it)
  static_assert(W == 1 || G == 1, "multi-wave rows use one row group per block");
  using P = Multi<SumP, R>;
  __shared__ P lds[2][W];

  const int tid = threadIdx.x % kThreads;
  const int wave = tid / 64, lane = tid % 64;
  const int g = __builtin_amdgcn_readfirstlane(threadIdx.x / kThreads);   // wave-uniform
  int parity = 0;

  // out-of-row vectors read the last vector of the row (an in-bounds address)
  // and are masked
  const int clast = cols - V;
  const float inv_cols = 1.f / float(cols);
  // rows that fill every slot of every lane need no masking (uniform)
  const bool full = !SHIFT && FS_LN_FULL_PATH && cols == kThreads * EPT;
  const bool affine = FS_LN_FULL_PATH && gamma != nullptr && (RMS || beta != nullptr);

  Raw<T, V> rg[NV], rb[NV];
  auto load_affine = [&]() {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c0 = (k * kThreads + tid) * V;
      const int cl = c0 < cols ? c0 : clast;
      if (gamma) rg[k].template load<false>(gamma + cl);
      if (beta) rb[k].template load<false>(beta + cl);
    }
  };

  if constexpr (kAffineResident) load_affine();
  extern __shared__ unsigned char ln_dyn[];
  Pair* pl = reinterpret_cast<Pair*>(ln_dyn);   // SHIFT: [V][Q]
  if constexpr (SHIFT) {
    // every staging load is issued before the first is used; stand-in
    // pointers keep them unconditional (1 and 0 replace what is absent)
    constexpr int kAll = 64 * W * G, NS = (V * Q + kAll - 1) / kAll;
    const T* gs = gamma ? gamma : x;
    const T* bs = beta ? beta : x;
    T gv[NS], bv[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int i = int(threadIdx.x) + t * kAll, q = i % Q;
      const int j = q * V + i / Q;
      const int jc = i < V * Q && j < cols ? j : 0;
      gv[t] = gs[jc];
      bv[t] = bs[jc];
    }
    const T one = std::is_same<T, float>::value ? T(1.f) : T(0x3F80), zero = T(0);
#pragma unroll
    for (int t = 0; t < NS; ++t) {
      const int i = int(threadIdx.x) + t * kAll, q = i % Q;
      const bool live = q * V + i / Q < cols;
      const T gg = !live ? zero : gamma ? gv[t] : one;
      const T bb = !live || RMS || !beta ? zero : bv[t];
      if (i < V * Q) pl[i] = AP::make(gg, bb);
    }
    __syncthreads();
  }

  for (int64_t row0 = (int64_t(blockIdx.x) * G + g) * R; row0 < rows;
       row0 += int64_t(gridDim.x) * G * R) {
    Raw<T, V> rx[R][NV], rres[R][HAS_RES ? NV : 1];
    // SHIFT: the body [hh, bend) of each row and the lanes' extra elements
    int hh[R], bend[R];
    T ex[R], er[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      // rows past the end re-read the last row (in bounds) and are not stored
      const int64_t row = row0 + r < rows ? row0 + r : rows - 1;
      int h0 = 0, be = cols;
      if constexpr (SHIFT) {
        const int phase = int(reinterpret_cast<uintptr_t>(x + row * ld_x) & 15) / int(sizeof(T));
        h0 = (V - phase) & (V - 1);
        be = h0 + ((cols - h0) / V) * V;
      }
      hh[r] = h0;
      bend[r] = be;
      const int last = SHIFT ? be - V : clast;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = h0 + (k * kThreads + tid) * V;
        const int cl = c0 < be ? c0 : last;
        rx[r][k].load(x + row * ld_x + cl);
        if constexpr (HAS_RES) rres[r][k].load(res + row * ld_r + cl);
      }
      if constexpr (SHIFT) {
        const int nx = cols - (be - h0);
        const int ce = tid < nx ? (tid < h0 ? tid : be - h0 + tid) : 0;
        ex[r] = x[row * ld_x + ce];
        if constexpr (HAS_RES) er[r] = res[row * ld_r + ce];
      }
    }
    __builtin_amdgcn_sched_barrier(0);

    float h[R][EPT], he[R];
    P part;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      // SHIFT: the extra element (0 for lanes without one)
      const int nx = cols - (bend[r] - hh[r]);
      const int ce = tid < hh[r] ? tid : bend[r] - hh[r] + tid;
      if constexpr (SHIFT) {
        float v = raw_f32(ex[r]);
        if constexpr (HAS_RES) v += raw_f32(er[r]);
        he[r] = tid < nx ? v : 0.f;
      }
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        float xv[V];
        rx[r][k].unpack(xv);
        if constexpr (HAS_RES) {
          float rv[V];
          rres[r][k].unpack(rv);
#pragma unroll
          for (int i = 0; i < V; ++i) xv[i] += rv[i];
        }
#pragma unroll
        for (int i = 0; i < V; ++i) h[r][k * V + i] = xv[i];
      }
      if (!full) {
        // slots past the row end hold 0 (they re-read the row's last vector)
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const bool in = hh[r] + (k * kThreads + tid) * V < bend[r];
#pragma unroll
          for (int i = 0; i < V; ++i) h[r][k * V + i] = in ? h[r][k * V + i] : 0.f;
        }
      }
      if (res_out && row0 + r < rows) {
        T* ro = res_out + (row0 + r) * ld_ro;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int c0 = hh[r] + (k * kThreads + tid) * V;
          if (c0 < bend[r]) stv<T, V>(ro + c0, h[r] + k * V);
        }
        if constexpr (SHIFT) {
          if (tid < nx) stv<T, 1>(ro + ce, &he[r]);
        }
      }
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < EPT; ++i) sum = RMS ? fmaf(h[r][i], h[r][i], sum) : sum + h[r][i];
      if constexpr (SHIFT) sum = RMS ? fmaf(he[r], he[r], sum) : sum + he[r];
      part.p[r] = SumP{sum};      // out-of-row slots hold 0
    }
    float mean[R];
    if constexpr (RMS) {
      // RMSNorm: the single reduction above is already sum(h^2)
#pragma unroll
      for (int r = 0; r < R; ++r) mean[r] = 0.f;
    } else {
      // pass 1: the row means
      const P tot = group_allreduce<W>(part, lds[parity], wave, lane);
      parity ^= 1;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        mean[r] = tot.p[r].s * inv_cols;
        // pass 2: squared deviations from the row mean, over the owned columns
        float m2 = 0.f;
        if (full) {
#pragma unroll
          for (int i = 0; i < EPT; ++i) {
            const float d = h[r][i] - mean[r];
            m2 = fmaf(d, d, m2);
          }
        } else {
#pragma unroll
          for (int k = 0; k < NV; ++k) {
            const bool in = hh[r] + (k * kThreads + tid) * V < bend[r];
#pragma unroll
            for (int i = 0; i < V; ++i) {
              const float d = in ? h[r][k * V + i] - mean[r] : 0.f;
              m2 = fmaf(d, d, m2);
            }
          }
          if constexpr (SHIFT) {
            const float d = tid < cols - (bend[r] - hh[r]) ? he[r] - mean[r] : 0.f;
            m2 = fmaf(d, d, m2);
          }
        }
        part.p[r] = SumP{m2};
      }
    }
    const P sq = group_allreduce<W>(part, lds[parity], wave, lane);
    parity ^= 1;
    if constexpr (!kAffineResident && !SHIFT) load_affine();

#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float rstd = rsqrtf(sq.p[r].s * inv_cols + eps);
      if (SHIFT && row0 + r < rows) {
        T* yr = y + (row0 + r) * ld_y;
        int off[V];
#pragma unroll
        for (int i = 0; i < V; ++i)
          off[i] = ((hh[r] + i) & (V - 1)) * Q + (hh[r] + i >= V ? 1 : 0) + tid;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int c0 = hh[r] + (k * kThreads + tid) * V;
          float o[V];
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const Pair pr = pl[off[i] + k * kThreads];
            o[i] = fmaf((h[r][k * V + i] - mean[r]) * rstd, AP::gamma(pr), AP::beta(pr));
          }
          if (c0 < bend[r]) stv<T, V>(yr + c0, o);
        }
        const int nx = cols - (bend[r] - hh[r]);
        if (tid < nx) {
          const int ce = tid < hh[r] ? tid : bend[r] - hh[r] + tid;
          const Pair pr = pl[(ce & (V - 1)) * Q + ce / V];
          const float o = fmaf((he[r] - mean[r]) * rstd, AP::gamma(pr), AP::beta(pr));
          stv<T, 1>(yr + ce, &o);
        }
      } else if (row0 + r < rows) {
        T* yr = y + (row0 + r) * ld_y;
        // the affine form is uniform: one loop for gamma and beta both given
        // (no per-element choice of 1 / 0), one for the other cases
        if (affine) {
          // keep gamma and beta packed between rows: unpacked copies hoisted
          // out of the row loop would double their registers
          if constexpr (kAffineResident) {
#pragma unroll
            for (int k = 0; k < NV; ++k) {
#pragma unroll
              for (int j = 0; j < Raw<T, V>::kWords; ++j) {
                asm volatile("" : "+v"(rg[k].w[j]));
                if constexpr (!RMS) asm volatile("" : "+v"(rb[k].w[j]));
              }
            }
          }
#pragma unroll
          for (int k = 0; k < NV; ++k) {
            const int c0 = (k * kThreads + tid) * V;
            float gv[V], bv[V], o[V];
            rg[k].unpack(gv);
            if constexpr (RMS) {
#pragma unroll
              for (int i = 0; i < V; ++i) bv[i] = 0.f;     // RMSNorm has no beta
            } else {
              rb[k].unpack(bv);
            }
#pragma unroll
            for (int i = 0; i < V; ++i)
              o[i] = fmaf((h[r][k * V + i] - mean[r]) * rstd, gv[i], bv[i]);
            if (full || c0 < cols) stv<T, V>(yr + c0, o);
          }
        } else {
#pragma unroll
          for (int k = 0; k < NV; ++k) {
            const int c0 = (k * kThreads + tid) * V;
            float gv[V], bv[V];
            if (gamma) rg[k].unpack(gv);
            else {
#pragma unroll
              for (int i = 0; i < V; ++i) gv[i] = 1.f;
            }
            if (beta) rb[k].unpack(bv);
            else {
#pragma unroll
              for (int i = 0; i < V; ++i) bv[i] = 0.f;
            }
            float o[V];
#pragma unroll
            for (int i = 0; i < V; ++i)
              o[i] = fmaf((h[r][k * V + i] - mean[r]) * rstd, gv[i], bv[i]);
            if (c0 < cols) stv<T, V>(yr + c0, o);
          }
        }
      }
    }
  }
}

// (count, mean, M2) merged with the pairwise update of Chan, Golub and
// LeVeque (1979), written so that combine(a, b) and combine(b, a) round
// identically: the statistics of a streamed row.
struct MeanM2P {
  float n, mean, m2;
  __device__ __forceinline__ static MeanM2P combine(const MeanM2P& a, const MeanM2P& b) {
    if (a.n == 0.f) return b;
    if (b.n == 0.f) return a;
    const float n = a.n + b.n;
    const float d = b.mean - a.mean;
    return {n, (a.n * a.mean + b.n * b.mean) / n, (a.m2 + b.m2) + d * d * ((a.n * b.n) / n)};
  }
  template <class F> __device__ __forceinline__ static MeanM2P map(const MeanM2P& a, F f) {
    return {f(a.n), f(a.mean), f(a.m2)};
  }
};

// Rows longer than the register-resident capacity: one block of W waves per
// row streams it twice.  Pass 1 reads x (+ residual) in trips of U vectors
// per lane and merges each trip's exact two-pass statistics into a running
// (count, mean, M2) (RMSNorm: a running sum of squares); pass 2 re-reads
// them, writes residual_out and y.  Writing both in pass 2 keeps in-place
// outputs (y == x, residual_out == residual) correct.
template <typename T, bool HAS_RES, bool RMS, int W, bool VEC>
__global__ __launch_bounds__(64 * W) void layernorm_stream_kernel(
    const T* __restrict__ x, int64_t ld_x, const T* __restrict__ res, int64_t ld_r,
    const T* __restrict__ gamma, const T* __restrict__ beta, T* y, int64_t ld_y, T* res_out,
    int64_t ld_ro, int64_t rows, int cols, float eps, int trips) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  constexpr int U = 4;
  using P = MeanM2P;
  __shared__ P lds[2][W];
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int clast = cols - V;
  int parity = 0;

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const T* xr = x + row * ld_x;
    const T* rr = HAS_RES ? res + row * ld_r : nullptr;
    auto trip_h = [&](int t, float (&h)[U * V]) {
      Raw<T, V> rx[U], rres[HAS_RES ? U : 1];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = ((t * U + u) * kThreads + tid) * V;
        const int cl = c0 < cols ? c0 : clast;
        rx[u].load(xr + cl);
        if constexpr (HAS_RES) rres[u].load(rr + cl);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float xv[V];
        rx[u].unpack(xv);
        if constexpr (HAS_RES) {
          float rv[V];
          rres[u].unpack(rv);
#pragma unroll
          for (int i = 0; i < V; ++i) xv[i] += rv[i];
        }
#pragma unroll
        for (int i = 0; i < V; ++i) h[u * V + i] = xv[i];
      }
    };

    // pass 1: statistics
    P run{0.f, 0.f, 0.f};
    for (int t = 0; t < trips; ++t) {
      float h[U * V];
      trip_h(t, h);
      float n = 0.f, sum = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = ((t * U + u) * kThreads + tid) * V < cols;
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const float v = in ? h[u * V + i] : 0.f;
          sum = RMS ? fmaf(v, v, sum) : sum + v;
        }
        n += in ? float(V) : 0.f;
      }
      if constexpr (RMS) {
        run.m2 += sum;                        // running sum of squares
      } else {
        const float mt = n > 0.f ? sum / n : 0.f;
        float m2 = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool in = ((t * U + u) * kThreads + tid) * V < cols;
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const float d = in ? h[u * V + i] - mt : 0.f;
            m2 = fmaf(d, d, m2);
          }
        }
        run = P::combine(run, P{n, mt, m2});
      }
    }
    if constexpr (RMS) run.n = 1.f;          // keep the fold from skipping lanes
    const P st = group_allreduce<W>(run, lds[parity], wave, lane);
    parity ^= 1;
    const float inv_cols = 1.f / float(cols);
    const float mean = RMS ? 0.f : st.mean;
    // RMS: every lane carried mean 0, so the fold added the sums of squares
    const float rstd = rsqrtf(st.m2 * inv_cols + eps);

    // pass 2: residual_out and y
    T* yr = y + row * ld_y;
    T* ro = res_out ? res_out + row * ld_ro : nullptr;
    for (int t = 0; t < trips; ++t) {
      float h[U * V];
      trip_h(t, h);
      Raw<T, V> rg[U], rb[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = ((t * U + u) * kThreads + tid) * V;
        const int cl = c0 < cols ? c0 : clast;
        if (gamma) rg[u].template load<false>(gamma + cl);
        if (beta) rb[u].template load<false>(beta + cl);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c0 = ((t * U + u) * kThreads + tid) * V;
        if (c0 < cols) {
          if (ro) stv<T, V>(ro + c0, h + u * V);
          float gv[V], bv[V], o[V];
          if (gamma) rg[u].unpack(gv);
          else {
#pragma unroll
            for (int i = 0; i < V; ++i) gv[i] = 1.f;
          }
          if (beta) rb[u].unpack(bv);
          else {
#pragma unroll
            for (int i = 0; i < V; ++i) bv[i] = 0.f;
          }
#pragma unroll
          for (int i = 0; i < V; ++i) o[i] = fmaf((h[u * V + i] - mean) * rstd, gv[i], bv[i]);
          stv<T, V>(yr + c0, o);
        }
      }
    }
  }
}

// Rows longer than the register-resident capacity, with a row cache: one
// block of 16 waves per row keeps h = x + residual (fp32) of its first
// 64*16*CL columns in LDS (CL per lane) and of the next 64*16*CR columns in
// registers, so those columns are read from HBM once; with TAIL, the `tail`
// vector slots per lane past both are read twice as in
// layernorm_stream_kernel.  Pass 1 writes residual_out of the cached columns
// (they are never read again, so in-place outputs stay correct) and merges
// each slot group's exact two-pass (count, mean, M2) into one running triple
// per lane (RMSNorm: a running sum of squares), combined once across the
// block; pass 2 writes y from the registers, from LDS and from the re-read
// tail, with the tail's residual_out.  Each lane reads back only the LDS
// words it wrote, so the cache needs no barrier.  One block per compute unit
// holds one row at a time, so the loads of the next row's first slot groups
// are issued before the block-wide combine: they are in flight while this
// row's outputs are written.
template <typename T, bool HAS_RES, bool RMS, bool VEC, int CL, int CR, bool TAIL>
__global__ __launch_bounds__(1024) void layernorm_cached_kernel(
    const T* __restrict__ x, int64_t ld_x, const T* __restrict__ res, int64_t ld_r,
    const T* __restrict__ gamma, const T* __restrict__ beta, T* y, int64_t ld_y, T* res_out,
    int64_t ld_ro, int64_t rows, int cols, float eps, int tail) {
  constexpr int W = 16, kThreads = 64 * W;
  constexpr int V = VEC ? Elem<T>::kVec : 1;   // elements per slot and lane
  constexpr int NL = CL / V, NR = CR / V, NS = NL + NR;   // vector slots per lane
  static_assert(CL % V == 0 && CR % V == 0 && CL % 4 == 0, "cache parts are whole vectors");
  // cached slots go in groups of G (about FS_LN_CACHE_GROUP_WORDS raw
  // registers each) with the loads of the next AH groups in flight
  constexpr int kWords = Raw<T, V>::kWords * (HAS_RES ? 2 : 1);
  constexpr int G0 = kWords >= FS_LN_CACHE_GROUP_WORDS ? 1 : FS_LN_CACHE_GROUP_WORDS / kWords;
  constexpr int G = VEC || G0 < 4 ? G0 : 4;   // element-wise slots: groups of 4
  constexpr int NG = NS / G, AH = FS_LN_CACHE_AHEAD, R = AH + 1;
  static_assert(NL % G == 0 && NR % G == 0, "slot groups split the cache parts");
  using P = MeanM2P;
  __shared__ f32x4 cache[CL / 4][kThreads];
  __shared__ P lds[2][W];
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int clast = cols - V;
  const int nslots = (cols + kThreads * V - 1) / (kThreads * V);   // slots the row uses
  int parity = 0;

  // loads of a slot of row `row`, clamped in bounds past the row end
  auto load = [&](int64_t row, int lt, int slot, Raw<T, V>& rx, Raw<T, V>& rres) {
    const int c0 = (slot * kThreads + lt) * V;
    const int cl = c0 < cols ? c0 : clast;
    rx.load(x + row * ld_x + cl);
    if constexpr (HAS_RES) rres.load(res + row * ld_r + cl);
  };
  Raw<T, V> rx[R][G], rres[R][G];
  // the first AH slot groups of a row.  Every load of the kernel is issued
  // unconditionally (addresses past the row are clamped in bounds, and the
  // row after the last is replaced by the last): with no branch around a
  // load, the waits for each group count exactly the loads issued after it
  auto prime = [&](int64_t row, int lt) {
#pragma unroll
    for (int g = 0; g < AH && g < NG; ++g) {
#pragma unroll
      for (int k = 0; k < G; ++k) load(row, lt, g * G + k, rx[g][k], rres[g][k]);
    }
  };
  // gamma and beta, or any valid address when absent (their values unused)
  const T* gsrc = gamma ? gamma : x;
  const T* bsrc = beta ? beta : x;
  prime(blockIdx.x, tid);

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    T* yr = y + row * ld_y;
    T* ro = res_out ? res_out + row * ld_ro : nullptr;
    // the lane index is re-read per row (an empty asm) so that per-lane
    // offsets and column tests are recomputed, not kept in registers
    // across rows
    int lt = tid;
    asm volatile("" : "+v"(lt));
    auto col_of = [&](int slot) { return (slot * kThreads + lt) * V; };
    auto hval = [&](const Raw<T, V>& rxs, const Raw<T, V>& rrs, float* h) {
      rxs.unpack(h);
      if constexpr (HAS_RES) {
        float rv[V];
        rrs.unpack(rv);
#pragma unroll
        for (int i = 0; i < V; ++i) h[i] += rv[i];
      }
    };
    // merge the statistics of K slots from s0 on into the lane's running triple
    P run{0.f, 0.f, 0.f};
    auto absorb = [&](auto kslots, int s0, const float* h) {
      constexpr int K = decltype(kslots)::value;
      float n = 0.f, sum = 0.f;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const bool in = col_of(s0 + k) < cols;
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const float v = in ? h[k * V + i] : 0.f;
          sum = RMS ? fmaf(v, v, sum) : sum + v;
        }
        n += in ? float(V) : 0.f;
      }
      if constexpr (RMS) {
        run.m2 += sum;                        // running sum of squares
      } else {
        const float mt = n > 0.f ? sum / n : 0.f;
        float m2 = 0.f;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const bool in = col_of(s0 + k) < cols;
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const float d = in ? h[k * V + i] - mt : 0.f;
            m2 = fmaf(d, d, m2);
          }
        }
        run = P::combine(run, P{n, mt, m2});
      }
    };
    auto store_res = [&](int slot, const float* h) {
      const int c0 = col_of(slot);
      if (ro && c0 < cols) stv<T, V>(ro + c0, h);
    };
    // the tail slots NS ... NS + tail - 1, one ahead: a slot's loads are in
    // flight while the previous slot is used.  Loads of slots past the row
    // are clamped in bounds (they count nothing and store nothing).
    auto over_tail = [&](auto use) {
      Raw<T, V> tx[2], tr[2];
      load(row, lt, NS, tx[0], tr[0]);
      for (int j = 0; j < tail; j += 2) {
        load(row, lt, NS + j + 1, tx[1], tr[1]);
        __builtin_amdgcn_sched_barrier(0);
        use(NS + j, tx[0], tr[0]);
        load(row, lt, NS + j + 2, tx[0], tr[0]);
        __builtin_amdgcn_sched_barrier(0);
        if (j + 1 < tail) use(NS + j + 1, tx[1], tr[1]);
      }
    };

    // pass 1: LDS part, register part (the first AH groups were issued
    // before), tail
    float hr[CR];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + AH < NG) {
#pragma unroll
        for (int k = 0; k < G; ++k)
          load(row, lt, (g + AH) * G + k, rx[(g + AH) % R][k], rres[(g + AH) % R][k]);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (g * G < nslots) {
        float h[G * V];
#pragma unroll
        for (int k = 0; k < G; ++k) hval(rx[g % R][k], rres[g % R][k], h + k * V);
        absorb(std::integral_constant<int, G>{}, g * G, h);
#pragma unroll
        for (int k = 0; k < G; ++k) store_res(g * G + k, h + k * V);
        if (g * G < NL) {
#pragma unroll
          for (int k = 0; k < G * V / 4; ++k)
            cache[g * G * V / 4 + k][lt] = f32x4{h[4 * k], h[4 * k + 1], h[4 * k + 2], h[4 * k + 3]};
        } else {
#pragma unroll
          for (int i = 0; i < G * V; ++i) hr[g * G * V - CL + i] = h[i];
        }
      }
    }
    if constexpr (TAIL) {
      over_tail([&](int slot, const Raw<T, V>& rxs, const Raw<T, V>& rrs) {
        float h[V];
        hval(rxs, rrs, h);
        absorb(std::integral_constant<int, 1>{}, slot, h);
      });
    }

    // gamma and beta of the cached slots are loaded D slots ahead of their
    // use in pass 2, the first D before the next row's loads and the
    // block-wide combine
    constexpr int D = FS_LN_CACHE_GB_AHEAD;
    auto slot_at = [](int i) { return i < NR ? NL + i : i - NR; };   // pass-2 order
    auto load_gb = [&](int slot, Raw<T, V>& rg, Raw<T, V>& rb) {
      const int c0 = col_of(slot);
      const int cl = c0 < cols ? c0 : clast;
      rg.template load<false>(gsrc + cl);
      if constexpr (!RMS) rb.template load<false>(bsrc + cl);
    };
    Raw<T, V> rg[D + 1], rb[D + 1];
#pragma unroll
    for (int i = 0; i < D && i < NS; ++i) load_gb(slot_at(i), rg[i], rb[i]);
    // the next row's first slot groups, in flight from here on
    const int64_t next = row + gridDim.x;
    prime(next < rows ? next : rows - 1, lt);

    if constexpr (RMS) run.n = 1.f;          // keep the fold from skipping lanes
    const P st = group_allreduce<W>(run, lds[parity], wave, lane);
    parity ^= 1;
    const float mean = RMS ? 0.f : st.mean;
    // RMS: every lane carried mean 0, so the fold added the sums of squares
    const float rstd = rsqrtf(st.m2 * (1.f / float(cols)) + eps);

    asm volatile("" : "+v"(lt));   // pass 2 recomputes its column tests too
    // pass 2: y, register part first (which frees its registers), then LDS
    auto emit = [&](int slot, const float* h, const Raw<T, V>& g, const Raw<T, V>& b) {
      const int c0 = col_of(slot);
      if (c0 >= cols) return;
      float gv[V], bv[V], o[V];
      if (gamma) g.unpack(gv);
      else {
#pragma unroll
        for (int i = 0; i < V; ++i) gv[i] = 1.f;
      }
      if (!RMS && beta) b.unpack(bv);
      else {
#pragma unroll
        for (int i = 0; i < V; ++i) bv[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] = fmaf((h[i] - mean) * rstd, gv[i], bv[i]);
      stv<T, V>(yr + c0, o);
    };
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      if (i + D < NS) load_gb(slot_at(i + D), rg[(i + D) % (D + 1)], rb[(i + D) % (D + 1)]);
      __builtin_amdgcn_sched_barrier(0);
      if (slot_at(i) >= nslots) continue;
      float h[V];
      if (i < NR) {
#pragma unroll
        for (int k = 0; k < V; ++k) h[k] = hr[i * V + k];
      } else if constexpr (V >= 4) {
#pragma unroll
        for (int k = 0; k < V / 4; ++k) {
          const f32x4 v = cache[(i - NR) * (V / 4) + k][lt];
          h[4 * k] = v.x; h[4 * k + 1] = v.y; h[4 * k + 2] = v.z; h[4 * k + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int k = 0; k < V; ++k) h[k] = cache[((i - NR) * V + k) / 4][lt][((i - NR) * V + k) % 4];
      }
      emit(slot_at(i), h, rg[i % (D + 1)], rb[i % (D + 1)]);
    }
    if constexpr (TAIL) {
      over_tail([&](int slot, const Raw<T, V>& rxs, const Raw<T, V>& rrs) {
        float h[V];
        hval(rxs, rrs, h);
        store_res(slot, h);
        Raw<T, V> g1, b1;
        load_gb(slot, g1, b1);
        emit(slot, h, g1, b1);
      });
    }
  }
}

// rows batched per group: enough that a one-wave group handles about
// FS_LN_BATCH_ELEMS elements per lane per trip
// Rows that fill one wave's 16-byte slots exactly (cols == 64 * EPT, every
// operand on 16-byte rows) with the affine parameters given: the one-wave
// rung of layernorm_kernel without its general cases.  A short kernel (the
// block's 64 MiB LN1) is bound by how soon its waves put their loads in
// flight, so each wave issues its row loads first -- before gamma and beta,
// before any other kernel argument is needed -- and the host passes 1/cols;
// there is no masking, no staging and no LDS.  R rows per wave share one
// shuffle sequence per statistic; rows past the end re-read the last row and
// are not stored.  LOOP: the grid is capped and waves loop over the rows;
// otherwise one trip covers them all.  Same arithmetic, in the same order, as
// layernorm_kernel.
// The arguments a wave needs before its first row loads (x, residual, rows,
// eps, gamma, beta) fill the first 64 bytes of the argument block, so one
// scalar-cache line serves them; the outputs' follow.
template <typename T, bool HAS_RES, bool RMS, int EPT, int R, bool LOOP>
__global__ __launch_bounds__(256) void layernorm_wave_kernel(
    const T* __restrict__ x, int64_t ld_x, const T* __restrict__ res, int64_t ld_r,
    int64_t rows, float eps, float inv_cols, const T* __restrict__ gamma,
    const T* __restrict__ beta, T* y, int64_t ld_y, T* res_out, int64_t ld_ro) {
  constexpr int V = Elem<T>::kVec;
  constexpr int NV = EPT / V;
  static_assert(EPT % V == 0, "EPT must be a multiple of the vector width");
  const int lane = threadIdx.x % 64;
  const int64_t wave = __builtin_amdgcn_readfirstlane(int(blockIdx.x) * 4 + int(threadIdx.x / 64));
  const int64_t step = int64_t(gridDim.x) * 4 * R;
  int64_t row0 = wave * R;
  // eps is tested with rows (the host guarantees eps >= 0) so that both come
  // in the wave's first scalar load instead of a load after the reductions
  if (row0 >= rows || !(eps >= 0.f)) return;
  Raw<T, V> rx[R][NV], rr[R][HAS_RES ? NV : 1], rg[NV], rb[NV];
  auto load_rows = [&](int64_t r0) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t row = r0 + r < rows ? r0 + r : rows - 1;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        rx[r][k].load(x + row * ld_x + (k * 64 + lane) * V);
        if constexpr (HAS_RES) rr[r][k].load(res + row * ld_r + (k * 64 + lane) * V);
      }
    }
  };
  // the first trip's rows go out before gamma and beta (loaded once, kept
  // in registers); later trips load their rows at the end of the previous
  // one
  load_rows(row0);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    rg[k].template load<false>(gamma + (k * 64 + lane) * V);
    if constexpr (!RMS) rb[k].template load<false>(beta + (k * 64 + lane) * V);
  }
  for (;;) {
    float h[R][EPT];
    Multi<SumP, R> part;
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        float xv[V];
        rx[r][k].unpack(xv);
        if constexpr (HAS_RES) {
          float rv[V];
          rr[r][k].unpack(rv);
#pragma unroll
          for (int i = 0; i < V; ++i) xv[i] += rv[i];
        }
#pragma unroll
        for (int i = 0; i < V; ++i) h[r][k * V + i] = xv[i];
      }
      if (res_out && row0 + r < rows) {
#pragma unroll
        for (int k = 0; k < NV; ++k)
          stv<T, V>(res_out + (row0 + r) * ld_ro + (k * 64 + lane) * V, h[r] + k * V);
      }
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < EPT; ++i) sum = RMS ? fmaf(h[r][i], h[r][i], sum) : sum + h[r][i];
      part.p[r] = SumP{sum};
    }
    float mean[R];
    if constexpr (RMS) {
#pragma unroll
      for (int r = 0; r < R; ++r) mean[r] = 0.f;
    } else {
      const Multi<SumP, R> tot = wave_allreduce(part);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        mean[r] = tot.p[r].s * inv_cols;
        float m2 = 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          const float d = h[r][i] - mean[r];
          m2 = fmaf(d, d, m2);
        }
        part.p[r] = SumP{m2};
      }
    }
    const Multi<SumP, R> sq = wave_allreduce(part);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (row0 + r >= rows) break;
      const float rstd = rsqrtf(sq.p[r].s * inv_cols + eps);
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        float gv[V], bv[V], o[V];
        rg[k].unpack(gv);
        if constexpr (RMS) {
#pragma unroll
          for (int i = 0; i < V; ++i) bv[i] = 0.f;
        } else {
          rb[k].unpack(bv);
        }
#pragma unroll
        for (int i = 0; i < V; ++i) o[i] = fmaf((h[r][k * V + i] - mean[r]) * rstd, gv[i], bv[i]);
        stv<T, V>(y + (row0 + r) * ld_y + (k * 64 + lane) * V, o);
      }
    }
    // one trip covers every row when the grid does (straight-line code: the
    // compiler then keeps gamma and beta packed until the outputs)
    if constexpr (!LOOP) break;
    row0 += step;
    if (row0 >= rows) break;
    load_rows(row0);
  }
}

template <int W, int EPT>
struct RowsPerGroup {
  static constexpr int value = (W == 1 && EPT < FS_LN_BATCH_ELEMS) ? FS_LN_BATCH_ELEMS / EPT : 1;
};

// the one-trip and the looping form of one layernorm_wave_kernel variant
template <typename T, bool HAS_RES, bool RMS, int EPT, int R>
struct WaveKernels {
  decltype(&layernorm_wave_kernel<T, HAS_RES, RMS, EPT, R, false>) one =
      layernorm_wave_kernel<T, HAS_RES, RMS, EPT, R, false>;
  decltype(&layernorm_wave_kernel<T, HAS_RES, RMS, EPT, R, true>) loop =
      layernorm_wave_kernel<T, HAS_RES, RMS, EPT, R, true>;
};

template <typename T, bool HAS_RES, bool RMS, bool VEC>
hipError_t dispatch(const LayerNormArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  const int64_t c = a.cols;
  auto launch = [&](auto kern, int threads, int rows_per_block, int blocks_per_cu) {
    int64_t want = (a.rows + rows_per_block - 1) / rows_per_block;
    int64_t cap = int64_t(cus) * blocks_per_cu * FS_LN_GRID_SCALE / 4;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s, static_cast<const T*>(a.x), a.ld_x,
                       static_cast<const T*>(a.res), a.ld_r, static_cast<const T*>(a.gamma),
                       static_cast<const T*>(a.beta), static_cast<T*>(a.y), a.ld_y,
                       static_cast<T*>(a.res_out), a.ld_ro, a.rows, int(a.cols), a.eps);
    return hipGetLastError();
  };
  // one-wave rows that fill every lane's slots, affine parameters given
  if constexpr (VEC) {
    if (FS_LN_WAVE_PATH && a.gamma != nullptr && (RMS || a.beta != nullptr) &&
        c < FS_LN_SPLIT_COLS) {
      auto wave = [&](auto kern, int r) {
        const int64_t want = (a.rows + 4 * r - 1) / (4 * r);
        const int64_t cap = int64_t(cus) * 8 * FS_LN_GRID_SCALE / 4;
        const int grid = int(want < cap ? (want < 1 ? 1 : want) : cap);
        hipLaunchKernelGGL(want <= cap ? kern.one : kern.loop, dim3(grid), dim3(256), 0, s,
                           static_cast<const T*>(a.x), a.ld_x, static_cast<const T*>(a.res),
                           a.ld_r, a.rows, a.eps, 1.f / float(a.cols),
                           static_cast<const T*>(a.gamma), static_cast<const T*>(a.beta),
                           static_cast<T*>(a.y), a.ld_y, static_cast<T*>(a.res_out), a.ld_ro);
        return hipGetLastError();
      };
#define FS_LNW(E)                                                                        \
  if (c == int64_t(64) * E)                                                             \
    return wave(WaveKernels<T, HAS_RES, RMS, E, RowsPerGroup<1, E>::value>{},           \
                RowsPerGroup<1, E>::value);
      FS_LNW(V)
      FS_LNW(2 * V)
      FS_LNW(4 * V)
#undef FS_LNW
    }
  }
// Variant ladder, in order: the first rung with at least min_w waves per row
  // and a row capacity 64 * W * EPT >= cols is launched.
  const int min_w = c >= FS_LN_SPLIT_COLS ? FS_LN_MIN_WAVES : 1;
  // rows that share a 16-byte phase: the vector ladder over each row's
  // aligned body, gamma and beta staged in LDS (a row of c columns has at
  // most c / V whole vectors in it)
  if constexpr (!VEC) {
    if (a.shifted && c <= FS_LN_SHIFT_REG_COLS) {
      constexpr int VS = Elem<T>::kVec;
      constexpr int kPair = sizeof(typename AffinePair<T>::type);
      auto shift = [&](auto kern, int threads, int rows_per_block, int wt) {
        const size_t lds = size_t(VS) * (wt + 1) * kPair;   // wt: vectors per row group
        int64_t want = (a.rows + rows_per_block - 1) / rows_per_block;
        // no more blocks than fit at once: every block stages the whole
        // table, so each should normalise many rows with it
        const int per_cu = int((160 * 1024) / (lds + 1024));
        int64_t cap = int64_t(cus) * (per_cu < 1 ? 1 : per_cu);
        int grid = int(want < cap ? want : cap);
        if (grid < 1) grid = 1;
        hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), lds, s, static_cast<const T*>(a.x),
                           a.ld_x, static_cast<const T*>(a.res), a.ld_r,
                           static_cast<const T*>(a.gamma), static_cast<const T*>(a.beta),
                           static_cast<T*>(a.y), a.ld_y, static_cast<T*>(a.res_out), a.ld_ro,
                           a.rows, int(a.cols), a.eps);
        return hipGetLastError();
      };
#define FS_LNS(Wv, E, Gv)                                                                       \
  if (Wv >= min_w && c <= int64_t(64) * Wv * E)                                                 \
    return shift(layernorm_kernel<T, HAS_RES, RMS, Wv, E, false, true, Gv, RowsPerGroup<Wv, E>::value>, \
                 64 * Wv * Gv, Gv * RowsPerGroup<Wv, E>::value, 64 * Wv * (E / VS));
      if constexpr (VS <= 4) { FS_LNS(1, 4, 4) }
      FS_LNS(1, 8, 4)
      FS_LNS(1, 16, 4)
      FS_LNS(1, 32, 4)
      FS_LNS(1, 64, 4)
      FS_LNS(2, 32, 1)
      FS_LNS(2, 64, 1)
      FS_LNS(4, 16, 1)
      FS_LNS(4, 32, 1)
      FS_LNS(4, 64, 1)
      FS_LNS(8, 8, 1)
      FS_LNS(8, 16, 1)
      FS_LNS(8, 32, 1)
#undef FS_LNS
    }
  }
#define FS_LN(Wv, E, Gv, BPC)                                                       \
  if (Wv >= min_w && c <= int64_t(64) * Wv * E &&                                 \
      (VEC || c <= FS_LN_ELEMENTWISE_REG_COLS))                                  \
    return launch(layernorm_kernel<T, HAS_RES, RMS, Wv, E, VEC, false, Gv, RowsPerGroup<Wv, E>::value>, \
                  64 * Wv * Gv, Gv * RowsPerGroup<Wv, E>::value, BPC);
  if constexpr (V <= 1) { FS_LN(1, 1, 4, 8) }
  if constexpr (V <= 2) { FS_LN(1, 2, 4, 8) }
  if constexpr (V <= 4) { FS_LN(1, 4, 4, 8) }
  FS_LN(1, 8, 4, 8)
  if constexpr (VEC) {
    FS_LN(1, 16, 4, 8)
    FS_LN(1, 32, 4, 8)
    FS_LN(1, 64, 4, 8)
    FS_LN(2, 32, 1, 16)
    FS_LN(2, 64, 1, 16)
    FS_LN(4, 16, 1, 8)
    FS_LN(4, 32, 1, 8)
    FS_LN(4, 64, 1, 8)
    FS_LN(8, 8, 1, 4)
    FS_LN(8, 16, 1, 4)
    FS_LN(8, 32, 1, 4)
    FS_LN(16, 24, 1, 1)
    // fp32 rows at 16 waves x 32 elements spill; bf16 rows fit
    if constexpr (sizeof(T) == 2) { FS_LN(16, 32, 1, 1) }
  } else {
    // element-wise loads take one register per value and one address per
    // element: wider rows take more waves at 8 elements per thread (16 and
    // more left 1-2 waves per SIMD), and past 8192 columns the row cache
    FS_LN(2, 8, 1, 16)
    FS_LN(4, 8, 1, 8)
    FS_LN(8, 8, 1, 4)
    FS_LN(16, 8, 1, 1)
  }
#undef FS_LN
  // longer rows: row cache in LDS and registers, the columns past it
  // streamed; one 16-wave block per compute unit
  // (element-wise rows only past FS_LN_ELEMENTWISE_CACHE_COLS: below it the
  // row cache's single-element slots cost more than the streamed re-read)
  if constexpr (VEC || FS_LN_CACHE_ELEMENTWISE) if (VEC || c > FS_LN_ELEMENTWISE_CACHE_COLS) {
    constexpr int CL = 32, CR = FS_LN_CACHE_REGS;
    constexpr int64_t kCached = int64_t(1024) * (CL + CR);
    auto go = [&](auto kern, int tail) {
      const int64_t grid = a.rows < cus ? a.rows : cus;
      hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(1024), 0, s, static_cast<const T*>(a.x),
                         a.ld_x, static_cast<const T*>(a.res), a.ld_r,
                         static_cast<const T*>(a.gamma), static_cast<const T*>(a.beta),
                         static_cast<T*>(a.y), a.ld_y, static_cast<T*>(a.res_out), a.ld_ro, a.rows,
                         int(a.cols), a.eps, tail);
      return hipGetLastError();
    };
    // rows that a 16-per-lane register part holds take it: no empty slots
    // are loaded (49152 columns: 4.5 -> 4.9 TB/s)
    if constexpr (CR > 16 && VEC) {
      if (c <= int64_t(1024) * (CL + 16))
        return go(layernorm_cached_kernel<T, HAS_RES, RMS, VEC, CL, 16, false>, 0);
    }
    if (c <= kCached) return go(layernorm_cached_kernel<T, HAS_RES, RMS, VEC, CL, CR, false>, 0);
    constexpr int64_t kSlot = int64_t(1024) * V;
    return go(layernorm_cached_kernel<T, HAS_RES, RMS, VEC, CL, CR, true>,
              int((c - kCached + kSlot - 1) / kSlot));
  }
  // longer rows, element-wise path: streamed, one block of FS_LN_STREAM_WAVES
  // waves per row
  {
    constexpr int W = FS_LN_STREAM_WAVES, U = 4;
    const int trips = int((c + int64_t(64) * W * V * U - 1) / (int64_t(64) * W * V * U));
    const int64_t cap = int64_t(cus) * FS_LN_STREAM_BPC;
    int64_t grid = a.rows < cap ? a.rows : cap;
    hipLaunchKernelGGL((layernorm_stream_kernel<T, HAS_RES, RMS, W, VEC>), dim3(unsigned(grid)),
                       dim3(64 * W), 0, s, static_cast<const T*>(a.x), a.ld_x,
                       static_cast<const T*>(a.res), a.ld_r, static_cast<const T*>(a.gamma),
                       static_cast<const T*>(a.beta), static_cast<T*>(a.y), a.ld_y,
                       static_cast<T*>(a.res_out), a.ld_ro, a.rows, int(a.cols), a.eps, trips);
    return hipGetLastError();
  }
}

template <typename T, bool RMS>
hipError_t by_res(const LayerNormArgs& a, int cus, hipStream_t s) {
  if (a.res == nullptr)
    return a.vec ? dispatch<T, false, RMS, true>(a, cus, s) : dispatch<T, false, RMS, false>(a, cus, s);
  return a.vec ? dispatch<T, true, RMS, true>(a, cus, s) : dispatch<T, true, RMS, false>(a, cus, s);
}

}  // namespace

hipError_t launch_layernorm(const LayerNormArgs& a, int cus, hipStream_t s) {
  if (a.rms) return a.dtype == FS_BF16 ? by_res<uint16_t, true>(a, cus, s) : by_res<float, true>(a, cus, s);
  return a.dtype == FS_BF16 ? by_res<uint16_t, false>(a, cus, s) : by_res<float, false>(a, cus, s);
}

}  // namespace fs
