// Fused row softmax with pre-scale, additive mask and causal masking.
//
// y[r, :] = softmax(x[r, :] * scale + mask[r, :]) -- KernelOPT Appendix A
// (Planner item 9, fused softmax; Codegen prompt, online softmax).
//
// Design (gfx950): one row per group of W wave64s; each thread holds EPT
// elements of the row in registers, so HBM is read once and written once.
// Per thread: logits a = x * scale + mask, the local max m, and the local
// sum d of exp(a - m) = 2^((a - m) log2 e) with the exponentials kept in
// registers.  The difference is taken before the scaling: exact near the
// maximum at any magnitude, so large logits keep full relative accuracy and
// rows filled with the most negative finite value (a common mask) stay
// finite.  (An exponent formed as one fma, a log2e - round(m log2e), carries
// the rounding of m log2e, which overflows the exponent once |m| passes
// about 1.5e9, or m log2e itself overflows.)  A single all-reduce combines
// the (m, d) pairs:
//     (m1, d1) + (m2, d2) = (M, d1 * e^(m1 - M) + d2 * e^(m2 - M)),  M = max
// with m = -inf acting as the identity (never evaluating -inf - -inf).  The
// output is the stored exponential times e^(m - M) / D: one exp2 per element.
#include "device_common.hpp"
#include "launch.hpp"

// Build-time tuning: rows of at least FS_SM_SPLIT_COLS columns use at least
// FS_SM_MIN_WAVES waves per row; one-wave rows are batched to about
// FS_SM_BATCH_ELEMS elements per lane per trip; the grid holds at most
// FS_SM_GRID_SCALE/4 times the per-variant blocks-per-CU figure.
#ifndef FS_SM_FULL_PATH
#define FS_SM_FULL_PATH 1   // no per-element mask for non-causal rows that fill every slot
#endif
#ifndef FS_SM_MIN_WAVES
#define FS_SM_MIN_WAVES 2
#endif
#ifndef FS_SM_SPLIT_COLS
#define FS_SM_SPLIT_COLS 2048
#endif
#ifndef FS_SM_BATCH_ELEMS
#define FS_SM_BATCH_ELEMS 16
#endif
#ifndef FS_SM_ELEMENTWISE_REG_COLS
#define FS_SM_ELEMENTWISE_REG_COLS 32768   // widest element-wise row on the register rungs
#endif
#ifndef FS_SM_SHIFT_REG_COLS
#define FS_SM_SHIFT_REG_COLS 16384  // widest row of a shared 16-byte phase on the register rungs
#endif
#ifndef FS_SM_CACHE_AHEAD
#define FS_SM_CACHE_AHEAD 3   // slot groups of loads in flight ahead in the row cache's pass 1
#endif
#ifndef FS_SM_CACHE_GROUP_WORDS
#define FS_SM_CACHE_GROUP_WORDS 8   // raw load registers per slot group of the row cache
#endif
#ifndef FS_SM_ONE_TRIP_MIN_W
#define FS_SM_ONE_TRIP_MIN_W 2   // vector rungs of at least this many waves per row have a one-trip form
#endif
#ifndef FS_SM_GRID_SCALE
#define FS_SM_GRID_SCALE 64
#endif

namespace fs {
namespace {

struct MaxSumP {
  float m, d;
  // (m1, d1) + (m2, d2) = (M, d_big + d_small * 2^-|m1 - m2|): the pair with
  // the larger max keeps weight 1, so one exp2 per combine.  Symmetric in its
  // arguments (swapping them selects the same big/small pair), so every lane
  // ends with identical bits.  m = -inf is the identity (d = 0).
  __device__ __forceinline__ static MaxSumP combine(const MaxSumP& a, const MaxSumP& b) {
    const float M = fmaxf(a.m, b.m);
    if (M == -INFINITY) return {-INFINITY, 0.f};
    const bool a_big = a.m > b.m;
    const float big = a_big ? a.d : b.d, small = a_big ? b.d : a.d;
    const float e = __builtin_amdgcn_exp2f(-fabsf(a.m - b.m) * kLog2e);   // 2^-inf = 0
    return {M, fmaf(small, e, big)};
  }
  template <class F> __device__ __forceinline__ static MaxSumP map(const MaxSumP& a, F f) {
    return {f(a.m), f(a.d)};
  }
};

// Plain maximum (one-wave rows reduce the max and the sum separately).
struct MaxF {
  float m;
  __device__ __forceinline__ static MaxF combine(const MaxF& a, const MaxF& b) {
    return {fmaxf(a.m, b.m)};
  }
  template <class F> __device__ __forceinline__ static MaxF map(const MaxF& a, F f) {
    return {f(a.m)};
  }
};

// Stores the V values of the vector at column c0 that lie before column
// `end` (a whole vector, a leading part of it, or nothing).
template <typename T, int V>
__device__ __forceinline__ void store_until(T* row, int c0, int end, const float (&o)[V]) {
  if (c0 + V <= end) {
    stv<T, V>(row + c0, o);
  } else if (c0 < end) {
#pragma unroll
    for (int i = 0; i < V; ++i)
      if (c0 + i < end) stv<T, 1>(row + c0 + i, &o[i]);
  }
}

// T: storage type of x and y; MT: storage type of the mask (used when
// HAS_MASK).  W waves per row; EPT elements per thread; VEC: 16-byte vector
// path; G row groups per block (W == 1 only); R rows per group per trip --
// narrow rows are batched so that a wave keeps R rows of loads in flight and
// reduces them with one shuffle sequence.
// SHIFT: rows that are not whole 16-byte vectors but whose x, mask and y
// start every row at one offset within a 16-byte unit.  The thread's vectors
// tile the row's aligned body, from its first 16-byte boundary (h columns
// in) to its last; the head and tail (at most V-1 columns each) are one
// extra element for each of the group's first lanes: lanes below h take
// the head, the next ones the tail.
// LOOP: groups walk the rows with a grid stride; without it every group
// takes one trip (the host launches that form when the grid covers the
// rows), as straight-line code with nothing computed for later trips.
// The arguments a wave needs before its first loads (x, the mask, rows,
// q_len, cols) fill the first 64 bytes of the argument block.
template <typename T, typename MT, bool HAS_MASK, int W, int EPT, bool VEC, bool SHIFT, int G,
          int R, bool LOOP>
__global__ __launch_bounds__(64 * W * G) void softmax_kernel(
    const T* __restrict__ x, int64_t ld_x, const MT* __restrict__ mask, int64_t ld_m,
    int64_t rows, int64_t q_len, int cols, int trim_shift, float scale, T* y, int64_t ld_y) {
  constexpr int kThreads = 64 * W;
  constexpr int V = VEC || SHIFT ? Elem<T>::kVec : 1;
  constexpr int NV = EPT / V;                       // vectors per thread
  static_assert(EPT % V == 0, "EPT must be a multiple of the vector width");
  // one LDS fold area and one barrier sequence per block: rows wider than a
  // wave take the whole block (the row loop is then uniform across it)
  static_assert(W == 1 || G == 1, "multi-wave rows use one row group per block");
  __shared__ Multi<MaxSumP, R> lds[W == 1 ? 1 : 2][W];

  const int tid = threadIdx.x % kThreads;
  const int wave = tid / 64, lane = tid % 64;
  // the row group is uniform across a wave: keep it (and all row
  // arithmetic) in scalar registers
  const int g = __builtin_amdgcn_readfirstlane(threadIdx.x / kThreads);
  int parity = 0;
  // rows without a causal rule that fill every slot of every lane have no
  // column to mask (uniform)
  const bool whole = !SHIFT && FS_SM_FULL_PATH && q_len == 0 && cols == kThreads * EPT;
  // every slot of every lane is stored: rows written whole (no trimming)
  // that fill every slot (uniform; causal rows included)
  const bool store_all = !SHIFT && trim_shift < 0 && cols == kThreads * EPT;

  // causal position of row0 (row0 mod q_len), advanced by the loop step
  // without a division per row.  The host sends q_len >= 2^30 to the row
  // cache, so positions and column limits fit in 32 bits here and
  // stay in scalar registers with native scalar compares (64-bit compares
  // run on the vector unit).
  const int64_t step = int64_t(gridDim.x) * G * R;
  int64_t row0 = (int64_t(blockIdx.x) * G + g) * R;
  const int q = int(q_len);
  const int coff = cols - q;                 // cols - q_len
  // A power-of-two q_len (the usual sequence length) takes a mask instead of
  // a division; the step's remainder is formed only by waves that take a
  // second trip (with the grid of one trip per wave, none does).  The load
  // addresses depend on the position, so this sits on every wave's path to
  // its first load.
  int pos0 = 0, step_mod = 0;
  const bool q_pow2 = q > 0 && (q & (q - 1)) == 0;
  if (q > 0) {
    pos0 = q_pow2 ? int(row0 & (q - 1)) : int(row0 % q_len);
    if constexpr (LOOP) {
      if (row0 + step < rows) step_mod = q_pow2 ? int(step & (q - 1)) : int(step % q_len);
    }
  }
  for (; row0 < rows; row0 += step) {
    Raw<T, V> rx[R][NV];
    Raw<MT, V> rm[R][HAS_MASK ? NV : 1];
    int lim[R], wend[R];
    // SHIFT: the body [hh, bend) and each lane's extra element (raw)
    int hh[R], bend[R];
    T ex[R];
    MT em[R];
    // one 64-bit row offset per trip; only the last trip can run past the
    // end, and its missing rows re-read the last row (in bounds, not stored)
    const bool full_trip = row0 + R <= rows;
    const T* xb = x + row0 * ld_x;
    const MT* mb = HAS_MASK ? mask + row0 * ld_m : nullptr;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const bool in = full_trip || row0 + r < rows;
      const T* xr = in ? xb + r * ld_x : x + (rows - 1) * ld_x;
      const MT* mr = HAS_MASK ? (in ? mb + r * ld_m : mask + (rows - 1) * ld_m) : nullptr;
      // last live column (inclusive) under the causal rule; -1 if none; and
      // the end of the written columns
      int limit = cols - 1, we = cols;
      if (q > 0) {
        int pos = pos0 + r;
        if (pos >= q) pos = q >= R ? pos - q : pos % q;
        limit = pos + coff;
        if (trim_shift >= 0) we = (((pos >> trim_shift) + 1) << trim_shift) + coff;
      }
      lim[r] = limit < cols - 1 ? (limit < -1 ? -1 : limit) : cols - 1;
      wend[r] = we < cols ? (we < 0 ? 0 : we) : cols;
      int h = 0, be = cols;
      if constexpr (SHIFT) {
        const int phase = int(reinterpret_cast<uintptr_t>(xr) & 15) / int(sizeof(T));
        h = (V - phase) & (V - 1);
        be = h + ((cols - h) / V) * V;
      }
      hh[r] = h;
      bend[r] = be;
      // vectors past lim (or past the body) are not read: their address is
      // clamped onto the vector holding the last body column to read
      // (fetched by a live lane), then masked
      const int lc = SHIFT && be - 1 < lim[r] ? be - 1 : lim[r];
      const int limv = SHIFT ? (lc < h ? h : h + ((lc - h) / V) * V) : (lc < 0 ? 0 : (lc / V) * V);
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = h + (k * kThreads + tid) * V;
        const int cl = c0 <= lc ? c0 : limv;
        rx[r][k].load(xr + cl);
        if constexpr (HAS_MASK) rm[r][k].load(mr + cl);
      }
      if constexpr (SHIFT) {
        const int nx = cols - (be - h);
        const int ce = tid < nx ? (tid < h ? tid : be - h + tid) : 0;
        ex[r] = xr[ce];
        if constexpr (HAS_MASK) em[r] = mr[ce];
      }
    }
    if (LOOP && q > 0) {
      pos0 += step_mod;
      if (pos0 >= q) pos0 -= q;
    }
    // keep every load of the trip ahead of the first use (one HBM round trip)
    __builtin_amdgcn_sched_barrier(0);

    // logits a = x * scale + mask (-inf past lim, and past the body); ae:
    // the extra element's (SHIFT)
    float a[R][EPT], ae[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if constexpr (SHIFT) {
        const int nx = cols - (bend[r] - hh[r]);
        const int ce = tid < hh[r] ? tid : bend[r] - hh[r] + tid;
        float xv = raw_f32(ex[r]) * scale;
        if constexpr (HAS_MASK) xv += raw_f32(em[r]);
        ae[r] = tid < nx && ce <= lim[r] ? xv : -INFINITY;
      }
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c0 = hh[r] + (k * kThreads + tid) * V;
        float xv[V];
        rx[r][k].unpack(xv);
        if constexpr (HAS_MASK) {
          float mv[V];
          rm[r][k].unpack(mv);
#pragma unroll
          for (int i = 0; i < V; ++i) xv[i] = fmaf(xv[i], scale, mv[i]);
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i) xv[i] *= scale;
        }
        if (whole) {
#pragma unroll
          for (int i = 0; i < V; ++i) a[r][k * V + i] = xv[i];
        } else {
#pragma unroll
          for (int i = 0; i < V; ++i)
            a[r][k * V + i] = (c0 + i <= lim[r] && (!SHIFT || c0 < bend[r])) ? xv[i] : -INFINITY;
        }
      }
    }

    // f[r]: the factor that turns the stored exponentials into probabilities
    float f[R];
    if constexpr (W == 1) {
      // One-wave rows: a max all-reduce, exponentials against the row max,
      // a sum all-reduce.  Two cheap shuffle sequences instead of one of
      // (max, sum) pairs, whose every combine costs an exp2 -- with only
      // EPT * R elements per lane that combine dominated the ALU work.
      Multi<MaxF, R> mx;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float m = SHIFT ? ae[r] : -INFINITY;
#pragma unroll
        for (int i = 0; i < EPT; ++i) m = fmaxf(m, a[r][i]);
        mx.p[r].m = m;
      }
      mx = wave_allreduce(mx);
      Multi<SumP, R> sm;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        // exp((a - M)) as exp2((a - M) log2 e), the difference first: exact
        // near the maximum at any magnitude (a row masked with the most
        // negative finite value included); an all-masked row keeps M = 0
        // (its exponentials are exp2(-inf) = 0)
        const float ms = mx.p[r].m == -INFINITY ? 0.f : mx.p[r].m;
        float d = 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          a[r][i] = __builtin_amdgcn_exp2f((a[r][i] - ms) * kLog2e);
          d += a[r][i];
        }
        if constexpr (SHIFT) {
          ae[r] = __builtin_amdgcn_exp2f((ae[r] - ms) * kLog2e);
          d += ae[r];
        }
        sm.p[r].s = d;
      }
      sm = wave_allreduce(sm);
#pragma unroll
      for (int r = 0; r < R; ++r)
        f[r] = sm.p[r].s > 0.f ? __builtin_amdgcn_rcpf(sm.p[r].s) : 0.f;   // D >= 1 when live
    } else {
      // Multi-wave rows: local (m, d) per thread with the exponentials
      // exp2((a - m) log2 e) kept in a[], one all-reduce of the pairs across
      // waves
      using P = Multi<MaxSumP, R>;
      P part;
      bool empty[R];
      float ml2[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float m = SHIFT ? ae[r] : -INFINITY;
#pragma unroll
        for (int i = 0; i < EPT; ++i) m = fmaxf(m, a[r][i]);
        empty[r] = (m == -INFINITY);
        ml2[r] = empty[r] ? 0.f : m;   // the slice's max (0 for an all-masked slice)
        float d = 0.f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
          a[r][i] = __builtin_amdgcn_exp2f((a[r][i] - ml2[r]) * kLog2e);   // exp2(-inf) = 0
          d += a[r][i];
        }
        if constexpr (SHIFT) {
          ae[r] = __builtin_amdgcn_exp2f((ae[r] - ml2[r]) * kLog2e);
          d += ae[r];
        }
        part.p[r] = MaxSumP{empty[r] ? -INFINITY : ml2[r], d};
      }
      const P tot = group_allreduce<W>(part, lds[parity], wave, lane);
      parity ^= 1;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        // a slice with no live element contributes zeros (and must not form
        // 0*inf); a fully masked row has M = -inf and comes out all zeros
        const MaxSumP p = tot.p[r];
        f[r] = (empty[r] || p.m == -INFINITY) ? 0.f
                                              : __builtin_amdgcn_exp2f((ml2[r] - p.m) * kLog2e) / p.d;
      }
    }

    T* yb = y + row0 * ld_y;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (full_trip || row0 + r < rows) {
        T* yr = yb + r * ld_y;
        const int send = SHIFT && bend[r] < wend[r] ? bend[r] : wend[r];
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int c0 = hh[r] + (k * kThreads + tid) * V;
          float o[V];
#pragma unroll
          for (int i = 0; i < V; ++i) o[i] = a[r][k * V + i] * f[r];
          if (store_all) stv<T, V>(yr + c0, o);
          else store_until(yr, c0, send, o);
        }
        if constexpr (SHIFT) {
          const int nx = cols - (bend[r] - hh[r]);
          const int ce = tid < hh[r] ? tid : bend[r] - hh[r] + tid;
          if (tid < nx && ce < wend[r]) {
            const float o = ae[r] * f[r];
            stv<T, 1>(yr + ce, &o);
          }
        }
      }
    }
    if constexpr (!LOOP) break;
  }
}

// Rows longer than the register-resident capacity, with a row cache: one
// block of 16 waves per row keeps the exponentials of its first 64*16*CL
// columns in LDS (fp32, CL per lane) and of the next 64*16*CR columns in
// registers, so those columns are read from HBM once; with TAIL, the `tail`
// slots per lane past both are streamed: read once for the running (m, d)
// and again for the outputs.  Pass 1 runs one online (m, d) per lane over the LDS part,
// the register part and the tail, combined once across the block; each
// cached slot group keeps exp(a - mg), mg the lane's running max after the
// group.  Pass 2 writes exp(a - M) / D as e * exp(mg - M) / D from the
// registers and from LDS (one product per element), and recomputes it for
// the re-read tail.
// Each lane reads back only the LDS words it wrote, so the cache needs no
// barrier.  One block per compute unit holds one row at a time, so the loads
// of the next row's first slot groups are issued before the block-wide
// combine: they are in flight while this row's outputs are written.
template <typename T, typename MT, bool HAS_MASK, bool VEC, bool SHIFT, int CL, int CR, bool TAIL>
__global__ __launch_bounds__(1024) void softmax_cached_kernel(
    const T* __restrict__ x, int64_t ld_x, const MT* __restrict__ mask, int64_t ld_m, T* y,
    int64_t ld_y, int64_t rows, int cols, float scale, int64_t q_len, int trim_shift, int tail) {
  constexpr int W = 16, kThreads = 64 * W;
  constexpr int V = VEC || SHIFT ? Elem<T>::kVec : 1;   // elements per slot and lane
  constexpr int NL = CL / V, NR = CR / V, NS = NL + NR;   // vector slots per lane
  static_assert(CL % V == 0 && CR % V == 0 && CL % 4 == 0, "cache parts are whole vectors");
  // cached slots go in groups of G (about FS_SM_CACHE_GROUP_WORDS raw
  // registers each) with the loads of the next AH groups in flight
  constexpr int kWords = Raw<T, V>::kWords + (HAS_MASK ? Raw<MT, V>::kWords : 0);
  constexpr int G0 = kWords >= FS_SM_CACHE_GROUP_WORDS ? 1 : FS_SM_CACHE_GROUP_WORDS / kWords;
  constexpr int G = V > 1 || G0 < 4 ? G0 : 4;   // element-wise slots: groups of 4
  constexpr int NG = NS / G, AH = FS_SM_CACHE_AHEAD, R = AH + 1;
  static_assert(NL % G == 0 && NR % G == 0, "slot groups split the cache parts");
  __shared__ f32x4 cache[CL / 4][kThreads];
  __shared__ MaxSumP lds[2][W];
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int nslots = (cols + kThreads * V - 1) / (kThreads * V);   // slots the row uses
  int parity = 0;

  // per-row context: row pointers, last live column (causal rule), end of
  // the written columns (trimmed causal rows).  With SHIFT the slots cover
  // the row's aligned body [h, bend), whole 16-byte units, and its h head
  // and cols - bend tail elements (at most 2 V - 2) are extra elements of
  // the first lanes; lim, limv and wendb then refer to the body
  struct Row {
    const T* xr;
    const MT* mr;
    int lim, limv, wend, wendb, h, bend, lime;
  };
  auto row_ctx = [&](int64_t row, int64_t pos) {
    Row c;
    c.xr = x + row * ld_x;
    c.mr = HAS_MASK ? mask + row * ld_m : nullptr;
    c.h = 0;
    c.bend = cols;
    if constexpr (SHIFT) {
      const int phase = int(reinterpret_cast<uintptr_t>(c.xr) & 15) / int(sizeof(T));
      c.h = (V - phase) % V;
      c.bend = c.h + ((cols - c.h) / V) * V;
    }
    const int64_t limit = q_len > 0 ? pos + (cols - q_len) : int64_t(cols) - 1;
    c.lime = int(limit < int64_t(cols) - 1 ? (limit < -1 ? -1 : limit) : int64_t(cols) - 1);
    c.lim = c.lime < c.bend - 1 ? c.lime : c.bend - 1;
    c.limv = c.lim < c.h ? c.h : c.h + ((c.lim - c.h) / V) * V;
    int64_t we = cols;
    if (q_len > 0 && trim_shift >= 0)
      we = (((pos >> trim_shift) + 1) << trim_shift) + (cols - q_len);
    c.wend = int(we < cols ? (we < 0 ? 0 : we) : cols);
    c.wendb = c.wend < c.bend ? c.wend : c.bend;
    return c;
  };
  // loads of a slot, clamped in bounds past the row's last live column
  auto load = [&](const Row& c, int lt, int slot, Raw<T, V>& rx, Raw<MT, V>& rm) {
    const int c0 = c.h + (slot * kThreads + lt) * V;
    const int cl = c0 <= c.lim ? c0 : c.limv;
    rx.load(c.xr + cl);
    if constexpr (HAS_MASK) rm.load(c.mr + cl);
  };
  Raw<T, V> rx[R][G];
  Raw<MT, V> rm[R][G];
  // the first AH slot groups of a row.  Every load of the kernel is issued
  // unconditionally (addresses past the live columns are clamped in bounds,
  // and the row after the last is replaced by the last): with no branch
  // around a load, the waits for each group count exactly the loads issued
  // after it
  auto prime = [&](const Row& c, int lt) {
#pragma unroll
    for (int g = 0; g < AH && g < NG; ++g) {
#pragma unroll
      for (int k = 0; k < G; ++k) load(c, lt, g * G + k, rx[g][k], rm[g][k]);
    }
  };

  // causal position row mod q_len, advanced by the grid stride
  const int64_t step_mod = q_len > 0 ? int64_t(gridDim.x) % q_len : 0;
  int64_t pos = q_len > 0 ? int64_t(blockIdx.x) % q_len : 0;
  Row cur = row_ctx(blockIdx.x, pos);
  prime(cur, tid);

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    // the lane index is re-read per row (an empty asm) so that per-lane
    // offsets and column tests are recomputed, not kept in registers
    // across rows
    int lt = tid;
    asm volatile("" : "+v"(lt));
    auto col_of = [&](int slot) { return cur.h + (slot * kThreads + lt) * V; };
    // SHIFT: the lane's extra element (head or tail), loaded first
    const int nx = cur.h + (cols - cur.bend);
    const bool has_x = SHIFT && lt < nx;
    const int ce = has_x ? (lt < cur.h ? lt : cur.bend + (lt - cur.h)) : 0;
    Raw<T, 1> ex;
    Raw<MT, 1> em;
    if constexpr (SHIFT) {
      ex.load(cur.xr + ce);
      if constexpr (HAS_MASK) em.load(cur.mr + ce);
    }
    auto logit = [&](int slot, const Raw<T, V>& rxs, const Raw<MT, V>& rms, float* a) {
      const int c0 = col_of(slot);
      float xv[V];
      rxs.unpack(xv);
      if constexpr (HAS_MASK) {
        float mv[V];
        rms.unpack(mv);
#pragma unroll
        for (int i = 0; i < V; ++i) xv[i] = fmaf(xv[i], scale, mv[i]);
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) xv[i] *= scale;
      }
#pragma unroll
      for (int i = 0; i < V; ++i) a[i] = (c0 + i <= cur.lim) ? xv[i] : -INFINITY;
    };
    // merge N logits into the lane's running (m, d); with KEEP the logits
    // are replaced by their exponentials exp2((a - m) log2 e), m the running
    // max after this merge (returned), so pass 2 needs one product per
    // element; differences are taken before the scaling (exact near the
    // maximum at any magnitude)
    float mrun = -INFINITY, drun = 0.f;
    auto absorb = [&](auto kn, auto keep, float* a) {
      constexpr int N = decltype(kn)::value;
      float tm = -INFINITY;
#pragma unroll
      for (int i = 0; i < N; ++i) tm = fmaxf(tm, a[i]);
      const float mnew = fmaxf(mrun, tm);
      const float msafe = mnew == -INFINITY ? 0.f : mnew;
      float dt = 0.f;
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const float e = __builtin_amdgcn_exp2f((a[i] - msafe) * kLog2e);
        dt += e;
        if constexpr (decltype(keep)::value) a[i] = e;
      }
      drun = fmaf(drun, __builtin_amdgcn_exp2f((mrun - msafe) * kLog2e), dt);   // 2^-inf = 0
      mrun = mnew;
      return msafe;
    };
    using Keep = std::true_type;
    using Drop = std::false_type;
    // the tail slots NS ... NS + tail - 1, one ahead: a slot's loads are in
    // flight while the previous slot is used.  Loads of slots past the row
    // are clamped in bounds (their logits are -inf and they store nothing).
    auto over_tail = [&](auto use) {
      Raw<T, V> tx[2];
      Raw<MT, V> tm[2];
      load(cur, lt, NS, tx[0], tm[0]);
      for (int j = 0; j < tail; j += 2) {
        load(cur, lt, NS + j + 1, tx[1], tm[1]);
        __builtin_amdgcn_sched_barrier(0);
        use(NS + j, tx[0], tm[0]);
        load(cur, lt, NS + j + 2, tx[0], tm[0]);
        __builtin_amdgcn_sched_barrier(0);
        if (j + 1 < tail) use(NS + j + 1, tx[1], tm[1]);
      }
    };

    // pass 1: LDS part, register part (the first AH groups were issued
    // before), tail.  The cached parts keep exponentials, each group's
    // relative to its own running max mg
    float ar[CR], mg[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + AH < NG) {
#pragma unroll
        for (int k = 0; k < G; ++k) load(cur, lt, (g + AH) * G + k, rx[(g + AH) % R][k], rm[(g + AH) % R][k]);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (g * G < nslots) {
        float a[G * V];
#pragma unroll
        for (int k = 0; k < G; ++k) logit(g * G + k, rx[g % R][k], rm[g % R][k], a + k * V);
        mg[g] = absorb(std::integral_constant<int, G * V>{}, Keep{}, a);
        if (g * G < NL) {
#pragma unroll
          for (int k = 0; k < G * V / 4; ++k)
            cache[g * G * V / 4 + k][lt] = f32x4{a[4 * k], a[4 * k + 1], a[4 * k + 2], a[4 * k + 3]};
        } else {
#pragma unroll
          for (int i = 0; i < G * V; ++i) ar[g * G * V - CL + i] = a[i];
        }
      }
    }
    if constexpr (TAIL) {
      over_tail([&](int slot, const Raw<T, V>& rxs, const Raw<MT, V>& rms) {
        float a[V];
        logit(slot, rxs, rms, a);
        absorb(std::integral_constant<int, V>{}, Drop{}, a);
      });
    }
    float ax = -INFINITY;   // the extra element's logit
    if constexpr (SHIFT) {
      float xv, mv = 0.f;
      ex.unpack(&xv);
      if constexpr (HAS_MASK) em.unpack(&mv);
      const float v = HAS_MASK ? fmaf(xv, scale, mv) : xv * scale;
      ax = has_x && ce <= cur.lime ? v : -INFINITY;
      absorb(std::integral_constant<int, 1>{}, Drop{}, &ax);
    }

    // the next row's first slot groups, in flight from here on
    const int64_t next = row + gridDim.x;
    int64_t npos = pos + step_mod;
    if (npos >= q_len) npos -= q_len;
    const Row nxt = row_ctx(next < rows ? next : rows - 1, npos);
    prime(nxt, lt);

    const MaxSumP p = group_allreduce<W>(MaxSumP{mrun, drun}, lds[parity], wave, lane);
    parity ^= 1;
    const bool empty = p.m == -INFINITY;
    const float M = empty ? 0.f : p.m;
    const float inv_d = empty ? 0.f : 1.f / p.d;

    asm volatile("" : "+v"(lt));   // pass 2 recomputes its column tests too
    // pass 2: outputs (register part first, which frees its registers)
    T* yr = y + row * ld_y;
    auto emit = [&](int slot, const float* a) {
      float o[V];
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] = __builtin_amdgcn_exp2f((a[i] - M) * kLog2e) * inv_d;
      store_until(yr, col_of(slot), cur.wendb, o);
    };
    // a cached slot: its exponentials times 2^(mg - M) / D (at most 1 / D)
    auto emit_e = [&](int slot, const float* e) {
      const float f = __builtin_amdgcn_exp2f((mg[slot / G] - M) * kLog2e) * inv_d;
      float o[V];
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] = e[i] * f;
      store_until(yr, col_of(slot), cur.wendb, o);
    };
#pragma unroll
    for (int s = 0; s < NR; ++s)
      if (NL + s < nslots) emit_e(NL + s, ar + s * V);
#pragma unroll
    for (int s = 0; s < NL; ++s) {
      if (s >= nslots) continue;
      float e[V];
      if constexpr (V >= 4) {
#pragma unroll
        for (int k = 0; k < V / 4; ++k) {
          const f32x4 v = cache[s * (V / 4) + k][lt];
          e[4 * k] = v.x; e[4 * k + 1] = v.y; e[4 * k + 2] = v.z; e[4 * k + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) e[i] = cache[(s * V + i) / 4][lt][(s * V + i) % 4];
      }
      emit_e(s, e);
    }
    if constexpr (TAIL) {
      over_tail([&](int slot, const Raw<T, V>& rxs, const Raw<MT, V>& rms) {
        float a[V];
        logit(slot, rxs, rms, a);
        emit(slot, a);
      });
    }
    if constexpr (SHIFT) {
      if (has_x && ce < cur.wend) {
        const float o = __builtin_amdgcn_exp2f((ax - M) * kLog2e) * inv_d;
        stv<T, 1>(yr + ce, &o);
      }
    }
    cur = nxt;
    pos = npos;
  }
}

// rows batched per group: enough that a one-wave group handles about
// FS_SM_BATCH_ELEMS elements per lane per trip
template <int W, int EPT>
struct RowsPerGroup {
  static constexpr int value = (W == 1 && EPT < FS_SM_BATCH_ELEMS) ? FS_SM_BATCH_ELEMS / EPT : 1;
};

template <typename T, typename MT, bool HAS_MASK, bool VEC>
hipError_t dispatch(const SoftmaxArgs& a, int cus, hipStream_t s) {
  constexpr int V = VEC ? Elem<T>::kVec : 1;
  // smallest capacity >= cols; the vector path needs EPT >= V
  const int64_t c = a.cols;
  // kern_loop walks rows with a grid stride; kern_one (same arithmetic, one
  // trip per row group) is launched when the grid holds every row group
  auto launch = [&](auto kern_loop, auto kern_one, int threads, int rows_per_block,
                    int blocks_per_cu) {
    int64_t want = (a.rows + rows_per_block - 1) / rows_per_block;
    int64_t cap = int64_t(cus) * blocks_per_cu * FS_SM_GRID_SCALE / 4;
    int grid = int(want < cap ? want : cap);
    if (grid < 1) grid = 1;
    auto go = [&](auto kern) {
      hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s, static_cast<const T*>(a.x),
                         a.ld_x, static_cast<const MT*>(a.mask), a.ld_mask, a.rows,
                         a.causal_q_len, int(a.cols), a.trim_shift, a.scale,
                         static_cast<T*>(a.y), a.ld_y);
      return hipGetLastError();
    };
    return want <= cap ? go(kern_one) : go(kern_loop);
  };
  // Variant ladder, in order: the first rung with at least min_w waves per row
  // and a row capacity 64 * W * EPT >= cols is launched.
  const int min_w = c >= FS_SM_SPLIT_COLS ? FS_SM_MIN_WAVES : 1;
  // the register-resident kernel keeps causal positions in 32 bits
  const bool small_q = a.causal_q_len < (int64_t(1) << 30);
  // rows that share a 16-byte phase: the vector ladder over each row's
  // aligned body (a row of c columns has at most c / V whole vectors in it)
  if constexpr (!VEC && (!HAS_MASK || sizeof(MT) == sizeof(T) || sizeof(MT) == 1)) {
    if (a.shifted && c <= FS_SM_SHIFT_REG_COLS) {
      constexpr int VS = Elem<T>::kVec;
#define FS_SMS(Wv, E, Gv, BPC)                                                                  \
  if (small_q && Wv >= min_w && c <= int64_t(64) * Wv * E)                                      \
    return launch(softmax_kernel<T, MT, HAS_MASK, Wv, E, false, true, Gv, RowsPerGroup<Wv, E>::value, true>, \
                  softmax_kernel<T, MT, HAS_MASK, Wv, E, false, true, Gv, RowsPerGroup<Wv, E>::value, true>, \
                  64 * Wv * Gv, Gv * RowsPerGroup<Wv, E>::value, BPC);
      if constexpr (VS <= 4) { FS_SMS(1, 4, 4, 8) }
      FS_SMS(1, 8, 4, 8)
      FS_SMS(1, 16, 4, 8)
      FS_SMS(1, 32, 4, 8)
      FS_SMS(1, 64, 4, 8)
      FS_SMS(2, 32, 1, 16)
      FS_SMS(2, 64, 1, 16)
      FS_SMS(4, 16, 1, 8)
      FS_SMS(4, 32, 1, 8)
      FS_SMS(4, 64, 1, 8)
      FS_SMS(8, 8, 1, 4)
      FS_SMS(8, 16, 1, 4)
      FS_SMS(8, 32, 1, 4)
      FS_SMS(16, 24, 1, 1)
      FS_SMS(16, 32, 1, 1)
#undef FS_SMS
    }
  }
#define FS_SM(Wv, E, Gv, BPC)                                                       \
  if (small_q && Wv >= min_w && c <= int64_t(64) * Wv * E &&                     \
      (VEC || c <= (a.shifted ? FS_SM_SHIFT_REG_COLS : FS_SM_ELEMENTWISE_REG_COLS)))  \
    return launch(softmax_kernel<T, MT, HAS_MASK, Wv, E, VEC, false, Gv, RowsPerGroup<Wv, E>::value, true>, \
                  softmax_kernel<T, MT, HAS_MASK, Wv, E, VEC, false, Gv, RowsPerGroup<Wv, E>::value,  \
                                 !VEC || Wv < FS_SM_ONE_TRIP_MIN_W>,                                   \
                  64 * Wv * Gv, Gv * RowsPerGroup<Wv, E>::value, BPC);
  if constexpr (V <= 1) { FS_SM(1, 1, 4, 8) }
  if constexpr (V <= 2) { FS_SM(1, 2, 4, 8) }
  if constexpr (V <= 4) { FS_SM(1, 4, 4, 8) }
  FS_SM(1, 8, 4, 8)
  FS_SM(1, 16, 4, 8)
  FS_SM(1, 32, 4, 8)
  FS_SM(1, 64, 4, 8)
  FS_SM(2, 32, 1, 16)
  FS_SM(2, 64, 1, 16)
  FS_SM(4, 16, 1, 8)
  FS_SM(4, 32, 1, 8)
  FS_SM(4, 64, 1, 8)
  FS_SM(8, 8, 1, 4)
  FS_SM(8, 16, 1, 4)
  FS_SM(8, 32, 1, 4)
  FS_SM(16, 24, 1, 1)
  FS_SM(16, 32, 1, 1)
#undef FS_SM
  // longer rows (and causal rows with q_len >= 2^30): row cache in LDS and
  // registers, the columns past it streamed; one 16-wave block per compute
  // unit, 16-byte or element-wise slots
  {
    constexpr int CL = 32, CR = 32;
    constexpr int64_t kCached = int64_t(1024) * (CL + CR);
    auto go = [&](auto kern, int tail) {
      const int64_t grid = a.rows < cus ? a.rows : cus;
      hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(1024), 0, s, static_cast<const T*>(a.x),
                         a.ld_x, static_cast<const MT*>(a.mask), a.ld_mask, static_cast<T*>(a.y),
                         a.ld_y, a.rows, int(a.cols), a.scale, a.causal_q_len, a.trim_shift, tail);
      return hipGetLastError();
    };
    constexpr int64_t kSlot = int64_t(1024) * V;
    if constexpr (!VEC && (!HAS_MASK || sizeof(MT) == sizeof(T) || sizeof(MT) == 1)) {
      if (a.shifted) {
        // 16-byte slots over each row's aligned body
        constexpr int64_t kVSlot = int64_t(1024) * Elem<T>::kVec;
        if (c <= kCached) return go(softmax_cached_kernel<T, MT, HAS_MASK, false, true, CL, CR, false>, 0);
        return go(softmax_cached_kernel<T, MT, HAS_MASK, false, true, CL, CR, true>,
                  int((c - kCached + kVSlot - 1) / kVSlot));
      }
    }
    if (c <= kCached) return go(softmax_cached_kernel<T, MT, HAS_MASK, VEC, false, CL, CR, false>, 0);
    return go(softmax_cached_kernel<T, MT, HAS_MASK, VEC, false, CL, CR, true>,
              int((c - kCached + kSlot - 1) / kSlot));
  }
}

template <typename T, typename MT>
hipError_t by_vec(const SoftmaxArgs& a, int cus, hipStream_t s) {
  if (a.mask == nullptr)
    return a.vec ? dispatch<T, T, false, true>(a, cus, s) : dispatch<T, T, false, false>(a, cus, s);
  return a.vec ? dispatch<T, MT, true, true>(a, cus, s) : dispatch<T, MT, true, false>(a, cus, s);
}

}  // namespace

hipError_t launch_softmax(const SoftmaxArgs& a, int cus, hipStream_t s) {
  if (a.dtype == FS_BF16) {
    if (a.mask_dtype == FS_U8) return by_vec<uint16_t, uint8_t>(a, cus, s);
    if (a.mask_dtype == FS_BF16) return by_vec<uint16_t, uint16_t>(a, cus, s);
    return by_vec<uint16_t, float>(a, cus, s);
  }
  if (a.mask_dtype == FS_U8) return by_vec<float, uint8_t>(a, cus, s);
  if (a.mask_dtype == FS_BF16) return by_vec<float, uint16_t>(a, cus, s);
  return by_vec<float, float>(a, cus, s);
}

}  // namespace fs
