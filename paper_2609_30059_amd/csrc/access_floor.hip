// Access-shape floors of the fused sub-kernels: a calibration library for the
// benchmark (not a sub-kernel; nothing in libfusedsub calls it).
//
// Each floor kernel moves exactly the compulsory bytes of one sub-kernel
// launch of the benchmark step, in that launch's shape: the same input and
// output streams, the same row geometry (16-byte vectors per lane, waves
// per row, rows per wave), the same causal read pattern and the same grid,
// with non-temporal 16-byte loads and stores as the sub-kernels use -- but
// none of the arithmetic: an output vector is the bitwise combination of the
// input vectors of its slot, and no statistic crosses lanes.  Its dispatch
// time is the time HBM needs for that access pattern, the floor the fused
// sub-kernel's own time is compared with.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(u32x4* p, const u32x4& v) { __builtin_nontemporal_store(v, p); }

// Row groups of W waves, G groups per block, R rows per group per trip, NV
// vectors per lane per row and stream.  A row is row_vecs = 64 * W * NV
// vectors of a [rows, ld] array of vectors; col_blocks > 1 splits each row's
// ld vectors into that many slabs of row_vecs, one slab per block (block b
// takes slab b % col_blocks), as the pointwise kernel does.  CAUSAL: row r
// reads its vectors up to (r mod q) / epv (lanes past it re-read that vector)
// and stores zeros past it.  LOOP: groups walk their trips with a grid
// stride; otherwise every group takes one trip.
template <int NIN, int NOUT, int W, int NV, int G, int R, bool CAUSAL, bool LOOP>
__global__ __launch_bounds__(64 * W * G) void floor_rows_kernel(
    const u32x4* __restrict__ in0, const u32x4* __restrict__ in1, u32x4* __restrict__ out0,
    u32x4* __restrict__ out1, int64_t rows, int64_t ld, int col_blocks, int q, int epv) {
  constexpr int kThreads = 64 * W;
  const int tid = threadIdx.x % kThreads;
  const int g = threadIdx.x / kThreads;
  const int cb = int(blockIdx.x % unsigned(col_blocks));
  const int64_t groups = int64_t(gridDim.x / unsigned(col_blocks)) * G;
  const int64_t col0 = int64_t(cb) * kThreads * NV;
  u32x4 keep = {0u, 0u, 0u, 0u};
  for (int64_t row0 = (int64_t(blockIdx.x / unsigned(col_blocks)) * G + g) * R; row0 < rows;
       row0 += groups * R) {
    u32x4 a[R][NV], b[R][NV];
    int lim[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t row = row0 + r < rows ? row0 + r : rows - 1;
      lim[r] = CAUSAL ? int(row % q) / epv : kThreads * NV;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int v = k * kThreads + tid;
        const int64_t at = row * ld + col0 + (CAUSAL && v > lim[r] ? lim[r] : v);
        if constexpr (NIN >= 1) a[r][k] = ld_nt(in0 + at);
        if constexpr (NIN >= 2) b[r][k] = ld_nt(in1 + at);
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t row = row0 + r;
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int v = k * kThreads + tid;
        u32x4 o = a[r][k];
        if constexpr (NIN >= 2) o ^= b[r][k];
        if (CAUSAL && v > lim[r]) o = u32x4{0u, 0u, 0u, 0u};
        if constexpr (NOUT == 0) {
          keep ^= o;
        } else if (row < rows) {
          st_nt(out0 + row * ld + col0 + v, o);
          if constexpr (NOUT >= 2) st_nt(out1 + row * ld + col0 + v, a[r][k]);
        }
      }
    }
    if constexpr (!LOOP) break;
  }
  // read-only floors: the loads stay live through a store that the data
  // never triggers (out0 holds at least one vector)
  if (NOUT == 0 && keep.x == 0x9e3779b9u && keep.y == 0x7f4a7c15u && keep.z == 0x2545f491u)
    out0[0] = keep;
}

struct Geometry {
  int nin, nout;
  int64_t rows, ld;   // vectors
};

// The benchmark step's launches, in the order of fsx_access_floor's shape
// argument: shapes and launch geometry of the sub-kernel each one mirrors.
constexpr Geometry kShapes[] = {
    {2, 1, 256, 256},        // 0 pointwise fp32 [256, 1024] + bias: one row per 4-wave block
    {2, 1, 262144, 256},     // 1 pointwise fp32 [262144, 1024]: 4 rows per trip, 16 blocks/CU
    {2, 1, 8192, 512},       // 2 softmax bf16 [8192, 4096] + mask: one row per 2-wave block
    {2, 2, 16384, 512},      // 3 LayerNorm + residual bf16 [16384, 4096]: one row per 2-wave block
    {1, 0, 8192, 1024},      // 4 GEMM epilogue bf16 C [8192, 8192]: one row per wave, 16-wave blocks
    {1, 1, 16384, 128},      // 5 block LN1 bf16 [16384, 1024]: one row per wave
    {1, 1, 262144, 64},      // 6 block causal softmax bf16 [32 * 16 * 512, 512]: 2 rows per wave
    {2, 2, 16384, 128},      // 7 block LN2 + residual bf16 [16384, 1024]: one row per wave
    {1, 1, 16384, 512},      // 8 block bias + GELU bf16 [16384, 4096]: two column slabs per row
    {2, 1, 8192, 256},       // 9 block residual add bf16 [16384, 1024] as 8192 chunks of 256 vectors
};
constexpr int kNumShapes = int(sizeof(kShapes) / sizeof(kShapes[0]));

template <typename K>
int go(K kern, int64_t grid, int threads, const Geometry& s, const u32x4* i0, const u32x4* i1,
       u32x4* o0, u32x4* o1, int col_blocks, int q, int epv, hipStream_t st) {
  hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(threads), 0, st, i0, i1, o0, o1, s.rows,
                     s.ld, col_blocks, q, epv);
  return int(hipGetLastError());
}

bool fits(const void* p, size_t bytes, int64_t need) {
  return p != nullptr && reinterpret_cast<uintptr_t>(p) % 16 == 0 && bytes >= size_t(need);
}

}  // namespace

// Launches the floor of step launch `shape` (0..9, see kShapes) on `stream`.
// Buffers are device pointers with their sizes in bytes: every input the
// shape reads and every output it writes must hold rows * ld vectors of 16
// bytes (the read-only shape 4 needs one vector of out0); unused pointers
// may be NULL.  Returns 0, -1 for a bad buffer, -2 for an unknown shape,
// -3 for cus < 1, or the HIP error of the launch.
extern "C" __attribute__((visibility("default"))) int fsx_access_floor(
    int shape, const void* in0, size_t in0_bytes, const void* in1, size_t in1_bytes, void* out0,
    size_t out0_bytes, void* out1, size_t out1_bytes, int cus, hipStream_t stream) {
  if (shape < 0 || shape >= kNumShapes) return -2;
  if (cus < 1) return -3;
  const Geometry& s = kShapes[shape];
  const int64_t need = s.rows * s.ld * 16;
  if (!fits(in0, in0_bytes, need)) return -1;
  if (s.nin >= 2 && !fits(in1, in1_bytes, need)) return -1;
  if (!fits(out0, out0_bytes, s.nout == 0 ? 16 : need)) return -1;
  if (s.nout >= 2 && !fits(out1, out1_bytes, need)) return -1;
  const u32x4* i0 = static_cast<const u32x4*>(in0);
  const u32x4* i1 = static_cast<const u32x4*>(s.nin >= 2 ? in1 : in0);
  u32x4* o0 = static_cast<u32x4*>(out0);
  u32x4* o1 = static_cast<u32x4*>(s.nout >= 2 ? out1 : out0);
  const int64_t cu = cus;
  switch (shape) {
    case 0: return go(floor_rows_kernel<2, 1, 4, 1, 1, 1, false, false>, s.rows, 256, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 1: return go(floor_rows_kernel<2, 1, 4, 1, 1, 4, false, true>, cu * 16, 256, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 2: return go(floor_rows_kernel<2, 1, 2, 4, 1, 1, false, false>, s.rows, 128, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 3: return go(floor_rows_kernel<2, 2, 2, 4, 1, 1, false, false>, s.rows, 128, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 4: return go(floor_rows_kernel<1, 0, 1, 16, 16, 1, false, false>, s.rows / 16, 1024, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 5: return go(floor_rows_kernel<1, 1, 1, 2, 4, 1, false, false>, s.rows / 4, 256, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 6: return go(floor_rows_kernel<1, 1, 1, 1, 4, 2, true, false>, s.rows / 8, 256, s, i0, i1, o0, o1, 1, 512, 8, stream);
    case 7: return go(floor_rows_kernel<2, 2, 1, 2, 4, 1, false, false>, s.rows / 4, 256, s, i0, i1, o0, o1, 1, 1, 1, stream);
    case 8: return go(floor_rows_kernel<1, 1, 4, 1, 1, 4, false, true>, cu * 16, 256, s, i0, i1, o0, o1, 2, 1, 1, stream);
    case 9: return go(floor_rows_kernel<2, 1, 1, 4, 4, 1, false, true>, cu * 4, 256, s, i0, i1, o0, o1, 1, 1, 1, stream);
  }
  return -2;
}

// Number of shapes (for the caller's own checks).
extern "C" __attribute__((visibility("default"))) int fsx_access_floor_shapes(void) {
  return kNumShapes;
}

// Bytes one launch of shape `shape` reads and writes (whole 16-byte vectors;
// the causal shape reads each row up to its last live vector), or -1 for an
// unknown shape: the caller compares them with the sub-kernel's compulsory
// bytes.
extern "C" __attribute__((visibility("default"))) int64_t fsx_access_floor_bytes(int shape) {
  if (shape < 0 || shape >= kNumShapes) return -1;
  const Geometry& s = kShapes[shape];
  int64_t read_vecs = s.rows * s.ld;
  if (shape == 6) {   // causal rows of 512 bf16 (8 per vector) in periods of 512 rows
    int64_t per_period = 0;
    for (int pos = 0; pos < 512; ++pos) per_period += pos / 8 + 1;
    read_vecs = s.rows / 512 * per_period;
  }
  return 16 * (read_vecs * s.nin + s.rows * s.ld * s.nout);
}
