// Calibration copy: the achievable HBM bandwidth of a plain streaming kernel
// on this device (16-byte non-temporal loads and stores), and the reference
// against which hardware byte counters are scaled.  Also the batched strided
// copy that moves activations between token-major and head-major layouts.
#include <type_traits>

#include "device_common.hpp"
#include "launch.hpp"

#ifndef FS_COPY_CHUNK
#define FS_COPY_CHUNK 4
#endif
#ifndef FS_COPY_BLOCKS_PER_CU
#define FS_COPY_BLOCKS_PER_CU 32
#endif
#ifndef FS_STRIDED_UNROLL
#define FS_STRIDED_UNROLL 4
#endif
#ifndef FS_STRIDED_TILE_UNITS
#define FS_STRIDED_TILE_UNITS 1024   // at most 256 * kMaxItems
#endif
#ifndef FS_STRIDED_BLOCKS_PER_CU
#define FS_STRIDED_BLOCKS_PER_CU 8
#endif

namespace fs {
namespace {

constexpr int kMaxItems = 8;   // items per thread per tile of the strided copy
static_assert(FS_STRIDED_TILE_UNITS <= 256 * kMaxItems, "tile larger than a block's items");

// Each wave copies whole chunks of 64 * C vectors (C 16-byte accesses per
// lane, all loads issued before the stores) and strides over the chunks; the
// vectors after the last whole chunk are copied one per thread.  Chunks of
// contiguous kilobytes per wave measured faster than a grid-stride loop of
// single vectors (5.9 against 5.4 TB/s for a 1 GiB copy on MI355X).
template <int C>
__global__ __launch_bounds__(256) void copy128_kernel(const u32x4* __restrict__ src,
                                                       u32x4* __restrict__ dst, int64_t n) {
  constexpr int64_t kChunk = int64_t(64) * C;
  const int lane = threadIdx.x % 64;
  const int64_t wave = int64_t(blockIdx.x) * 4 + threadIdx.x / 64;
  const int64_t waves = int64_t(gridDim.x) * 4;
  const int64_t nchunks = n / kChunk;
  for (int64_t c = wave; c < nchunks; c += waves) {
    const int64_t base = c * kChunk + lane;
    u32x4 v[C];
#pragma unroll
    for (int k = 0; k < C; ++k) v[k] = ld128<true>(src + base + k * 64);
#pragma unroll
    for (int k = 0; k < C; ++k) st128<true>(dst + base + k * 64, v[k]);
  }
  for (int64_t i = nchunks * kChunk + int64_t(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * 256)
    st128<true>(dst + i, ld128<true>(src + i));
}

__global__ __launch_bounds__(256) void copy8_kernel(const uint8_t* __restrict__ src,
                                                     uint8_t* __restrict__ dst, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
    dst[i] = src[i];
}


// Batched strided 2-D copy (a layout transform such as a head split or
// merge): dst[b, r, c] = src[b, r, c].  A block copies tiles of rb rows; the
// items of a tile are ordered (row, batch, unit) with the unit (16 bytes, or
// one element) fastest, so the items of one row of a head split read one
// contiguous source row and write whole 128-byte segments.  Every tile has
// the same shape, so each thread splits its K items of a tile into (row,
// batch, unit) once, before the tile loop, and keeps their offsets relative
// to the tile's first row; the loop itself has no division.  All K loads of
// a tile are issued before its stores (items past the last row re-read the
// tile's first item and are not stored).
template <typename U, int K>
__global__ __launch_bounds__(256) void copy_strided_kernel(
    const U* __restrict__ src, int64_t ld_s, int64_t st_s, U* __restrict__ dst, int64_t ld_d,
    int64_t st_d, int64_t rows, int upr, int per_row, int rb) {
  const int items = rb * per_row;
  int64_t rel_s[K], rel_d[K];
  int row_of[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int i0 = int(threadIdx.x) + k * 256;
    const int i = i0 < items ? i0 : items - 1;
    const int rr = i / per_row;
    const int rem = i - rr * per_row;
    const int bb = rem / upr;
    const int c = rem - bb * upr;
    rel_s[k] = bb * st_s + rr * ld_s + c;
    rel_d[k] = bb * st_d + rr * ld_d + c;
    row_of[k] = i0 < items ? rr : rb;     // rb: never stored
  }
  for (int64_t r0 = int64_t(blockIdx.x) * rb; r0 < rows; r0 += int64_t(gridDim.x) * rb) {
    const U* s0 = src + r0 * ld_s;
    U* d0 = dst + r0 * ld_d;
    const int live_rows = int(rows - r0 < rb ? rows - r0 : rb);
    U v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) v[k] = s0[row_of[k] < live_rows ? rel_s[k] : 0];
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (row_of[k] < live_rows) d0[rel_d[k]] = v[k];
  }
}

// Rows of more than 256 * kMaxItems units: one row per block, the items of
// the row in a loop.
template <typename U>
__global__ __launch_bounds__(256) void copy_strided_rows_kernel(
    const U* __restrict__ src, int64_t ld_s, int64_t st_s, U* __restrict__ dst, int64_t ld_d,
    int64_t st_d, int64_t rows, int upr, int per_row) {
  constexpr int UN = FS_STRIDED_UNROLL;
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    for (int j0 = threadIdx.x; j0 < per_row; j0 += 256 * UN) {
      U v[UN];
      int64_t di[UN];
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        int j = j0 + u * 256;
        j = j < per_row ? j : per_row - 1;
        const int bb = j / upr;
        const int c = j - bb * upr;
        v[u] = src[bb * st_s + r * ld_s + c];
        di[u] = bb * st_d + r * ld_d + c;
      }
#pragma unroll
      for (int u = 0; u < UN; ++u)
        if (j0 + u * 256 < per_row) dst[di[u]] = v[u];
    }
  }
}

}  // namespace

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int cus, hipStream_t s) {
  const bool vec = (reinterpret_cast<uintptr_t>(src) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(dst) % 16 == 0) && (bytes % 16 == 0);
  const int64_t n = vec ? bytes / 16 : bytes;
  int64_t grid = (n + 255) / 256;
  const int64_t cap = int64_t(cus) * FS_COPY_BLOCKS_PER_CU;
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  if (vec)
    hipLaunchKernelGGL(copy128_kernel<FS_COPY_CHUNK>, dim3(unsigned(grid)), dim3(256), 0, s,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), n);
  else
    hipLaunchKernelGGL(copy8_kernel, dim3(unsigned(grid)), dim3(256), 0, s,
                       static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), n);
  return hipGetLastError();
}

hipError_t launch_copy_strided(const CopyStridedArgs& a, int cus, hipStream_t s) {
  // units: 16-byte vectors when every address, stride and row is a multiple
  // of 16 bytes, else single elements
  const int es = a.es;
  const bool vec = (reinterpret_cast<uintptr_t>(a.src) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(a.dst) % 16 == 0) && (a.cols * es) % 16 == 0 &&
                   (a.ld_src * es) % 16 == 0 && (a.ld_dst * es) % 16 == 0 &&
                   (a.stride_src * es) % 16 == 0 && (a.stride_dst * es) % 16 == 0;
  const int ue = vec ? 16 : es;                      // bytes per unit
  const int upr = int(a.cols * es / ue);
  const int per_row = int(a.batch) * upr;
  const int64_t cap = int64_t(cus) * FS_STRIDED_BLOCKS_PER_CU;
  auto go = [&](auto* tag) {
    using U = std::remove_pointer_t<decltype(tag)>;
    const int64_t k = ue / es;                       // elements per unit
    const U* sp = static_cast<const U*>(a.src);
    U* dp = static_cast<U*>(a.dst);
    if (per_row > 256 * kMaxItems) {
      const int64_t grid = a.rows < cap ? a.rows : cap;
      hipLaunchKernelGGL(copy_strided_rows_kernel<U>, dim3(unsigned(grid)), dim3(256), 0, s, sp,
                         a.ld_src / k, a.stride_src / k, dp, a.ld_dst / k, a.stride_dst / k,
                         a.rows, upr, per_row);
      return hipGetLastError();
    }
    // rows per tile: as many as fill the tile's 256 * kMaxItems items
    int rb = FS_STRIDED_TILE_UNITS / per_row;
    if (rb < 1) rb = 1;
    if (int64_t(rb) > a.rows) rb = int(a.rows);
    const int items = rb * per_row;
    int64_t grid = (a.rows + rb - 1) / rb;
    if (grid > cap) grid = cap;
    auto launch = [&](auto kern) {
      hipLaunchKernelGGL(kern, dim3(unsigned(grid)), dim3(256), 0, s, sp, a.ld_src / k,
                         a.stride_src / k, dp, a.ld_dst / k, a.stride_dst / k, a.rows, upr,
                         per_row, rb);
      return hipGetLastError();
    };
    if (items <= 256) return launch(copy_strided_kernel<U, 1>);
    if (items <= 512) return launch(copy_strided_kernel<U, 2>);
    if (items <= 1024) return launch(copy_strided_kernel<U, 4>);
    return launch(copy_strided_kernel<U, kMaxItems>);
  };
  if (vec) return go(static_cast<u32x4*>(nullptr));
  if (es == 4) return go(static_cast<uint32_t*>(nullptr));
  return go(static_cast<uint16_t*>(nullptr));
}

}  // namespace fs
