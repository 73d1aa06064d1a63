// C ABI of libfusedsub: argument validation (host only, before any HIP call),
// choice of the 16-byte vector path, aliasing checks, and dispatch to the
// kernels.  The contract of every entry point is documented in fusedsub.h.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "fusedsub.h"
#include "launch.hpp"

namespace {

thread_local char g_msg[512] = "";

void clear_msg() { g_msg[0] = '\0'; }

fs_status fail(fs_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return st;
}

fs_status hip_fail(hipError_t e, const char* what) {
  return fail(FS_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), int(e));
}

// compute-unit count per device, filled on first use
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

fs_status device_cus(int* cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(FS_ERR_HIP, "device index %d out of range", dev);
  int v = g_cus[dev].load(std::memory_order_relaxed);
  if (v <= 0) {
    e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    if (v <= 0) v = 1;
    g_cus[dev].store(v, std::memory_order_relaxed);
  }
  *cus = v;
  return FS_OK;
}

int elem_size(fs_dtype d) { return d == FS_F32 ? 4 : d == FS_BF16 ? 2 : 1; }
// data dtypes; the byte mask FS_U8 is accepted by fs_row_softmax's mask only
bool dtype_ok(int d) { return d == FS_F32 || d == FS_BF16; }
int vec_width(fs_dtype d) { return 16 / elem_size(d); }

uintptr_t addr(const void* p) { return reinterpret_cast<uintptr_t>(p); }
bool aligned(const void* p, int n) { return addr(p) % uintptr_t(n) == 0; }

// byte extent of a [rows, cols] tensor with row stride ld
struct Extent {
  uintptr_t lo = 0, hi = 0;   // [lo, hi)
  const void* p = nullptr;
  int64_t ld = 0;
};
Extent mat_extent(const void* p, int64_t rows, int64_t cols, int64_t ld, int es) {
  Extent e;
  e.p = p;
  e.ld = ld;
  e.lo = addr(p);
  e.hi = e.lo + uintptr_t(((rows - 1) * ld + cols) * es);
  return e;
}
Extent vec_extent(const void* p, int64_t n, int es) {
  Extent e;
  e.p = p;
  e.ld = -1;
  e.lo = addr(p);
  e.hi = e.lo + uintptr_t(n * es);
  return e;
}
bool overlap(const Extent& a, const Extent& b) {
  if (!a.p || !b.p) return false;
  return a.lo < b.hi && b.lo < a.hi;
}
// an output may coincide exactly with a row-shaped input of the same dtype
bool identical(const Extent& a, const Extent& b) {
  return a.p && a.p == b.p && a.ld == b.ld && a.ld >= 0;
}

// shape checks shared by the [rows, cols] entry points
fs_status check_shape(int64_t rows, int64_t cols, int64_t max_cols) {
  if (rows < 0 || cols < 0) return fail(FS_ERR_BAD_SHAPE, "rows=%lld cols=%lld must be >= 0",
                                        (long long)rows, (long long)cols);
  if (cols > max_cols) return fail(FS_ERR_BAD_SHAPE, "cols=%lld exceeds the limit %lld",
                                   (long long)cols, (long long)max_cols);
  return FS_OK;
}

fs_status check_ld(const char* name, int64_t ld, int64_t rows, int64_t cols) {
  if (ld < cols) return fail(FS_ERR_BAD_STRIDE, "%s=%lld < cols=%lld", name, (long long)ld,
                             (long long)cols);
  // the last element offset must fit comfortably in int64 bytes
  if (rows > 0 && ld > 0 && (rows - 1) > (INT64_MAX / 8 - cols) / ld)
    return fail(FS_ERR_BAD_SHAPE, "%s * rows overflows", name);
  return FS_OK;
}

// Row strides are only bounded by the overflow guard when there are several
// rows, so the byte products below are taken in uint64 arithmetic: exact mod
// 16, since 2^64 is a multiple of 16.
bool vec_ok(const void* p, int64_t ld, int es, int unit = 16) {
  return p == nullptr || (aligned(p, unit) && (uint64_t(ld) * uint64_t(es)) % uint64_t(unit) == 0);
}

// q (or NULL) starts every row at the same offset within a 16-byte unit as p
bool same_phase(const void* p, int64_t ld, const void* q, int64_t ldq, int es) {
  return q == nullptr ||
         ((addr(p) - addr(q)) % 16 == 0 && ((uint64_t(ld) - uint64_t(ldq)) * uint64_t(es)) % 16 == 0);
}

// the byte mask q (or NULL) starts every row at the same element offset
// within its v-byte unit as p (elements of es bytes) within its 16-byte unit:
// the aligned body of p's rows then meets whole v-byte units of q's
bool same_byte_phase(const void* p, int64_t ld, int es, const void* q, int64_t ldq, int v) {
  return q == nullptr ||
         ((addr(p) / uintptr_t(es) - addr(q)) % uintptr_t(v) == 0 &&
          (uint64_t(ld) - uint64_t(ldq)) % uint64_t(v) == 0);
}

}  // namespace

extern "C" {

const char* fs_status_string(fs_status s) {
  switch (s) {
    case FS_OK: return "FS_OK";
    case FS_ERR_NULL_POINTER: return "FS_ERR_NULL_POINTER: a required pointer is NULL";
    case FS_ERR_BAD_SHAPE: return "FS_ERR_BAD_SHAPE: invalid rows/cols";
    case FS_ERR_BAD_STRIDE: return "FS_ERR_BAD_STRIDE: row stride smaller than cols";
    case FS_ERR_UNSUPPORTED_DTYPE: return "FS_ERR_UNSUPPORTED_DTYPE: unsupported dtype";
    case FS_ERR_ALIASING: return "FS_ERR_ALIASING: forbidden overlap of an output";
    case FS_ERR_BAD_ARGUMENT: return "FS_ERR_BAD_ARGUMENT: invalid argument value";
    case FS_ERR_HIP: return "FS_ERR_HIP: HIP runtime error";
  }
  return "FS_ERR_UNKNOWN: unknown status code";
}

const char* fs_last_error_message(void) { return g_msg; }

int fs_abi_version(void) { return FS_ABI_VERSION; }

fs_status fs_pointwise_chain(const void* x, int64_t ld_x, const void* bias, const void* residual,
                             int64_t ld_r, void* y, int64_t ld_y, int64_t rows, int64_t cols,
                             float scale, fs_act act, fs_dtype dtype, hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (int(act) < FS_ACT_NONE || int(act) > FS_ACT_RELU)
    return fail(FS_ERR_BAD_ARGUMENT, "act=%d", int(act));
  if (!std::isfinite(scale)) return fail(FS_ERR_BAD_ARGUMENT, "scale is not finite");
  fs_status st = check_shape(rows, cols, INT32_MAX / 2);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_y", ld_y, rows, cols)) != FS_OK) return st;
  if (residual && (st = check_ld("ld_r", ld_r, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0) return FS_OK;
  if (!x || !y) return fail(FS_ERR_NULL_POINTER, "x and y are required");
  const int es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(y, es) || !aligned(bias, es) || !aligned(residual, es))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent ex = mat_extent(x, rows, cols, ld_x, es), ey = mat_extent(y, rows, cols, ld_y, es);
  const Extent er = residual ? mat_extent(residual, rows, cols, ld_r, es) : Extent{};
  const Extent eb = bias ? vec_extent(bias, cols, es) : Extent{};
  if ((overlap(ey, ex) && !identical(ey, ex)) || (overlap(ey, er) && !identical(ey, er)) ||
      overlap(ey, eb))
    return fail(FS_ERR_ALIASING, "y overlaps an input other than exactly x or residual");

  fs::PointwiseArgs a{x, ld_x, bias, residual, ld_r, y, ld_y, rows, cols, scale, act, dtype, false};
  a.vec = cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es) && vec_ok(y, ld_y, es) &&
          vec_ok(residual, ld_r, es) && (bias == nullptr || aligned(bias, 16));
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype) && same_phase(x, ld_x, y, ld_y, es) &&
              same_phase(x, ld_x, residual, ld_r, es);
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_pointwise(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "pointwise_chain launch");
}

fs_status fs_pointwise_program(const void* x, int64_t ld_x, const fs_op* ops, int n_ops,
                               const void* bias, const void* col, const void* residual,
                               int64_t ld_r, void* y, int64_t ld_y, int64_t rows, int64_t cols,
                               fs_dtype dtype, hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (n_ops < 0 || n_ops > FS_PROGRAM_MAX_OPS)
    return fail(FS_ERR_BAD_ARGUMENT, "n_ops=%d outside 0..%d", n_ops, FS_PROGRAM_MAX_OPS);
  if (n_ops > 0 && !ops) return fail(FS_ERR_NULL_POINTER, "ops is NULL with n_ops=%d", n_ops);
  fs::ProgramArgs a{};
  bool need_bias = false, need_col = false, need_res = false;
  for (int k = 0; k < n_ops; ++k) {
    const fs_op& o = ops[k];
    switch (o.code) {
      case FS_OP_SCALE: case FS_OP_SHIFT: case FS_OP_LEAKY_RELU:
        if (!std::isfinite(o.a)) return fail(FS_ERR_BAD_ARGUMENT, "ops[%d].a is not finite", k);
        break;
      case FS_OP_CLAMP:
        if (std::isnan(o.a) || std::isnan(o.b) || o.a > o.b)
          return fail(FS_ERR_BAD_ARGUMENT, "ops[%d]: clamp bounds must be ordered, not NaN", k);
        break;
      case FS_OP_ADD_BIAS: need_bias = true; break;
      case FS_OP_MUL_COLUMN: need_col = true; break;
      case FS_OP_ADD_RESIDUAL: case FS_OP_MUL_RESIDUAL: need_res = true; break;
      case FS_OP_GELU_ERF: case FS_OP_SIGMOID: case FS_OP_RELU: case FS_OP_TANH: case FS_OP_SILU:
        break;
      default: return fail(FS_ERR_BAD_ARGUMENT, "ops[%d].code=%d", k, int(o.code));
    }
    a.prog.code[k] = o.code;
    a.prog.a[k] = o.a;
    a.prog.b[k] = o.b;
  }
  a.prog.n = n_ops;
  fs_status st = check_shape(rows, cols, INT32_MAX / 2);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_y", ld_y, rows, cols)) != FS_OK) return st;
  if (need_res && (st = check_ld("ld_r", ld_r, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0) return FS_OK;
  if (!x || !y) return fail(FS_ERR_NULL_POINTER, "x and y are required");
  if ((need_bias && !bias) || (need_col && !col) || (need_res && !residual))
    return fail(FS_ERR_NULL_POINTER, "the program reads a NULL bias, col or residual");
  // operands the program does not read are not touched
  if (!need_bias) bias = nullptr;
  if (!need_col) col = nullptr;
  if (!need_res) residual = nullptr;
  const int es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(y, es) || !aligned(bias, es) || !aligned(col, es) ||
      !aligned(residual, es))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent ex = mat_extent(x, rows, cols, ld_x, es), ey = mat_extent(y, rows, cols, ld_y, es);
  const Extent er = residual ? mat_extent(residual, rows, cols, ld_r, es) : Extent{};
  const Extent eb = bias ? vec_extent(bias, cols, es) : Extent{};
  const Extent ec = col ? vec_extent(col, cols, es) : Extent{};
  if ((overlap(ey, ex) && !identical(ey, ex)) || (overlap(ey, er) && !identical(ey, er)) ||
      overlap(ey, eb) || overlap(ey, ec))
    return fail(FS_ERR_ALIASING, "y overlaps an input other than exactly x or residual");

  a.x = x; a.ld_x = ld_x; a.bias = bias; a.col = col; a.res = residual; a.ld_r = ld_r;
  a.y = y; a.ld_y = ld_y; a.rows = rows; a.cols = cols; a.dtype = dtype;
  a.vec = cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es) && vec_ok(y, ld_y, es) &&
          vec_ok(residual, ld_r, es) && (bias == nullptr || aligned(bias, 16)) &&
          (col == nullptr || aligned(col, 16));
  // bias and col are staged element by element: their alignment does not matter
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype) && same_phase(x, ld_x, y, ld_y, es) &&
              same_phase(x, ld_x, residual, ld_r, es);
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_program(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "pointwise_program launch");
}

fs_status fs_row_softmax(const void* x, int64_t ld_x, const void* mask, int64_t ld_mask,
                         fs_dtype mask_dtype, void* y, int64_t ld_y, int64_t rows, int64_t cols,
                         float scale, int64_t causal_q_len, fs_dtype dtype, hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (mask && !dtype_ok(mask_dtype) && mask_dtype != FS_U8)
    return fail(FS_ERR_UNSUPPORTED_DTYPE, "mask_dtype=%d", int(mask_dtype));
  if (!mask) mask_dtype = dtype;
  if (!std::isfinite(scale)) return fail(FS_ERR_BAD_ARGUMENT, "scale is not finite");
  if (causal_q_len < 0) return fail(FS_ERR_BAD_ARGUMENT, "causal_q_len=%lld < 0",
                                    (long long)causal_q_len);
  fs_status st = check_shape(rows, cols, FS_SOFTMAX_MAX_COLS);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_y", ld_y, rows, cols)) != FS_OK) return st;
  if (mask && (st = check_ld("ld_mask", ld_mask, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0) return FS_OK;
  if (!x || !y) return fail(FS_ERR_NULL_POINTER, "x and y are required");
  const int es = elem_size(dtype), ms = elem_size(mask_dtype);
  if (!aligned(x, es) || !aligned(y, es) || !aligned(mask, ms))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent ex = mat_extent(x, rows, cols, ld_x, es), ey = mat_extent(y, rows, cols, ld_y, es);
  const Extent em = mask ? mat_extent(mask, rows, cols, ld_mask, ms) : Extent{};
  if ((overlap(ey, ex) && !identical(ey, ex)) || overlap(ey, em))
    return fail(FS_ERR_ALIASING, "y overlaps the mask or partially overlaps x");

  fs::SoftmaxArgs a{x, ld_x, mask, ld_mask, mask_dtype, y, ld_y, rows, cols, scale,
                    causal_q_len, dtype, false};
  // the mask's share of a 16-byte vector of x: 16 bytes, or 8 / 4 of a byte mask
  const int mask_unit = std::min(16, vec_width(dtype) * ms);
  a.vec = cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es) && vec_ok(y, ld_y, es) &&
          vec_ok(mask, ld_mask, ms, mask_unit);
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype) && same_phase(x, ld_x, y, ld_y, es) &&
              (mask_dtype == FS_U8 ? same_byte_phase(x, ld_x, es, mask, ld_mask, vec_width(dtype))
                                   : ms == es && same_phase(x, ld_x, mask, ld_mask, es));
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_softmax(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "row_softmax launch");
}

fs_status fs_causal_softmax_trimmed(const void* x, int64_t ld_x, void* y, int64_t ld_y,
                                    int64_t rows, int64_t cols, float scale,
                                    int64_t causal_q_len, int64_t block, fs_dtype dtype,
                                    hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (!std::isfinite(scale)) return fail(FS_ERR_BAD_ARGUMENT, "scale is not finite");
  if (causal_q_len < 1)
    return fail(FS_ERR_BAD_ARGUMENT, "causal_q_len=%lld must be >= 1", (long long)causal_q_len);
  if (block < 1 || block > (int64_t(1) << 30) || (block & (block - 1)) != 0)
    return fail(FS_ERR_BAD_ARGUMENT, "block=%lld must be a power of two", (long long)block);
  fs_status st = check_shape(rows, cols, FS_SOFTMAX_MAX_COLS);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_y", ld_y, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0) return FS_OK;
  if (!x || !y) return fail(FS_ERR_NULL_POINTER, "x and y are required");
  const int es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(y, es))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent ex = mat_extent(x, rows, cols, ld_x, es), ey = mat_extent(y, rows, cols, ld_y, es);
  if (overlap(ey, ex) && !identical(ey, ex))
    return fail(FS_ERR_ALIASING, "y partially overlaps x");

  fs::SoftmaxArgs a{x, ld_x, nullptr, 0, dtype, y, ld_y, rows, cols, scale,
                    causal_q_len, dtype, false};
  a.vec = cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es) && vec_ok(y, ld_y, es);
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype) && same_phase(x, ld_x, y, ld_y, es);
  int shift = 0;
  while ((int64_t(1) << shift) < block) ++shift;
  a.trim_shift = shift;
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_softmax(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "causal_softmax_trimmed launch");
}

}  // extern "C"

namespace {

// shared by LayerNorm and RMSNorm (rms: no mean, no beta)
fs_status norm_residual(const void* x, int64_t ld_x, const void* residual, int64_t ld_r,
                        const void* gamma, const void* beta, void* y, int64_t ld_y,
                        void* residual_out, int64_t ld_ro, int64_t rows, int64_t cols, float eps,
                        fs_dtype dtype, hipStream_t stream, bool rms) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (!std::isfinite(eps) || eps < 0.f) return fail(FS_ERR_BAD_ARGUMENT, "eps must be finite, >= 0");
  fs_status st = check_shape(rows, cols, FS_LAYERNORM_MAX_COLS);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_y", ld_y, rows, cols)) != FS_OK) return st;
  if (residual && (st = check_ld("ld_r", ld_r, rows, cols)) != FS_OK) return st;
  if (residual_out && (st = check_ld("ld_ro", ld_ro, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0) return FS_OK;
  if (!x || !y) return fail(FS_ERR_NULL_POINTER, "x and y are required");
  const int es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(y, es) || !aligned(residual, es) || !aligned(gamma, es) ||
      !aligned(beta, es) || !aligned(residual_out, es))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent ex = mat_extent(x, rows, cols, ld_x, es), ey = mat_extent(y, rows, cols, ld_y, es);
  const Extent er = residual ? mat_extent(residual, rows, cols, ld_r, es) : Extent{};
  const Extent eo = residual_out ? mat_extent(residual_out, rows, cols, ld_ro, es) : Extent{};
  const Extent eg = gamma ? vec_extent(gamma, cols, es) : Extent{};
  const Extent eb = beta ? vec_extent(beta, cols, es) : Extent{};
  for (const Extent* out : {&ey, &eo}) {
    if ((overlap(*out, ex) && !identical(*out, ex)) || (overlap(*out, er) && !identical(*out, er)) ||
        overlap(*out, eg) || overlap(*out, eb))
      return fail(FS_ERR_ALIASING, "an output overlaps an input other than exactly x or residual");
  }
  if (overlap(ey, eo)) return fail(FS_ERR_ALIASING, "y overlaps residual_out");

  fs::LayerNormArgs a{x, ld_x, residual, ld_r, gamma, beta, y, ld_y, residual_out, ld_ro,
                      rows, cols, eps, dtype, false, rms};
  a.vec = cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es) && vec_ok(y, ld_y, es) &&
          vec_ok(residual, ld_r, es) && vec_ok(residual_out, ld_ro, es) &&
          (gamma == nullptr || aligned(gamma, 16)) && (beta == nullptr || aligned(beta, 16));
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype) && same_phase(x, ld_x, y, ld_y, es) &&
              same_phase(x, ld_x, residual, ld_r, es) && same_phase(x, ld_x, residual_out, ld_ro, es);
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_layernorm(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, rms ? "rmsnorm_residual launch"
                                                   : "layernorm_residual launch");
}

// shared by the row reductions (argmax when out_i is set)
fs_status row_reduce(const void* x, int64_t ld_x, fs_dtype dtype, fs_row_op op, float* out_f,
                     int64_t* out_i, int64_t rows, int64_t cols, hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (!out_i && op != FS_ROW_SUM && op != FS_ROW_MEAN && op != FS_ROW_MAX &&
      op != FS_ROW_LOGSUMEXP)
    return fail(FS_ERR_BAD_ARGUMENT, "op=%d", int(op));
  fs_status st = check_shape(rows, cols, INT32_MAX / 2);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_x", ld_x, rows, cols)) != FS_OK) return st;
  if (rows == 0) return FS_OK;
  if (cols == 0 && (out_i || op != FS_ROW_SUM))
    return fail(FS_ERR_BAD_SHAPE, "this reduction needs cols >= 1");
  if (!(out_f || out_i) || (cols > 0 && !x)) return fail(FS_ERR_NULL_POINTER, "x and out are required");
  const int es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(out_f, 4) || !aligned(out_i, 8))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent eo = out_i ? vec_extent(out_i, rows, 8) : vec_extent(out_f, rows, 4);
  const Extent ex = cols ? mat_extent(x, rows, cols, ld_x, es) : Extent{};
  if (overlap(eo, ex)) return fail(FS_ERR_ALIASING, "out overlaps x");
  fs::ReduceArgs a{x, ld_x, dtype, op, out_f, out_i, rows, cols, false};
  a.vec = cols > 0 && cols % vec_width(dtype) == 0 && vec_ok(x, ld_x, es);
  a.shifted = !a.vec && cols >= 2 * vec_width(dtype);
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = fs::launch_reduce(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, out_i ? "row_argmax launch" : "row_reduce launch");
}

}  // namespace

extern "C" {

fs_status fs_layernorm_residual(const void* x, int64_t ld_x, const void* residual, int64_t ld_r,
                                const void* gamma, const void* beta, void* y, int64_t ld_y,
                                void* residual_out, int64_t ld_ro, int64_t rows, int64_t cols,
                                float eps, fs_dtype dtype, hipStream_t stream) {
  return norm_residual(x, ld_x, residual, ld_r, gamma, beta, y, ld_y, residual_out, ld_ro, rows,
                       cols, eps, dtype, stream, false);
}

fs_status fs_rmsnorm_residual(const void* x, int64_t ld_x, const void* residual, int64_t ld_r,
                              const void* gamma, void* y, int64_t ld_y, void* residual_out,
                              int64_t ld_ro, int64_t rows, int64_t cols, float eps,
                              fs_dtype dtype, hipStream_t stream) {
  return norm_residual(x, ld_x, residual, ld_r, gamma, nullptr, y, ld_y, residual_out, ld_ro,
                       rows, cols, eps, dtype, stream, true);
}

fs_status fs_row_reduce(const void* x, int64_t ld_x, fs_dtype dtype, fs_row_op op, float* out,
                        int64_t rows, int64_t cols, hipStream_t stream) {
  return row_reduce(x, ld_x, dtype, op, out, nullptr, rows, cols, stream);
}

fs_status fs_row_argmax(const void* x, int64_t ld_x, fs_dtype dtype, int64_t* out, int64_t rows,
                        int64_t cols, hipStream_t stream) {
  if (!out) {
    clear_msg();
    if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
    if (rows < 0 || cols < 0) return fail(FS_ERR_BAD_SHAPE, "negative shape");
    if (rows == 0) return FS_OK;
    return fail(FS_ERR_NULL_POINTER, "out is required");
  }
  return row_reduce(x, ld_x, dtype, FS_ROW_MAX, nullptr, out, rows, cols, stream);
}

fs_status fs_gemm_epilogue_reduce(const void* c, int64_t ld_c, fs_dtype c_dtype, const void* bias,
                                  fs_dtype bias_dtype, const float* col_scale, fs_act act,
                                  fs_reduce reduce, float* row_out, int64_t rows, int64_t cols,
                                  hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(c_dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "c_dtype=%d", int(c_dtype));
  if (bias && !dtype_ok(bias_dtype))
    return fail(FS_ERR_UNSUPPORTED_DTYPE, "bias_dtype=%d", int(bias_dtype));
  if (!bias) bias_dtype = FS_F32;
  if (int(act) < FS_ACT_NONE || int(act) > FS_ACT_RELU)
    return fail(FS_ERR_BAD_ARGUMENT, "act=%d", int(act));
  if (int(reduce) < FS_REDUCE_SUM || int(reduce) > FS_REDUCE_LOGSUMEXP)
    return fail(FS_ERR_BAD_ARGUMENT, "reduce=%d", int(reduce));
  fs_status st = check_shape(rows, cols, INT32_MAX / 2);
  if (st != FS_OK) return st;
  if ((st = check_ld("ld_c", ld_c, rows, cols)) != FS_OK) return st;
  if (rows == 0) return FS_OK;
  if (cols == 0 && reduce != FS_REDUCE_SUM)
    return fail(FS_ERR_BAD_SHAPE, "this reduction needs cols >= 1");
  if (!row_out || (cols > 0 && !c)) return fail(FS_ERR_NULL_POINTER, "c and row_out are required");
  const int es = elem_size(c_dtype), bs = elem_size(bias_dtype);
  if (!aligned(c, es) || !aligned(bias, bs) || !aligned(col_scale, 4) || !aligned(row_out, 4))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  const Extent eo = vec_extent(row_out, rows, 4);
  const Extent ec = cols ? mat_extent(c, rows, cols, ld_c, es) : Extent{};
  const Extent eb = bias ? vec_extent(bias, cols, bs) : Extent{};
  const Extent es_ = col_scale ? vec_extent(col_scale, cols, 4) : Extent{};
  if (overlap(eo, ec) || overlap(eo, eb) || overlap(eo, es_))
    return fail(FS_ERR_ALIASING, "row_out overlaps an input");

  fs::EpilogueArgs a{c, ld_c, c_dtype, bias, bias_dtype, col_scale, act, reduce, row_out,
                     rows, cols, false};
  a.vec = cols > 0 && cols % vec_width(c_dtype) == 0 && vec_ok(c, ld_c, es);
  a.coef_vec = aligned(bias, 16) && aligned(col_scale, 16);
  a.shifted = !a.vec && cols >= 2 * vec_width(c_dtype);
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  hipError_t e = reduce == FS_REDUCE_MAX || reduce == FS_REDUCE_LOGSUMEXP
                     ? fs::launch_epilogue_maxlse(a, cus, stream)
                     : fs::launch_epilogue(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "gemm_epilogue_reduce launch");
}

fs_status fs_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream) {
  clear_msg();
  if (bytes < 0) return fail(FS_ERR_BAD_SHAPE, "bytes=%lld < 0", (long long)bytes);
  if (bytes == 0) return FS_OK;
  if (!src || !dst) return fail(FS_ERR_NULL_POINTER, "src and dst are required");
  if (overlap(vec_extent(src, bytes, 1), vec_extent(dst, bytes, 1)))
    return fail(FS_ERR_ALIASING, "src and dst overlap");
  int cus = 0;
  fs_status st = device_cus(&cus);
  if (st != FS_OK) return st;
  hipError_t e = fs::launch_copy(src, dst, bytes, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "copy launch");
}

fs_status fs_copy_strided(const void* src, int64_t ld_src, int64_t stride_src, void* dst,
                          int64_t ld_dst, int64_t stride_dst, int64_t rows, int64_t cols,
                          int64_t batch, fs_dtype dtype, hipStream_t stream) {
  clear_msg();
  if (!dtype_ok(dtype)) return fail(FS_ERR_UNSUPPORTED_DTYPE, "dtype=%d", int(dtype));
  if (rows < 0 || cols < 0 || batch < 0)
    return fail(FS_ERR_BAD_SHAPE, "rows=%lld cols=%lld batch=%lld must be >= 0",
                (long long)rows, (long long)cols, (long long)batch);
  if (batch > 0 && cols > ((int64_t(1) << 30) - 1) / batch)
    return fail(FS_ERR_BAD_SHAPE, "batch * cols must be < 2^30");
  if (stride_src < 0 || stride_dst < 0)
    return fail(FS_ERR_BAD_STRIDE, "batch strides must be >= 0");
  fs_status st;
  if ((st = check_ld("ld_src", ld_src, rows, cols)) != FS_OK) return st;
  if ((st = check_ld("ld_dst", ld_dst, rows, cols)) != FS_OK) return st;
  if (rows == 0 || cols == 0 || batch == 0) return FS_OK;
  // the last element offset of each side must fit in int64 bytes
  for (int64_t sb : {stride_src, stride_dst})
    if (batch > 1 && sb > 0 && (batch - 1) > (INT64_MAX / 8 - (rows - 1) * std::max(ld_src, ld_dst) - cols) / sb)
      return fail(FS_ERR_BAD_SHAPE, "batch * stride overflows");
  // every destination element distinct: batches one after another, or
  // interleaved within each destination row
  const bool outer = stride_dst >= (rows - 1) * ld_dst + cols;
  const bool inner = stride_dst >= cols && ld_dst >= (batch - 1) * stride_dst + cols;
  if (batch > 1 && !outer && !inner)
    return fail(FS_ERR_BAD_STRIDE, "destination batches overlap each other");
  if (!src || !dst) return fail(FS_ERR_NULL_POINTER, "src and dst are required");
  const int es = elem_size(dtype);
  if (!aligned(src, es) || !aligned(dst, es))
    return fail(FS_ERR_BAD_ARGUMENT, "pointers must be aligned to the element size");
  auto span = [&](const void* p, int64_t ld, int64_t sb) {
    return vec_extent(p, (batch - 1) * sb + (rows - 1) * ld + cols, es);
  };
  if (overlap(span(src, ld_src, stride_src), span(dst, ld_dst, stride_dst)))
    return fail(FS_ERR_ALIASING, "the spans of src and dst overlap");
  int cus = 0;
  if ((st = device_cus(&cus)) != FS_OK) return st;
  fs::CopyStridedArgs a{src, ld_src, stride_src, dst, ld_dst, stride_dst, rows, cols, batch, es};
  hipError_t e = fs::launch_copy_strided(a, cus, stream);
  return e == hipSuccess ? FS_OK : hip_fail(e, "strided copy launch");
}

}  // extern "C"
