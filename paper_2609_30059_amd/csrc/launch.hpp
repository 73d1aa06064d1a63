// Host-side launch interface between the C ABI (api.hip) and the kernels.
// Arguments arrive here already validated; `vec` selects the 16-byte path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fusedsub.h"

namespace fs {

struct PointwiseArgs {
  const void* x; int64_t ld_x;
  const void* bias;
  const void* res; int64_t ld_r;
  void* y; int64_t ld_y;
  int64_t rows, cols;
  float scale;
  fs_act act;
  fs_dtype dtype;
  bool vec;
  // not vec, rows of at least two 16-byte vectors, and x, res and y start
  // every row at one offset within a 16-byte unit
  bool shifted = false;
};

struct SoftmaxArgs {
  const void* x; int64_t ld_x;
  const void* mask; int64_t ld_mask; fs_dtype mask_dtype;
  void* y; int64_t ld_y;
  int64_t rows, cols;
  float scale;
  int64_t causal_q_len;
  fs_dtype dtype;
  bool vec;
  int trim_shift = -1;   // causal block trimming: log2(block), or -1 (write whole rows)
  // not vec, but x, mask and y start every row at one offset within a
  // 16-byte unit: the row cache loads the aligned span of each row 16 bytes
  // at a time and its few head and tail elements one at a time
  bool shifted = false;
};

struct LayerNormArgs {
  const void* x; int64_t ld_x;
  const void* res; int64_t ld_r;
  const void* gamma; const void* beta;
  void* y; int64_t ld_y;
  void* res_out; int64_t ld_ro;
  int64_t rows, cols;
  float eps;
  fs_dtype dtype;
  bool vec;
  bool rms;        // RMSNorm: no mean, no beta
  // not vec, rows of at least two 16-byte vectors, and x, res, y and res_out
  // start every row at one offset within a 16-byte unit
  bool shifted = false;
};

struct EpilogueArgs {
  const void* c; int64_t ld_c; fs_dtype c_dtype;
  const void* bias; fs_dtype bias_dtype;
  const float* col_scale;
  fs_act act; fs_reduce reduce;
  float* out;
  int64_t rows, cols;
  bool vec;
  bool coef_vec = false;   // bias and col_scale (when given) are 16-byte aligned
  bool shifted = false;    // not vec, rows of at least two 16-byte vectors
};

// `cus` is the compute-unit count of the current device.
hipError_t launch_pointwise(const PointwiseArgs& a, int cus, hipStream_t s);
// A pointwise program as the kernel takes it: by value, in the argument block.
struct Program {
  int n;
  int32_t code[FS_PROGRAM_MAX_OPS];
  float a[FS_PROGRAM_MAX_OPS], b[FS_PROGRAM_MAX_OPS];
};

struct ProgramArgs {
  const void* x; int64_t ld_x;
  const void* bias; const void* col;
  const void* res; int64_t ld_r;   // NULL unless an operation reads it
  void* y; int64_t ld_y;
  int64_t rows, cols;
  fs_dtype dtype;
  bool vec;
  bool shifted = false;   // not vec, rows of at least two 16-byte vectors, one phase
  Program prog;
};

hipError_t launch_program(const ProgramArgs& a, int cus, hipStream_t s);
hipError_t launch_softmax(const SoftmaxArgs& a, int cus, hipStream_t s);
hipError_t launch_layernorm(const LayerNormArgs& a, int cus, hipStream_t s);
hipError_t launch_epilogue(const EpilogueArgs& a, int cus, hipStream_t s);
// FS_REDUCE_MAX and FS_REDUCE_LOGSUMEXP (epilogue_maxlse.hip)
hipError_t launch_epilogue_maxlse(const EpilogueArgs& a, int cus, hipStream_t s);
hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int cus, hipStream_t s);

struct CopyStridedArgs {
  const void* src; int64_t ld_src, stride_src;
  void* dst; int64_t ld_dst, stride_dst;
  int64_t rows, cols, batch;   // batch * cols < 2^30, rows * ld within int64
  int es;                      // element size in bytes (2 or 4)
};
hipError_t launch_copy_strided(const CopyStridedArgs& a, int cus, hipStream_t s);

struct ReduceArgs {
  const void* x; int64_t ld_x; fs_dtype dtype;
  fs_row_op op;
  float* out_f;      // sum / mean / max
  int64_t* out_i;    // argmax
  int64_t rows, cols;
  bool vec;
  bool shifted = false;   // not vec, element-aligned rows of at least two vectors
};
hipError_t launch_reduce(const ReduceArgs& a, int cus, hipStream_t s);

}  // namespace fs
