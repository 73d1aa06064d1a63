/*
 * libfusedsub -- fused sub-kernels of a compiled model graph, for AMD
 * Instinct MI355X (CDNA4, gfx950).
 *
 * A compiled model is a set of generated sub-kernels plus fixed vendor
 * library calls (KernelOPT, Def. 1 in Section 3).  The GEMMs stay library
 * calls; this library implements the generated part: fused pointwise chains
 * and programs, row reductions (softmax, LayerNorm and RMSNorm with residual,
 * sum, mean, max, argmax) and GEMM epilogues with a row reduction (Appendix A, Codegen and Fusion Agent prompts: epilogue
 * fusion, cross-reduction fusion, pointwise + pointwise, residual + norm).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers are DEVICE pointers; the caller owns every buffer.  The library
 * allocates no device memory, keeps no state apart from a lazily filled
 * per-device table of compute-unit counts, and never synchronises the
 * stream.  Work is enqueued on `stream` (0 = the null stream) and the call
 * returns after the enqueue.
 *
 * Layout: 2-D tensors are row-major with unit inner stride; `ld_*` is the row
 * stride in ELEMENTS and must be >= cols.  A batched tensor whose leading
 * dimensions are contiguous is passed flattened to rows (e.g. attention
 * scores [B, H, S, S] are rows = B*H*S, cols = S).  Vectors indexed by
 * column (bias, gamma, beta, col_scale) are contiguous [cols].
 *
 * rows == 0 or cols == 0 is an empty problem and returns FS_OK without
 * launching anything (except where an entry point says otherwise).
 *
 * Arithmetic is fp32 in registers for every dtype; bf16 values are widened
 * exactly on load and rounded to nearest even once, on the final store
 * (Appendix A, Executor prompt: accumulate in fp32, cast on the final store).
 *
 * Alignment: every pointer must be aligned to its element size (a float at a
 * multiple of 4 bytes, a bf16 value at a multiple of 2; FS_ERR_BAD_ARGUMENT
 * otherwise; a byte mask may start anywhere).  Within that, any address, row stride and width is accepted:
 * base pointers aligned to 16 bytes with ld*sizeof(elem) a multiple of 16 (and
 * cols a multiple of the 16-byte vector width) take the 128-bit vector path,
 * rows whose operands share one offset within a 16-byte unit load their
 * aligned body 16 bytes at a time, and anything else takes a correct
 * element-wise path.
 *
 * Errors: every entry point validates its arguments on the host, before any
 * HIP call, and returns a status; it never aborts.  A launch failure returns
 * FS_ERR_HIP with the HIP error text in fs_last_error_message().  Faults that
 * occur while a kernel runs surface at the caller's next synchronisation.
 *
 * Aliasing: an output may coincide exactly (same pointer, same ld) with a
 * row-shaped input where the entry point says so; any other overlap between
 * an output and another argument returns FS_ERR_ALIASING.
 *
 * Thread safety: calls may be made from several host threads; calls that
 * share output buffers on overlapping streams race like any kernels do.
 */
#ifndef FUSEDSUB_H
#define FUSEDSUB_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FS_ABI_VERSION 2
#define FS_API __attribute__((visibility("default")))

typedef enum fs_status {
  FS_OK = 0,
  FS_ERR_NULL_POINTER = 1,      /* a required pointer is NULL                  */
  FS_ERR_BAD_SHAPE = 2,         /* rows/cols negative or beyond a limit        */
  FS_ERR_BAD_STRIDE = 3,        /* ld < cols                                   */
  FS_ERR_UNSUPPORTED_DTYPE = 4, /* dtype value or combination not supported    */
  FS_ERR_ALIASING = 5,          /* forbidden overlap of an output              */
  FS_ERR_BAD_ARGUMENT = 6,      /* enum out of range, negative q_len, bad eps  */
  FS_ERR_HIP = 7                /* the HIP runtime reported an error           */
} fs_status;

/* FS_U8 is a byte mask, accepted only as the mask_dtype of fs_row_softmax: a
 * nonzero byte excludes its position (the additive value -inf), a zero byte
 * keeps it (0).  Added in ABI version 2. */
typedef enum fs_dtype { FS_F32 = 0, FS_BF16 = 1, FS_U8 = 2 } fs_dtype;

typedef enum fs_act {
  FS_ACT_NONE = 0,
  FS_ACT_GELU_ERF = 1,          /* z * (1 + erf(z / sqrt 2)) / 2               */
  FS_ACT_SIGMOID = 2,           /* 1 / (1 + exp(-z))                           */
  FS_ACT_RELU = 3               /* max(z, 0)                                   */
} fs_act;

typedef enum fs_reduce {
  FS_REDUCE_SUM = 0,
  FS_REDUCE_MEAN = 1,
  FS_REDUCE_MAX = 2,        /* added in ABI version 2 */
  FS_REDUCE_LOGSUMEXP = 3   /* added in ABI version 2 */
} fs_reduce;

typedef enum fs_row_op {
  FS_ROW_SUM = 0,
  FS_ROW_MEAN = 1,
  FS_ROW_MAX = 2,
  FS_ROW_LOGSUMEXP = 3   /* added in ABI version 2 */
} fs_row_op;

/*
 * Fused pointwise chain (Appendix A, Fusion Agent: pointwise + pointwise and
 * activation + bias fusion -- load once, apply every op, store once).
 *
 *   y[r, j] = act(x[r, j] * scale + bias[j]) + residual[r, j]
 *
 * x, residual, y : [rows, cols] of `dtype`, row strides ld_x, ld_r, ld_y.
 * bias           : [cols] of `dtype`, or NULL (no bias).
 * residual       : or NULL (no residual; ld_r is then ignored).
 * y may be x or residual exactly (in place).  scale must be finite.
 */
FS_API fs_status fs_pointwise_chain(const void* x, int64_t ld_x, const void* bias,
                             const void* residual, int64_t ld_r, void* y, int64_t ld_y,
                             int64_t rows, int64_t cols, float scale, fs_act act,
                             fs_dtype dtype, hipStream_t stream);

/*
 * Fused pointwise program: the general form of the chain above, for the
 * groups of adjacent elementwise operations a compiled graph merges into one
 * kernel (Section 3: adjacent fusible groups, e.g. a multiply, a hardtanh and
 * a GELU after a linear layer; Appendix A, Fusion Agent: pointwise +
 * pointwise, activation + bias fusion).
 *
 *   v = x[r, j];  for i < n_ops: v = op_i(v);  y[r, j] = v
 *
 * Every step is evaluated in fp32 registers (one rounding per step); y is
 * rounded to `dtype` once.  x, residual, y: [rows, cols] of `dtype` with row
 * strides ld_x, ld_r, ld_y; bias, col: [cols] of `dtype`.  bias, col and
 * residual may be NULL unless an operation reads them (FS_ERR_NULL_POINTER).
 * y may be x or residual exactly (in place) and must not overlap bias or
 * col.  ops: n_ops (0 ... FS_PROGRAM_MAX_OPS) operations, read on the host
 * during the call (the caller keeps ownership); a and b as listed, finite
 * (clamp bounds may be infinite, with a <= b), else FS_ERR_BAD_ARGUMENT.
 * Rows of whole 16-byte vectors are read and written 16 bytes at a time;
 * other rows element by element.  Added in ABI version 2.
 */
#define FS_PROGRAM_MAX_OPS 16
typedef enum fs_op_code {
  FS_OP_SCALE = 0,          /* v * a                                       */
  FS_OP_SHIFT = 1,          /* v + a                                       */
  FS_OP_ADD_BIAS = 2,       /* v + bias[j]                                 */
  FS_OP_MUL_COLUMN = 3,     /* v * col[j]                                  */
  FS_OP_ADD_RESIDUAL = 4,   /* v + residual[r, j]                          */
  FS_OP_MUL_RESIDUAL = 5,   /* v * residual[r, j]                          */
  FS_OP_CLAMP = 6,          /* min(max(v, a), b); hardtanh: a = -1, b = 1  */
  FS_OP_GELU_ERF = 7,       /* v * (1 + erf(v / sqrt 2)) / 2               */
  FS_OP_SIGMOID = 8,        /* 1 / (1 + exp(-v))                           */
  FS_OP_RELU = 9,           /* max(v, 0)                                   */
  FS_OP_TANH = 10,          /* tanh(v)                                     */
  FS_OP_SILU = 11,          /* v * sigmoid(v)                              */
  FS_OP_LEAKY_RELU = 12     /* v >= 0 ? v : a * v                          */
} fs_op_code;
typedef struct fs_op {
  int32_t code;             /* an fs_op_code                               */
  float a, b;               /* parameters (unused ones are ignored)        */
} fs_op;
FS_API fs_status fs_pointwise_program(const void* x, int64_t ld_x, const fs_op* ops, int n_ops,
                                      const void* bias, const void* col, const void* residual,
                                      int64_t ld_r, void* y, int64_t ld_y, int64_t rows,
                                      int64_t cols, fs_dtype dtype, hipStream_t stream);

/*
 * Fused row softmax with pre-scale and additive mask (Appendix A, Planner
 * item 9 and Codegen prompt: fused softmax, online softmax).
 *
 *   a[r, j] = x[r, j] * scale + mask[r, j]   (additive mask, e.g. 0 / -inf)
 *   y[r, :] = exp(a[r, :] - max_j a[r, j]) / sum_j exp(a[r, j] - max)
 *
 * x, y   : [rows, cols] of `dtype`; y may be x exactly (in place).
 * mask   : [rows, cols] of `mask_dtype` with row stride ld_mask, or NULL.
 *          FS_U8 (a byte mask: nonzero = excluded, i.e. -inf; zero = 0) reads
 *          1 byte per element instead of 2 or 4.  The 16-byte path of x reads
 *          the mask elements of each x vector at once: 8 bytes (bf16 x) or 4
 *          (fp32 x) of a byte mask, 8 of a bf16 mask beside fp32 x, 16 bytes
 *          otherwise; it needs the mask's rows to start at multiples of that
 *          many bytes.  For rows that are not whole 16-byte vectors, a byte
 *          mask whose rows start at x's element offset within those units
 *          (contiguous tensors, for instance) shares x's aligned body below.
 *          A byte mask gives the same result, bit for bit, as the additive
 *          mask of 0 and -inf it stands for, on the same path.
 * causal_q_len > 0 additionally masks element (r, j) when
 *          j > (r mod causal_q_len) + (cols - causal_q_len); masked
 *          elements are not read and are written as +0.  0 = off.
 * Entries whose logit is -inf come out exactly +0; a fully masked row comes
 * out all +0.  Rows up to 32768 columns are held in registers and read from
 * HBM once, with a single (max, sum) online combine per row.  Longer rows
 * keep the exponentials of their first 65536 columns on chip (LDS and
 * registers, one row per compute unit) and read those columns once; the
 * columns past them are streamed: one pass keeps a running (max, sum) and a
 * second re-reads x (and mask) to write y (2 reads + 1 write per element).
 * Rows that are not whole 16-byte vectors load one element per lane, except
 * rows of at least two vectors whose x, mask (of x's dtype) and y start each
 * row at the same offset within a 16-byte unit (contiguous tensors, for
 * instance), or with a byte mask at x's element phase: there the aligned
 * body of every row is loaded 16 bytes at a time.  Rows may be up to
 * FS_SOFTMAX_MAX_COLS columns.
 * scale must be finite; mask values may be any float or -inf.
 */
#define FS_SOFTMAX_MAX_COLS 16777216
FS_API fs_status fs_row_softmax(const void* x, int64_t ld_x, const void* mask, int64_t ld_mask,
                         fs_dtype mask_dtype, void* y, int64_t ld_y, int64_t rows,
                         int64_t cols, float scale, int64_t causal_q_len, fs_dtype dtype,
                         hipStream_t stream);

/*
 * Causal row softmax that leaves the zero blocks no consumer reads unwritten
 * (fused softmax with the causal mask, Appendix A, Planner item 9; the
 * writes it skips are dead stores once the P.V product is issued per row
 * block with K limited to the causal extent, the way the stitched block
 * does it).
 *
 *   a[r, j] = x[r, j] * scale, masked (-inf) when j > s + (cols - q),
 *   s = r mod causal_q_len, q = causal_q_len
 *   y[r, j] = softmax_j(a[r, :]) for j < w(r),
 *   w(r) = min(cols, (floor(s / block) + 1) * block + (cols - q)), clamped at 0
 *
 * Columns j >= w(r) of y are not written (they keep their contents); masked
 * columns below w(r) are written as +0.  For square attention (cols == q)
 * and block B, the rows of causal positions [i B, (i+1) B) write their first
 * (i+1) B columns: exactly what a P.V product over K = (i+1) B reads.
 * block must be a power of two (1 ... 2^30) and causal_q_len >= 1
 * (FS_ERR_BAD_ARGUMENT otherwise).  x, y, dtype, scale, shapes, strides and
 * aliasing as fs_row_softmax without a mask.
 */
FS_API fs_status fs_causal_softmax_trimmed(const void* x, int64_t ld_x, void* y, int64_t ld_y,
                                           int64_t rows, int64_t cols, float scale,
                                           int64_t causal_q_len, int64_t block, fs_dtype dtype,
                                           hipStream_t stream);

/*
 * LayerNorm fused with the residual add (Appendix A, Fusion Agent:
 * normalisation fusion -- mean and variance in one pass, normalise, scale and
 * bias in the same kernel, fp32 accumulation; residual + norm in one memory
 * pass; Codegen prompt: single-pass LayerNorm).
 *
 *   h = x + residual                     (fp32)
 *   y = (h - mean(h)) / sqrt(var(h) + eps) * gamma + beta   (biased variance)
 *   residual_out = h rounded to `dtype`
 *
 * x, residual, y, residual_out : [rows, cols] of `dtype`.
 * residual     : or NULL (plain LayerNorm, h = x).
 * residual_out : or NULL (not stored).
 * gamma, beta  : [cols] of `dtype`, or NULL (1 and 0).
 * y and residual_out may each be x or residual exactly; they may not overlap
 * each other.  eps must be finite and >= 0.  Rows of whole 16-byte vectors up
 * to 16384 columns (32768 for bf16), rows up to 16384 columns whose x,
 * residual, y and residual_out start each row at one offset within a 16-byte
 * unit (the aligned body of each row loaded 16 bytes at a time, gamma and
 * beta staged on chip), and other rows up to 8192 columns, are held in
 * registers: x and residual are read once and the statistics take two exact
 * passes over the registers.  Longer rows (for rows that are not
 * whole 16-byte vectors: past 32768 columns) keep h of their first 65536
 * columns on chip (LDS and registers, one row per compute unit) and read
 * those columns once, merging per-chunk (count, mean, M2) statistics; the
 * columns past them, and the other rows that are not whole 16-byte vectors,
 * are streamed: a first pass merges the statistics, a second re-reads x and
 * residual and writes residual_out and y.  Rows may be up to
 * FS_LAYERNORM_MAX_COLS columns.
 */
#define FS_LAYERNORM_MAX_COLS 16777216
FS_API fs_status fs_layernorm_residual(const void* x, int64_t ld_x, const void* residual,
                                int64_t ld_r, const void* gamma, const void* beta, void* y,
                                int64_t ld_y, void* residual_out, int64_t ld_ro, int64_t rows,
                                int64_t cols, float eps, fs_dtype dtype, hipStream_t stream);

/*
 * RMSNorm fused with the residual add (Appendix A, Fusion Agent: the
 * LayerNorm/RMSNorm normalisation fusion; residual + norm in one memory pass).
 *
 *   h = x + residual                     (fp32)
 *   y = h / sqrt(mean(h^2) + eps) * gamma
 *   residual_out = h rounded to `dtype`
 *
 * Arguments, layouts, aliasing rules and limits as fs_layernorm_residual,
 * without beta.
 */
FS_API fs_status fs_rmsnorm_residual(const void* x, int64_t ld_x, const void* residual,
                                     int64_t ld_r, const void* gamma, void* y, int64_t ld_y,
                                     void* residual_out, int64_t ld_ro, int64_t rows,
                                     int64_t cols, float eps, fs_dtype dtype,
                                     hipStream_t stream);

/*
 * Plain row reduction (Section 6 counts sum/mean reductions among the
 * optimised sub-kernel classes; Appendix A, Executor prompt: accumulate in
 * fp32).
 *
 *   out[i] = sum_j x[i, j]   (FS_ROW_SUM)
 *          = that / cols     (FS_ROW_MEAN)
 *          = max_j x[i, j]   (FS_ROW_MAX; a NaN in the row gives NaN)
 *          = log sum_j exp(x[i, j])   (FS_ROW_LOGSUMEXP, as m + log sum_j
 *            exp(x[i, j] - m) with running maxima m, so it never overflows;
 *            a row of -inf gives -inf, a +inf gives +inf, a NaN gives NaN;
 *            the reductions the paper's level-2 case study chains after a
 *            linear layer: sum, max, mean, log-sum-exp)
 *
 * x   : [rows, cols] of `dtype`, row stride ld_x.  Rows of any length: the
 *       row is streamed, not held in registers.
 * out : [rows] fp32, contiguous; must not overlap x.
 * cols == 0 with rows > 0: SUM writes zeros, MEAN, MAX and LOGSUMEXP return
 * FS_ERR_BAD_SHAPE.
 */
FS_API fs_status fs_row_reduce(const void* x, int64_t ld_x, fs_dtype dtype, fs_row_op op,
                               float* out, int64_t rows, int64_t cols, hipStream_t stream);

/*
 * Row argmax, bit-exact: out[i] is the index of the largest x[i, j]; the
 * lowest index wins a tie, and a NaN counts as larger than any number (the
 * first NaN wins).  x as in fs_row_reduce; out: [rows] int64, contiguous,
 * not overlapping x.  cols must be >= 1.
 */
FS_API fs_status fs_row_argmax(const void* x, int64_t ld_x, fs_dtype dtype, int64_t* out,
                               int64_t rows, int64_t cols, hipStream_t stream);

/*
 * GEMM epilogue with a row reduction, applied to the output C of a library
 * GEMM (Appendix A, Codegen prompt: keep the matmul a library call and fuse
 * only its epilogue; Fusion Agent: reduction + pointwise).
 *
 *   row_out[i] = reduce_j act((C[i, j] + bias[j]) * col_scale[j])
 *
 * reduce: FS_REDUCE_SUM, FS_REDUCE_MEAN, FS_REDUCE_MAX (a NaN gives NaN) or
 * FS_REDUCE_LOGSUMEXP (log sum_j exp(.), as max + log sum exp(. - max), so
 * it never overflows; -inf for a row of -inf, +inf and NaN propagate): the
 * reductions the paper's level-2 case study chains after a linear layer.
 * c         : [rows, cols] of c_dtype, row stride ld_c.
 * bias      : [cols] of bias_dtype, or NULL (0).
 * col_scale : [cols] fp32, or NULL (1).
 * row_out   : [rows] fp32 (contiguous).  With cols == 0 and rows > 0, SUM
 *             writes zeros and the other reductions return FS_ERR_BAD_SHAPE.
 * The sum is accumulated in fp32 (per-thread partial sums, then a tree).
 */
FS_API fs_status fs_gemm_epilogue_reduce(const void* c, int64_t ld_c, fs_dtype c_dtype,
                                  const void* bias, fs_dtype bias_dtype,
                                  const float* col_scale, fs_act act, fs_reduce reduce,
                                  float* row_out, int64_t rows, int64_t cols,
                                  hipStream_t stream);

/*
 * Batched strided 2-D copy: the layout transforms a compiled graph places
 * between library GEMMs (the .contiguous() copies that transposed or
 * permuted strides force, Section 4.4, Gate 4), e.g. splitting a token-major
 * [tokens, 3 * hidden] QKV projection into head-major [3 * heads, tokens,
 * head_dim] operands for one strided-batched attention GEMM, and merging
 * head-major attention output back into [tokens, hidden].
 *
 *   dst[b * stride_dst + r * ld_dst + c] = src[b * stride_src + r * ld_src + c]
 *   for b < batch, r < rows, c < cols
 *
 * Strides and leading dimensions are in elements of `dtype` (only the size
 * matters: bits are copied unchanged, NaN payloads included).
 * ld_src, ld_dst >= cols; stride_src, stride_dst >= 0 (0 broadcasts the
 * source).  batch * cols < 2^30.  Destination elements must be distinct:
 * either stride_dst >= (rows - 1) * ld_dst + cols (batches one after another)
 * or stride_dst >= cols and ld_dst >= (batch - 1) * stride_dst + cols
 * (batches interleaved within each row), else FS_ERR_BAD_STRIDE.  The spans
 * of src and dst must not overlap (FS_ERR_ALIASING).  16-byte units are used
 * when every address, stride and row length is a multiple of 16 bytes.
 */
FS_API fs_status fs_copy_strided(const void* src, int64_t ld_src, int64_t stride_src, void* dst,
                                 int64_t ld_dst, int64_t stride_dst, int64_t rows,
                                 int64_t cols, int64_t batch, fs_dtype dtype,
                                 hipStream_t stream);

/*
 * Calibration utility (not a sub-kernel): copies `bytes` bytes from src to
 * dst with 128-bit loads and stores when both are 16-byte aligned and bytes
 * is a multiple of 16, else byte by byte.  Used to measure the achievable
 * HBM bandwidth and to scale hardware byte counters.  src and dst must not
 * overlap.
 */
FS_API fs_status fs_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream);

/* Static text for a status code (never NULL; unknown codes included). */
FS_API const char* fs_status_string(fs_status s);

/* Detail of the last non-OK status returned on the calling host thread
 * ("" if none).  Valid until the next call on that thread. */
FS_API const char* fs_last_error_message(void);

/* FS_ABI_VERSION of the built library. */
FS_API int fs_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* FUSEDSUB_H */
