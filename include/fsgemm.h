/*
 * libfsgemm -- the fixed vendor-library GEMM calls around the fused
 * sub-kernels, as plain hipBLASLt calls.
 *
 * KernelOPT keeps the extern library calls of a compiled model fixed and
 * rewrites only the generated sub-kernels around them (Def. 1, Section 3;
 * Appendix A, Codegen prompt: keep matmul/conv as library calls).  This is
 * the MI355X counterpart of those library calls: a thin C ABI over
 * hipBLASLt, used by the stitched transformer block and by the GEMM whose
 * output feeds fs_gemm_epilogue_reduce.  It is not part of libfusedsub.
 *
 * Row-major operands, bf16 in and out, fp32 accumulation (HIPBLAS_COMPUTE_32F).
 * Device pointers, owned by the caller.  The library keeps one hipBLASLt
 * handle per device and caches the chosen algorithm per problem shape; it
 * allocates no device memory (the caller passes the workspace).
 */
#ifndef FSGEMM_H
#define FSGEMM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FSG_API __attribute__((visibility("default")))

typedef enum fsg_status {
  FSG_OK = 0,
  FSG_ERR_NULL_POINTER = 1,
  FSG_ERR_BAD_SHAPE = 2,      /* m, n, k, batch out of range              */
  FSG_ERR_BAD_STRIDE = 3,     /* a leading dimension is too small         */
  FSG_ERR_BAD_ARGUMENT = 4,   /* trans_b not 0/1, non-finite alpha        */
  FSG_ERR_LIBRARY = 5,        /* hipBLASLt returned an error              */
  FSG_ERR_NO_ALGO = 6,        /* hipBLASLt found no algorithm             */
  FSG_ERR_HIP = 7
} fsg_status;

/*
 * For every batch index i < batch:
 *   C_i = alpha * A_i @ op(B_i) (+ bias)          (row-major, bf16)
 *
 * A_i : [m, k], row stride lda >= k,  A_i = a + i * stride_a (elements).
 * B_i : trans_b == 0: [k, n], ldb >= n;  trans_b == 1: stored [n, k] with
 *       ldb >= k and used transposed.     B_i = b + i * stride_b.
 * C_i : [m, n], row stride ldc >= n,     C_i = c + i * stride_c.
 * bias: [n] bf16 added to every row (hipBLASLt BIAS epilogue), or NULL.
 * workspace: device buffer of workspace_bytes (may be NULL with 0 bytes).
 * Strides are ignored when batch == 1.  C must not overlap A, B or bias.
 */
FSG_API fsg_status fsg_gemm_bf16(const void* a, int64_t lda, int64_t stride_a, const void* b,
                                 int64_t ldb, int64_t stride_b, int trans_b, void* c,
                                 int64_t ldc, int64_t stride_c, int64_t m, int64_t n, int64_t k,
                                 int64_t batch, float alpha, const void* bias, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Activation applied by the GEMM's own epilogue, after bias.  hipBLASLt's
 * SIGMOID epilogue is not offered: with this ROCm release it returns success
 * for bf16 output without applying the activation or the bias. */
typedef enum fsg_act {
  FSG_ACT_NONE = 0,
  FSG_ACT_GELU = 1,       /* hipBLASLt's GELU (its own approximation, not erf) */
  FSG_ACT_RELU = 2
} fsg_act;

/*
 * The GEMM with hipBLASLt's built-in epilogue, for placing a thin epilogue
 * inside the library call instead of in a separate sub-kernel (the paper's
 * observation that thin epilogues after a GEMM can lose to dispatch overhead,
 * Section 6.2, library dominance; Section 6.3):
 *
 *   C_i = act( alpha_col (.) (A_i @ op(B_i)) + beta * Cin_i + bias )
 *
 * alpha_col : [n] fp32 per-column scale (device), or NULL for the scalar
 *             alpha; with a vector, alpha must be 1.
 * bias      : [n] per-column, bf16 (bias_f32 = 0) or fp32 (bias_f32 = 1), or NULL.
 * c_in      : [m, n] bf16 with row stride ld_cin >= n and batch stride
 *             stride_cin, read when beta != 0 (e.g. a residual added inside
 *             the GEMM); may equal c exactly.  beta != 0 requires c_in.
 * Other arguments as fsg_gemm_bf16.
 */
FSG_API fsg_status fsg_gemm_bf16_ex(const void* a, int64_t lda, int64_t stride_a, const void* b,
                                    int64_t ldb, int64_t stride_b, int trans_b, void* c,
                                    int64_t ldc, int64_t stride_c, int64_t m, int64_t n,
                                    int64_t k, int64_t batch, float alpha,
                                    const float* alpha_col, const void* bias, int bias_f32,
                                    fsg_act act, const void* c_in, int64_t ld_cin,
                                    int64_t stride_cin, float beta, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream);

/* Detail of the last non-OK status on the calling thread (never NULL). */
FSG_API const char* fsg_last_error_message(void);

#ifdef __cplusplus
}
#endif
#endif /* FSGEMM_H */
