// libfsgemm: row-major bf16 GEMMs as plain hipBLASLt calls (see fsgemm.h).
//
// hipBLASLt is column-major.  A row-major [r, c] matrix with row stride ld is
// the column-major [c, r] matrix with the same ld, so
//     C = A op(B)   (row-major)   <=>   C^T = op(B)^T A^T   (column-major)
// and the call passes B as hipBLASLt's "A" operand and A as its "B" operand.
// The BIAS epilogue adds a vector along the rows of the column-major result,
// which is the per-column bias of the row-major C.
#include <hipblaslt/hipblaslt.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <map>
#include <mutex>
#include <tuple>

#include "fsgemm.h"

namespace {

thread_local char g_msg[512] = "";

fsg_status fail(fsg_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return st;
}

struct Req {
  const void* a; int64_t lda, stride_a;
  const void* b; int64_t ldb, stride_b; int trans_b;
  void* c; int64_t ldc, stride_c;
  int64_t m, n, k, batch;
  float alpha; const float* alpha_col;
  const void* bias; int bias_f32;
  fsg_act act;
  const void* c_in; int64_t ld_cin, stride_cin; float beta;
  void* workspace; size_t workspace_bytes;
};

using Key = std::tuple<int, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int, int64_t,
                       int64_t, int64_t, int64_t, size_t, int, int, int, int, int64_t, int64_t>;

struct Plan {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr, lcin = nullptr;
  hipblasLtMatmulAlgo_t algo{};
};

struct State {
  std::mutex mu;
  std::map<int, hipblasLtHandle_t> handles;
  std::map<Key, Plan> plans;
};
State& state() {
  static State* s = new State();   // never destroyed: handles outlive static teardown
  return *s;
}

#define LT(call)                                                                       \
  do {                                                                                 \
    hipblasStatus_t _s = (call);                                                       \
    if (_s != HIPBLAS_STATUS_SUCCESS) return fail(FSG_ERR_LIBRARY, "%s -> %d", #call, int(_s)); \
  } while (0)

fsg_status make_layout(hipblasLtMatrixLayout_t* l, uint64_t rows, uint64_t cols, int64_t ld,
                       int64_t batch, int64_t stride) {
  LT(hipblasLtMatrixLayoutCreate(l, HIP_R_16BF, rows, cols, ld));
  if (batch > 1) {
    int32_t bc = int32_t(batch);
    LT(hipblasLtMatrixLayoutSetAttribute(*l, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc, sizeof(bc)));
    LT(hipblasLtMatrixLayoutSetAttribute(*l, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &stride,
                                         sizeof(stride)));
  }
  return FSG_OK;
}

uint32_t epilogue_of(bool bias, fsg_act act) {
  switch (act) {
    case FSG_ACT_GELU: return bias ? HIPBLASLT_EPILOGUE_GELU_BIAS : HIPBLASLT_EPILOGUE_GELU;
    case FSG_ACT_RELU: return bias ? HIPBLASLT_EPILOGUE_RELU_BIAS : HIPBLASLT_EPILOGUE_RELU;
    default: return bias ? HIPBLASLT_EPILOGUE_BIAS : HIPBLASLT_EPILOGUE_DEFAULT;
  }
}

hipblasStatus_t launch(hipblasLtHandle_t h, const Plan& p, const Req& r,
                       const hipblasLtMatmulAlgo_t* algo, hipStream_t stream) {
  const void* alpha = r.alpha_col ? static_cast<const void*>(r.alpha_col)
                                  : static_cast<const void*>(&r.alpha);
  const bool has_cin = r.c_in != nullptr && r.beta != 0.f;
  return hipblasLtMatmul(h, p.desc, alpha, r.b, p.la, r.a, p.lb, &r.beta,
                         has_cin ? r.c_in : r.c, has_cin ? p.lcin : p.lc, r.c, p.lc, algo,
                         r.workspace, r.workspace_bytes, stream);
}

fsg_status run(const Req& r, hipStream_t stream) {
  if (r.trans_b != 0 && r.trans_b != 1) return fail(FSG_ERR_BAD_ARGUMENT, "trans_b=%d", r.trans_b);
  if (!std::isfinite(r.alpha) || !std::isfinite(r.beta))
    return fail(FSG_ERR_BAD_ARGUMENT, "alpha and beta must be finite");
  if (r.act < FSG_ACT_NONE || r.act > FSG_ACT_RELU)
    return fail(FSG_ERR_BAD_ARGUMENT, "act=%d", int(r.act));
  if (r.bias_f32 != 0 && r.bias_f32 != 1) return fail(FSG_ERR_BAD_ARGUMENT, "bias_f32=%d", r.bias_f32);
  if (r.alpha_col && r.alpha != 1.f)
    return fail(FSG_ERR_BAD_ARGUMENT, "alpha must be 1 with a per-column alpha vector");
  if (r.m < 0 || r.n < 0 || r.k < 0 || r.batch < 1 || r.batch > INT32_MAX)
    return fail(FSG_ERR_BAD_SHAPE, "m=%lld n=%lld k=%lld batch=%lld", (long long)r.m,
                (long long)r.n, (long long)r.k, (long long)r.batch);
  if (r.lda < r.k || r.ldc < r.n || r.ldb < (r.trans_b ? r.k : r.n))
    return fail(FSG_ERR_BAD_STRIDE, "lda=%lld ldb=%lld ldc=%lld", (long long)r.lda,
                (long long)r.ldb, (long long)r.ldc);
  const bool has_cin = r.c_in != nullptr && r.beta != 0.f;
  if (has_cin && r.ld_cin < r.n)
    return fail(FSG_ERR_BAD_STRIDE, "ld_cin=%lld < n", (long long)r.ld_cin);
  if (r.m == 0 || r.n == 0) return FSG_OK;
  if (r.k == 0) return fail(FSG_ERR_BAD_SHAPE, "k=0 is not supported");
  if (!r.a || !r.b || !r.c) return fail(FSG_ERR_NULL_POINTER, "a, b and c are required");
  if (r.beta != 0.f && !r.c_in) return fail(FSG_ERR_NULL_POINTER, "beta != 0 needs c_in");
  if (r.workspace_bytes && !r.workspace) return fail(FSG_ERR_NULL_POINTER, "workspace is NULL");
  Req q = r;
  if (q.batch == 1) q.stride_a = q.stride_b = q.stride_c = q.stride_cin = 0;
  if (!has_cin) q.ld_cin = q.stride_cin = 0;

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(FSG_ERR_HIP, "hipGetDevice failed");

  State& st = state();
  std::lock_guard<std::mutex> lock(st.mu);
  auto hit = st.handles.find(dev);
  if (hit == st.handles.end()) {
    hipblasLtHandle_t h = nullptr;
    LT(hipblasLtCreate(&h));
    hit = st.handles.emplace(dev, h).first;
  }
  hipblasLtHandle_t handle = hit->second;

  const Key key{dev, q.m, q.n, q.k, q.lda, q.ldb, q.ldc, q.trans_b, q.stride_a, q.stride_b,
                q.stride_c, q.batch, q.workspace_bytes, (q.bias ? 1 : 0) | (q.bias_f32 << 1),
                int(q.act), q.alpha_col ? 1 : 0, has_cin ? 1 : 0, q.ld_cin, q.stride_cin};
  auto pit = st.plans.find(key);
  if (pit == st.plans.end()) {
    Plan p;
    LT(hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F));
    // hipBLASLt "A" = row-major B: column-major [n, k] (trans_b = 0) or
    // stored column-major [k, n] used transposed (trans_b = 1).
    int32_t opa = q.trans_b ? HIPBLAS_OP_T : HIPBLAS_OP_N, opb = HIPBLAS_OP_N;
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opa, sizeof(opa)));
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opb, sizeof(opb)));
    const uint32_t epi = epilogue_of(q.bias != nullptr, q.act);
    if (epi != HIPBLASLT_EPILOGUE_DEFAULT)
      LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_EPILOGUE, &epi, sizeof(epi)));
    if (q.bias) {
      int32_t bt = q.bias_f32 ? HIP_R_32F : HIP_R_16BF;
      LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_BIAS_DATA_TYPE, &bt,
                                         sizeof(bt)));
    }
    if (q.alpha_col) {
      int32_t pm = HIPBLASLT_POINTER_MODE_ALPHA_DEVICE_VECTOR_BETA_HOST;
      LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_POINTER_MODE, &pm,
                                         sizeof(pm)));
    }
    fsg_status s2;
    if ((s2 = q.trans_b ? make_layout(&p.la, q.k, q.n, q.ldb, q.batch, q.stride_b)
                        : make_layout(&p.la, q.n, q.k, q.ldb, q.batch, q.stride_b)) != FSG_OK)
      return s2;
    if ((s2 = make_layout(&p.lb, q.k, q.m, q.lda, q.batch, q.stride_a)) != FSG_OK) return s2;
    if ((s2 = make_layout(&p.lc, q.n, q.m, q.ldc, q.batch, q.stride_c)) != FSG_OK) return s2;
    if (has_cin &&
        (s2 = make_layout(&p.lcin, q.n, q.m, q.ld_cin, q.batch, q.stride_cin)) != FSG_OK)
      return s2;
    hipblasLtMatmulPreference_t pref = nullptr;
    LT(hipblasLtMatmulPreferenceCreate(&pref));
    uint64_t ws = q.workspace_bytes;
    LT(hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws,
                                             sizeof(ws)));
    hipblasLtMatmulHeuristicResult_t res[1];
    int found = 0;
    hipblasStatus_t hs = hipblasLtMatmulAlgoGetHeuristic(handle, p.desc, p.la, p.lb,
                                                         has_cin ? p.lcin : p.lc, p.lc, pref, 1,
                                                         res, &found);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (hs != HIPBLAS_STATUS_SUCCESS || found < 1)
      return fail(FSG_ERR_NO_ALGO, "no hipBLASLt algorithm (status %d, found %d)", int(hs), found);
    p.algo = res[0].algo;
    pit = st.plans.emplace(key, p).first;
  }
  Plan& p = pit->second;
  if (q.bias)
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_BIAS_POINTER, &q.bias,
                                       sizeof(q.bias)));
  LT(launch(handle, p, q, &p.algo, stream));
  return FSG_OK;
}

}  // namespace

extern "C" {

const char* fsg_last_error_message(void) { return g_msg; }

fsg_status fsg_gemm_bf16(const void* a, int64_t lda, int64_t stride_a, const void* b, int64_t ldb,
                         int64_t stride_b, int trans_b, void* c, int64_t ldc, int64_t stride_c,
                         int64_t m, int64_t n, int64_t k, int64_t batch, float alpha,
                         const void* bias, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  g_msg[0] = '\0';
  Req r{a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c, m, n, k, batch,
        alpha, nullptr, bias, 0, FSG_ACT_NONE, nullptr, 0, 0, 0.f, workspace, workspace_bytes};
  return run(r, stream);
}

fsg_status fsg_gemm_bf16_ex(const void* a, int64_t lda, int64_t stride_a, const void* b,
                            int64_t ldb, int64_t stride_b, int trans_b, void* c, int64_t ldc,
                            int64_t stride_c, int64_t m, int64_t n, int64_t k, int64_t batch,
                            float alpha, const float* alpha_col, const void* bias, int bias_f32,
                            fsg_act act, const void* c_in, int64_t ld_cin, int64_t stride_cin,
                            float beta, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  g_msg[0] = '\0';
  Req r{a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c, m, n, k, batch,
        alpha, alpha_col, bias, bias_f32, act, c_in, ld_cin, stride_cin, beta, workspace,
        workspace_bytes};
  return run(r, stream);
}

}  // extern "C"
