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

using Key = std::tuple<int, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int, int64_t,
                       int64_t, int64_t, int64_t, bool, size_t>;

struct Plan {
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
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

}  // namespace

extern "C" {

const char* fsg_last_error_message(void) { return g_msg; }

fsg_status fsg_gemm_bf16(const void* a, int64_t lda, int64_t stride_a, const void* b, int64_t ldb,
                         int64_t stride_b, int trans_b, void* c, int64_t ldc, int64_t stride_c,
                         int64_t m, int64_t n, int64_t k, int64_t batch, float alpha,
                         const void* bias, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  g_msg[0] = '\0';
  if (trans_b != 0 && trans_b != 1) return fail(FSG_ERR_BAD_ARGUMENT, "trans_b=%d", trans_b);
  if (!std::isfinite(alpha)) return fail(FSG_ERR_BAD_ARGUMENT, "alpha is not finite");
  if (m < 0 || n < 0 || k < 0 || batch < 1 || batch > INT32_MAX)
    return fail(FSG_ERR_BAD_SHAPE, "m=%lld n=%lld k=%lld batch=%lld", (long long)m, (long long)n,
                (long long)k, (long long)batch);
  if (lda < k || ldc < n || ldb < (trans_b ? k : n))
    return fail(FSG_ERR_BAD_STRIDE, "lda=%lld ldb=%lld ldc=%lld", (long long)lda,
                (long long)ldb, (long long)ldc);
  if (m == 0 || n == 0) return FSG_OK;
  if (k == 0) return fail(FSG_ERR_BAD_SHAPE, "k=0 is not supported");
  if (!a || !b || !c) return fail(FSG_ERR_NULL_POINTER, "a, b and c are required");
  if (workspace_bytes && !workspace) return fail(FSG_ERR_NULL_POINTER, "workspace is NULL");
  if (batch == 1) stride_a = stride_b = stride_c = 0;

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

  const Key key{dev, m, n, k, lda, ldb, ldc, trans_b, stride_a, stride_b, stride_c, batch,
                bias != nullptr, workspace_bytes};
  auto pit = st.plans.find(key);
  if (pit == st.plans.end()) {
    Plan p;
    LT(hipblasLtMatmulDescCreate(&p.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F));
    // hipBLASLt "A" = row-major B: column-major [n, k] (trans_b = 0) or
    // stored column-major [k, n] used transposed (trans_b = 1).
    int32_t opa = trans_b ? HIPBLAS_OP_T : HIPBLAS_OP_N, opb = HIPBLAS_OP_N;
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opa, sizeof(opa)));
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opb, sizeof(opb)));
    if (bias) {
      uint32_t epi = HIPBLASLT_EPILOGUE_BIAS;
      int32_t bt = HIP_R_16BF;
      LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_EPILOGUE, &epi, sizeof(epi)));
      LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_BIAS_DATA_TYPE, &bt,
                                         sizeof(bt)));
    }
    fsg_status s2;
    if ((s2 = trans_b ? make_layout(&p.la, k, n, ldb, batch, stride_b)
                      : make_layout(&p.la, n, k, ldb, batch, stride_b)) != FSG_OK)
      return s2;
    if ((s2 = make_layout(&p.lb, k, m, lda, batch, stride_a)) != FSG_OK) return s2;
    if ((s2 = make_layout(&p.lc, n, m, ldc, batch, stride_c)) != FSG_OK) return s2;

    hipblasLtMatmulPreference_t pref = nullptr;
    LT(hipblasLtMatmulPreferenceCreate(&pref));
    uint64_t ws = workspace_bytes;
    LT(hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws,
                                             sizeof(ws)));
    hipblasLtMatmulHeuristicResult_t res[1];
    int found = 0;
    hipblasStatus_t hs = hipblasLtMatmulAlgoGetHeuristic(handle, p.desc, p.la, p.lb, p.lc, p.lc,
                                                         pref, 1, res, &found);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (hs != HIPBLAS_STATUS_SUCCESS || found < 1)
      return fail(FSG_ERR_NO_ALGO, "no hipBLASLt algorithm (status %d, found %d)", int(hs), found);
    p.algo = res[0].algo;
    pit = st.plans.emplace(key, p).first;
  }
  Plan& p = pit->second;
  if (bias) {
    LT(hipblasLtMatmulDescSetAttribute(p.desc, HIPBLASLT_MATMUL_DESC_BIAS_POINTER, &bias,
                                       sizeof(bias)));
  }
  const float beta = 0.f;
  LT(hipblasLtMatmul(handle, p.desc, &alpha, b, p.la, a, p.lb, &beta, c, p.lc, c, p.lc, &p.algo,
                     workspace, workspace_bytes, stream));
  return FSG_OK;
}

}  // extern "C"
