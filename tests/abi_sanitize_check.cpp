// Host-only check of libfusedsub's C-ABI layer (csrc/api.hip) under
// AddressSanitizer and UndefinedBehaviorSanitizer.
//
// api.hip is compiled as plain C++ (it holds no device code) and linked with
// stand-ins for the three HIP runtime calls it makes and for the kernel
// launchers of launch.hpp.  The launchers record what they are handed, so
// every entry point runs its whole host path -- validation, overflow guards,
// alias checks, the choice of the 16-byte and aligned-body paths -- without a
// GPU.  Two parts:
//   1. fixed cases with known statuses and known path choices;
//   2. a deterministic sweep over extreme integers and odd pointers for every
//      entry point; any status may come back, but a sanitizer report, a
//      launch for an empty or rejected problem, or a launch whose arguments
//      differ from the call's is a failure.
// Exit status 0 means every check passed; the sanitizers abort on their own
// reports (-fno-sanitize-recover).
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "fusedsub.h"
#include "launch.hpp"

// ---- stand-ins: the HIP runtime ---------------------------------------------
static int g_cus = 256;
extern "C" hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
extern "C" hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = g_cus;
  return hipSuccess;
}
extern "C" const char* hipGetErrorString(hipError_t) { return "stand-in launch error"; }

// ---- stand-ins: the kernel launchers (record their arguments) ---------------
namespace rec {
int launches = 0;
hipError_t result = hipSuccess;
fs::PointwiseArgs pw;
fs::ProgramArgs pg;
fs::SoftmaxArgs sm;
fs::LayerNormArgs ln;
fs::EpilogueArgs ep;
bool ep_maxlse = false;
fs::ReduceArgs rd;
fs::CopyStridedArgs cs;
int64_t copy_bytes = 0;
}  // namespace rec

namespace fs {
hipError_t launch_pointwise(const PointwiseArgs& a, int, hipStream_t) { ++rec::launches; rec::pw = a; return rec::result; }
hipError_t launch_program(const ProgramArgs& a, int, hipStream_t) { ++rec::launches; rec::pg = a; return rec::result; }
hipError_t launch_softmax(const SoftmaxArgs& a, int, hipStream_t) { ++rec::launches; rec::sm = a; return rec::result; }
hipError_t launch_layernorm(const LayerNormArgs& a, int, hipStream_t) { ++rec::launches; rec::ln = a; return rec::result; }
hipError_t launch_epilogue(const EpilogueArgs& a, int, hipStream_t) { ++rec::launches; rec::ep = a; rec::ep_maxlse = false; return rec::result; }
hipError_t launch_epilogue_maxlse(const EpilogueArgs& a, int, hipStream_t) { ++rec::launches; rec::ep = a; rec::ep_maxlse = true; return rec::result; }
hipError_t launch_reduce(const ReduceArgs& a, int, hipStream_t) { ++rec::launches; rec::rd = a; return rec::result; }
hipError_t launch_copy(const void*, void*, int64_t bytes, int, hipStream_t) { ++rec::launches; rec::copy_bytes = bytes; return rec::result; }
hipError_t launch_copy_strided(const CopyStridedArgs& a, int, hipStream_t) { ++rec::launches; rec::cs = a; return rec::result; }
}  // namespace fs

// ---- checks -------------------------------------------------------------------
static int g_failures = 0;
#define EXPECT(cond, ...)                                                       \
  do {                                                                          \
    if (!(cond)) {                                                              \
      ++g_failures;                                                             \
      std::fprintf(stderr, "FAILED %s:%d: %s -- ", __FILE__, __LINE__, #cond); \
      std::fprintf(stderr, __VA_ARGS__);                                        \
      std::fprintf(stderr, "\n");                                               \
    }                                                                           \
  } while (0)

// fake device addresses: never dereferenced (the launchers are stand-ins)
static const char* P(uintptr_t a) { return reinterpret_cast<const char*>(a); }
static char* W(uintptr_t a) { return reinterpret_cast<char*>(a); }
static const uintptr_t A = 0x10000000, B = 0x20000000, C = 0x30000000, D = 0x40000000;

static void fixed_cases() {
  // pointwise: statuses
  auto pw = [](const void* x, int64_t ldx, const void* b, const void* r, int64_t ldr, void* y,
               int64_t ldy, int64_t rows, int64_t cols, float s, int act, int dt) {
    return fs_pointwise_chain(x, ldx, b, r, ldr, y, ldy, rows, cols, s, fs_act(act), fs_dtype(dt), 0);
  };
  EXPECT(pw(nullptr, 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_ERR_NULL_POINTER, "x null");
  EXPECT(pw(P(A), 63, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_ERR_BAD_STRIDE, "ld_x");
  EXPECT(pw(P(A), 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 9, 0) == FS_ERR_BAD_ARGUMENT, "act");
  EXPECT(pw(P(A + 2), 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_ERR_BAD_ARGUMENT, "align");
  EXPECT(pw(P(A), 64, nullptr, nullptr, 0, W(A + 4), 64, 4, 64, 1.f, 0, 0) == FS_ERR_ALIASING, "overlap");
  EXPECT(pw(P(A), 64, nullptr, nullptr, 0, W(A), 64, 4, 64, 1.f, 0, 0) == FS_OK, "in place");
  EXPECT(pw(P(A), INT64_MAX, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_ERR_BAD_SHAPE, "ld overflow");
  EXPECT(std::strstr(fs_last_error_message(), "overflows") != nullptr, "%s", fs_last_error_message());
  // pointwise: path choice
  pw(P(A), 64, P(C), P(D), 64, W(B), 64, 4, 64, 1.f, 1, 0);
  EXPECT(rec::pw.vec && !rec::pw.shifted && rec::pw.rows == 4 && rec::pw.cols == 64, "fp32 vec");
  pw(P(A), 1001, nullptr, P(D), 1001, W(B), 1001, 4, 1001, 1.f, 0, 1);
  EXPECT(!rec::pw.vec && rec::pw.shifted, "bf16 1001 columns share a phase per row");
  pw(P(A + 2), 1001, nullptr, nullptr, 0, W(B), 1001, 4, 1001, 1.f, 0, 1);
  EXPECT(!rec::pw.vec && !rec::pw.shifted, "x and y at different phases");
  // a launch error becomes FS_ERR_HIP with the runtime's text
  rec::result = hipErrorInvalidValue;
  EXPECT(pw(P(A), 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_ERR_HIP, "launch error");
  EXPECT(std::strstr(fs_last_error_message(), "stand-in launch error") != nullptr, "%s", fs_last_error_message());
  rec::result = hipSuccess;
  EXPECT(pw(P(A), 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, 0, 0) == FS_OK && fs_last_error_message()[0] == 0,
         "message cleared");

  // pointwise program: operations validated and copied, operands it does
  // not read dropped, the vector path for aligned rows
  {
    const fs_op chain[4] = {{FS_OP_ADD_BIAS, 0.f, 0.f}, {FS_OP_SCALE, 0.5f, 0.f},
                            {FS_OP_CLAMP, -1.f, 1.f}, {FS_OP_GELU_ERF, 0.f, 0.f}};
    EXPECT(fs_pointwise_program(P(A), 64, chain, 4, P(C), P(D), P(D + 4096), 64, W(B), 64, 4, 64,
                                FS_F32, 0) == FS_OK &&
               rec::pg.prog.n == 4 && rec::pg.prog.code[2] == FS_OP_CLAMP && rec::pg.prog.b[2] == 1.f &&
               rec::pg.bias == P(C) && rec::pg.col == nullptr && rec::pg.res == nullptr && rec::pg.vec,
           "program recorded");
    EXPECT(fs_pointwise_program(P(A), 63, chain, 4, P(C), nullptr, nullptr, 0, W(B), 63, 4, 63, FS_F32, 0) ==
               FS_OK && !rec::pg.vec && rec::pg.shifted, "odd width, one phase: aligned body");
    EXPECT(fs_pointwise_program(P(A), 63, chain, 4, P(C), nullptr, nullptr, 0, W(B), 63, 4, 7, FS_F32, 0) ==
               FS_OK && !rec::pg.vec && !rec::pg.shifted, "rows under two vectors: element path");
    EXPECT(fs_pointwise_program(P(A), 64, chain, 4, nullptr, nullptr, nullptr, 0, W(B), 64, 4, 64, FS_F32, 0) ==
               FS_ERR_NULL_POINTER, "bias read but NULL");
    EXPECT(fs_pointwise_program(P(A), 64, chain, 4, P(B + 64), nullptr, nullptr, 0, W(B), 64, 4, 64, FS_F32,
                                0) == FS_ERR_ALIASING, "bias inside y");
    const fs_op bad_clamp[1] = {{FS_OP_CLAMP, 1.f, -1.f}};
    EXPECT(fs_pointwise_program(P(A), 64, bad_clamp, 1, nullptr, nullptr, nullptr, 0, W(B), 64, 4, 64, FS_F32,
                                0) == FS_ERR_BAD_ARGUMENT, "clamp bounds out of order");
    const fs_op open_clamp[1] = {{FS_OP_CLAMP, -INFINITY, 0.f}};
    EXPECT(fs_pointwise_program(P(A), 64, open_clamp, 1, nullptr, nullptr, nullptr, 0, W(B), 64, 4, 64, FS_F32,
                                0) == FS_OK, "one-sided clamp");
    const fs_op bad_code[1] = {{13, 0.f, 0.f}};
    EXPECT(fs_pointwise_program(P(A), 64, bad_code, 1, nullptr, nullptr, nullptr, 0, W(B), 64, 4, 64, FS_F32,
                                0) == FS_ERR_BAD_ARGUMENT, "unknown code");
    EXPECT(fs_pointwise_program(P(A), 64, chain, FS_PROGRAM_MAX_OPS + 1, P(C), nullptr, nullptr, 0, W(B), 64,
                                4, 64, FS_F32, 0) == FS_ERR_BAD_ARGUMENT, "too many operations");
    EXPECT(fs_pointwise_program(P(A), 64, nullptr, 0, nullptr, nullptr, nullptr, 0, W(B), 64, 4, 64, FS_BF16,
                                0) == FS_OK && rec::pg.prog.n == 0, "empty program: a copy");
    const fs_op res_op[1] = {{FS_OP_MUL_RESIDUAL, 0.f, 0.f}};
    EXPECT(fs_pointwise_program(P(A), 64, res_op, 1, nullptr, nullptr, P(B), 64, W(B), 64, 4, 64, FS_BF16, 0) ==
               FS_OK && rec::pg.res == P(B), "in place on the residual");
  }

  // epilogue reductions: sum and mean in one kernel family, max and log-sum-exp in another
  {
    float* ofp = reinterpret_cast<float*>(W(D));
    EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, P(B), FS_BF16, reinterpret_cast<const float*>(P(C)),
                                   FS_ACT_SIGMOID, FS_REDUCE_SUM, ofp, 16, 8192, 0) == FS_OK && !rec::ep_maxlse,
           "sum epilogue");
    EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, P(B), FS_BF16, reinterpret_cast<const float*>(P(C)),
                                   FS_ACT_RELU, FS_REDUCE_MAX, ofp, 16, 8192, 0) == FS_OK && rec::ep_maxlse &&
               rec::ep.reduce == FS_REDUCE_MAX && rec::ep.vec && rec::ep.coef_vec,
           "max epilogue");
    EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, nullptr, FS_BF16, nullptr, FS_ACT_NONE,
                                   FS_REDUCE_LOGSUMEXP, ofp, 16, 8192, 0) == FS_OK && rec::ep_maxlse &&
               rec::ep.reduce == FS_REDUCE_LOGSUMEXP, "log-sum-exp epilogue");
    EXPECT(fs_gemm_epilogue_reduce(P(A), 0, FS_BF16, nullptr, FS_BF16, nullptr, FS_ACT_NONE, FS_REDUCE_MAX, ofp,
                                   16, 0, 0) == FS_ERR_BAD_SHAPE, "max over no columns");
    EXPECT(fs_gemm_epilogue_reduce(P(A), 64, FS_BF16, nullptr, FS_BF16, nullptr, FS_ACT_NONE, fs_reduce(4), ofp,
                                   16, 64, 0) == FS_ERR_BAD_ARGUMENT, "reduce out of range");
  }

  // softmax
  EXPECT(fs_row_softmax(P(A), 128, P(C), 128, FS_BF16, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK, "ok");
  EXPECT(rec::sm.vec, "softmax vec");
  EXPECT(fs_row_softmax(P(A), 128, P(B + 64), 128, FS_BF16, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) ==
             FS_ERR_ALIASING, "mask overlaps y");
  EXPECT(fs_row_softmax(P(A), 128, nullptr, 0, FS_BF16, W(B), 128, 4, 128, 0.125f, -1, FS_BF16, 0) ==
             FS_ERR_BAD_ARGUMENT, "q_len");
  EXPECT(fs_row_softmax(P(A), 1 << 25, nullptr, 0, FS_BF16, W(B), 1 << 25, 4, FS_SOFTMAX_MAX_COLS + 1,
                        1.f, 0, FS_BF16, 0) == FS_ERR_BAD_SHAPE, "too wide");
  // byte masks: the 16-byte path of x with 8-byte (bf16 x) or 4-byte (fp32 x)
  // mask vectors; any byte address is accepted
  EXPECT(fs_row_softmax(P(A), 128, P(C + 8), 136, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             rec::sm.vec && rec::sm.mask_dtype == FS_U8, "byte mask, 8-byte vectors");
  EXPECT(fs_row_softmax(P(A), 128, P(C + 4), 128, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.vec && !rec::sm.shifted, "byte mask off its 8-byte unit: element path");
  EXPECT(fs_row_softmax(P(A), 128, P(C), 132, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.vec, "byte mask rows 132 bytes apart: element path");
  EXPECT(fs_row_softmax(P(A), 128, P(C + 4), 132, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_F32, 0) == FS_OK &&
             rec::sm.vec, "byte mask, 4-byte vectors for fp32 x");
  EXPECT(fs_row_softmax(P(A), 128, P(C + 3), 128, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_F32, 0) == FS_OK &&
             !rec::sm.vec, "byte mask at an odd address");
  // a bf16 mask beside fp32 x: 8 bytes of mask per 16-byte vector of x
  EXPECT(fs_row_softmax(P(A), 128, P(C + 8), 132, FS_BF16, W(B), 128, 4, 128, 0.125f, 0, FS_F32, 0) == FS_OK &&
             rec::sm.vec, "bf16 mask on 8-byte boundaries with fp32 x");
  EXPECT(fs_row_softmax(P(A), 128, P(C + 4), 132, FS_BF16, W(B), 128, 4, 128, 0.125f, 0, FS_F32, 0) == FS_OK &&
             !rec::sm.vec, "bf16 mask off its 8-byte unit");
  // an fp32 mask beside bf16 x: 32 bytes of mask per vector, 16-byte loads
  EXPECT(fs_row_softmax(P(A), 128, P(C + 16), 132, FS_F32, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             rec::sm.vec, "fp32 mask on 16-byte boundaries with bf16 x");
  EXPECT(fs_row_softmax(P(A), 128, P(C + 8), 132, FS_F32, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.vec, "fp32 mask off its 16-byte unit");
  // odd widths: the aligned-body path when the byte mask's rows start at x's
  // element phase within their 8-byte (bf16 x) or 4-byte (fp32 x) units
  EXPECT(fs_row_softmax(P(A), 1001, P(C), 1001, FS_U8, W(B), 1001, 4, 1001, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.vec && rec::sm.shifted, "contiguous byte mask: aligned body");
  EXPECT(fs_row_softmax(P(A + 6), 1001, P(C + 3), 1009, FS_U8, W(B + 6), 1001, 4, 1001, 0.125f, 0, FS_BF16, 0) ==
             FS_OK && rec::sm.shifted, "byte mask at x's phase, rows 8 bytes wider");
  EXPECT(fs_row_softmax(P(A), 1001, P(C + 1), 1001, FS_U8, W(B), 1001, 4, 1001, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.vec && !rec::sm.shifted, "byte mask off x's phase: element path");
  EXPECT(fs_row_softmax(P(A), 1001, P(C), 1005, FS_U8, W(B), 1001, 4, 1001, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.shifted, "byte mask rows drifting from x's phase: element path");
  EXPECT(fs_row_softmax(P(A + 4), 1001, P(C + 1), 1001, FS_U8, W(B + 4), 1001, 4, 1001, 0.125f, 0, FS_F32, 0) ==
             FS_OK && rec::sm.shifted, "fp32 x one element in, byte mask one byte in");
  EXPECT(fs_row_softmax(P(A), 1001, P(C), 1001, FS_F32, W(B), 1001, 4, 1001, 0.125f, 0, FS_BF16, 0) == FS_OK &&
             !rec::sm.shifted, "fp32 mask beside bf16 x: element path");
  EXPECT(fs_row_softmax(P(A), 128, P(B + 511), 128, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) ==
             FS_ERR_ALIASING, "byte mask's last byte inside y");
  EXPECT(fs_row_softmax(P(A), 128, P(B + 1024 + 0), 128, FS_U8, W(B), 128, 4, 128, 0.125f, 0, FS_BF16, 0) == FS_OK,
         "byte mask just past y");
  EXPECT(fs_row_softmax(P(A), 128, nullptr, 0, FS_BF16, W(B), 128, 4, 128, 0.125f, 0, FS_U8, 0) ==
             FS_ERR_UNSUPPORTED_DTYPE, "bytes are a mask dtype only");
  EXPECT(fs_pointwise_chain(P(A), 64, nullptr, nullptr, 0, W(B), 64, 4, 64, 1.f, FS_ACT_NONE, FS_U8, 0) ==
             FS_ERR_UNSUPPORTED_DTYPE, "no byte pointwise chain");
  EXPECT(fs_gemm_epilogue_reduce(P(A), 64, FS_BF16, P(C), FS_U8, nullptr, FS_ACT_NONE, FS_REDUCE_SUM,
                                 reinterpret_cast<float*>(W(B)), 4, 64, 0) == FS_ERR_UNSUPPORTED_DTYPE,
         "no byte bias");
  EXPECT(fs_causal_softmax_trimmed(P(A), 512, W(B), 512, 1024, 512, 0.125f, 512, 3, FS_BF16, 0) ==
             FS_ERR_BAD_ARGUMENT, "block not a power of two");
  EXPECT(fs_causal_softmax_trimmed(P(A), 512, W(B), 512, 1024, 512, 0.125f, 512, 128, FS_BF16, 0) == FS_OK &&
             rec::sm.trim_shift == 7, "trim shift");

  // layernorm / rmsnorm: the aligned, the aligned-body and the element path
  EXPECT(fs_layernorm_residual(P(A), 1024, P(C), 1024, P(D), P(D + 4096), W(B), 1024, nullptr, 0, 16, 1024,
                               1e-5f, FS_BF16, 0) == FS_OK && rec::ln.vec && !rec::ln.rms, "ln vec");
  EXPECT(fs_layernorm_residual(P(A), 4095, P(C), 4095, P(D), P(D + 16384), W(B), 4095, nullptr, 0, 16, 4095,
                               1e-5f, FS_BF16, 0) == FS_OK && !rec::ln.vec && rec::ln.shifted, "ln shifted");
  EXPECT(fs_layernorm_residual(P(A), 1024, nullptr, 0, nullptr, nullptr, W(B), 1024, W(A + 64), 1024, 16,
                               1024, 1e-5f, FS_BF16, 0) == FS_ERR_ALIASING, "residual_out partly over x");
  EXPECT(fs_layernorm_residual(P(A), 1024, nullptr, 0, nullptr, nullptr, W(B), 1024, W(A), 1024, 16, 1024,
                               1e-5f, FS_BF16, 0) == FS_OK, "residual_out exactly x (in place)");
  EXPECT(fs_layernorm_residual(P(A), 1024, nullptr, 0, nullptr, nullptr, W(B), 1024, W(B + 2048), 1024, 16,
                               1024, 1e-5f, FS_BF16, 0) == FS_ERR_ALIASING, "y overlaps residual_out");
  EXPECT(fs_layernorm_residual(P(A), 1024, nullptr, 0, nullptr, nullptr, W(B), 1024, nullptr, 0, 16, 1024,
                               -1.f, FS_BF16, 0) == FS_ERR_BAD_ARGUMENT, "eps < 0");
  EXPECT(fs_rmsnorm_residual(P(A), 1024, P(C), 1024, P(D), W(B), 1024, W(C), 1024, 16, 1024, 1e-6f,
                             FS_F32, 0) == FS_OK && rec::ln.rms, "rms in place on the residual");

  // row reductions and argmax
  float* of = reinterpret_cast<float*>(W(C));
  int64_t* oi = reinterpret_cast<int64_t*>(W(C));
  EXPECT(fs_row_reduce(P(A), 4096, FS_BF16, FS_ROW_SUM, of, 16, 4096, 0) == FS_OK && rec::rd.vec, "sum");
  EXPECT(fs_row_reduce(P(A), 4096, FS_BF16, fs_row_op(7), of, 16, 4096, 0) == FS_ERR_BAD_ARGUMENT, "op");
  EXPECT(fs_row_reduce(P(A), 0, FS_BF16, FS_ROW_MAX, of, 16, 0, 0) == FS_ERR_BAD_SHAPE, "max of nothing");
  EXPECT(fs_row_reduce(P(A), 0, FS_BF16, FS_ROW_LOGSUMEXP, of, 16, 0, 0) == FS_ERR_BAD_SHAPE,
         "log-sum-exp of nothing");
  EXPECT(fs_row_reduce(P(A), 4096, FS_BF16, FS_ROW_LOGSUMEXP, of, 16, 4096, 0) == FS_OK &&
             rec::rd.op == FS_ROW_LOGSUMEXP && rec::rd.vec, "log-sum-exp");
  EXPECT(fs_row_argmax(P(A), 4095, FS_BF16, oi, 16, 4095, 0) == FS_OK && rec::rd.out_i == oi && rec::rd.shifted,
         "argmax aligned body");
  EXPECT(fs_row_argmax(P(A), 4095, FS_BF16, nullptr, 16, 4095, 0) == FS_ERR_NULL_POINTER, "argmax out");

  // epilogue
  EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, P(B), FS_BF16, reinterpret_cast<const float*>(P(C)),
                                 FS_ACT_SIGMOID, FS_REDUCE_SUM, reinterpret_cast<float*>(W(D)), 8192, 8192, 0) ==
             FS_OK && rec::ep.vec && rec::ep.coef_vec, "epilogue");
  EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, nullptr, FS_BF16, nullptr, FS_ACT_NONE, FS_REDUCE_MEAN,
                                 reinterpret_cast<float*>(W(D)), 8192, 0, 0) == FS_ERR_BAD_SHAPE,
         "mean over no columns");
  EXPECT(fs_gemm_epilogue_reduce(P(A), 8192, FS_BF16, nullptr, FS_BF16, nullptr, FS_ACT_NONE, FS_REDUCE_SUM,
                                 reinterpret_cast<float*>(W(A + 64)), 8192, 8192, 0) == FS_ERR_ALIASING,
         "row_out inside C");

  // copies
  EXPECT(fs_copy(P(A), W(B), 1 << 20, 0) == FS_OK && rec::copy_bytes == (1 << 20), "copy");
  EXPECT(fs_copy(P(A), W(A + 16), 1 << 20, 0) == FS_ERR_ALIASING, "copy overlap");
  EXPECT(fs_copy_strided(P(A), 3072, 64, W(B), 64, 16384 * 64, 16384, 64, 48, FS_BF16, 0) == FS_OK &&
             rec::cs.batch == 48 && rec::cs.es == 2, "head split");
  EXPECT(fs_copy_strided(P(A), 64, 64, W(B), 64, 32, 4, 64, 3, FS_BF16, 0) == FS_ERR_BAD_STRIDE,
         "destination batches overlap");
  EXPECT(fs_copy_strided(P(A), 64, INT64_MAX / 4, W(B), 64, 256, 4, 64, 5, FS_BF16, 0) == FS_ERR_BAD_SHAPE,
         "batch stride overflow");

  // version and strings
  EXPECT(fs_abi_version() == FS_ABI_VERSION, "version");
  EXPECT(std::strncmp(fs_status_string(fs_status(99)), "FS_ERR_UNKNOWN", 14) == 0, "unknown status");
}

// ---- sweep ----------------------------------------------------------------------
static uint64_t g_state = 0x243F6A8885A308D3ull;
static uint64_t next() {   // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static int64_t pick_int() {
  static const int64_t v[] = {0, 1, -1, 2, 3, 7, 8, 15, 16, 17, 63, 64, 100, 1000, 1001, 1024, 4095, 4096,
                              16384, 65536, 65537, 1 << 24, (1 << 24) + 1, INT32_MAX / 2, INT32_MAX / 2 + 1,
                              INT32_MAX, int64_t(1) << 40, INT64_MAX / 8, INT64_MAX - 1, INT64_MAX, INT64_MIN};
  return v[next() % (sizeof(v) / sizeof(v[0]))];
}
static uintptr_t pick_ptr() {
  static const uintptr_t v[] = {0, A, A + 2, A + 4, A + 16, B, B + 2, C, D, A + 1024};
  return v[next() % (sizeof(v) / sizeof(v[0]))];
}
static float pick_float() {
  static const float v[] = {0.f, 1.f, -1.f, 0.125f, 1e-5f, 1e30f, __builtin_inff(), -__builtin_inff(),
                            __builtin_nanf("")};
  return v[next() % (sizeof(v) / sizeof(v[0]))];
}
static int pick_enum() { return int(next() % 6) - 1; }   // -1 .. 4

static void sweep(int n) {
  for (int i = 0; i < n; ++i) {
    const int64_t rows = pick_int(), cols = pick_int(), l1 = pick_int(), l2 = pick_int(), l3 = pick_int(),
                  l4 = pick_int();
    const uintptr_t p1 = pick_ptr(), p2 = pick_ptr(), p3 = pick_ptr(), p4 = pick_ptr(), p5 = pick_ptr(),
                    p6 = pick_ptr();
    const float f = pick_float();
    const int e1 = pick_enum(), e2 = pick_enum(), e3 = pick_enum();
    const bool empty = rows == 0 || cols == 0;
    int before = rec::launches;
    fs_status st = fs_pointwise_chain(P(p1), l1, P(p2), P(p3), l2, W(p4), l3, rows, cols, f, fs_act(e1),
                                      fs_dtype(e2), 0);
    if (rec::launches != before) {
      EXPECT(st == FS_OK && !empty && rec::pw.rows == rows && rec::pw.cols == cols && rec::pw.ld_x == l1 &&
                 rec::pw.x == P(p1) && rec::pw.y == W(p4),
             "pointwise sweep %d", i);
    }
    before = rec::launches;
    {
      fs_op prog[FS_PROGRAM_MAX_OPS];
      const int n_ops = int(next() % (FS_PROGRAM_MAX_OPS + 3)) - 1;   // -1 .. max + 1
      for (fs_op& o : prog) o = fs_op{int32_t(next() % 15) - 1, pick_float(), pick_float()};
      st = fs_pointwise_program(P(p1), l1, n_ops > 0 ? prog : nullptr, n_ops, P(p2), P(p3), P(p5), l2,
                                W(p4), l3, rows, cols, fs_dtype(e2), 0);
      if (rec::launches != before)
        EXPECT(st == FS_OK && !empty && rec::pg.rows == rows && rec::pg.prog.n == n_ops,
               "program sweep %d", i);
    }
    before = rec::launches;
    st = fs_row_softmax(P(p1), l1, P(p2), l2, fs_dtype(e3), W(p4), l3, rows, cols, f, pick_int(),
                        fs_dtype(e2), 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && !empty && rec::sm.rows == rows && rec::sm.cols == cols, "softmax sweep %d", i);
    before = rec::launches;
    st = fs_causal_softmax_trimmed(P(p1), l1, W(p4), l3, rows, cols, f, pick_int(), pick_int(), fs_dtype(e2), 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && !empty && rec::sm.trim_shift >= 0, "trimmed softmax sweep %d", i);
    before = rec::launches;
    st = fs_layernorm_residual(P(p1), l1, P(p2), l2, P(p3), P(p5), W(p4), l3, W(p6), l4, rows, cols, f,
                               fs_dtype(e2), 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && !empty && rec::ln.rows == rows && !rec::ln.rms, "layernorm sweep %d", i);
    before = rec::launches;
    st = fs_rmsnorm_residual(P(p1), l1, P(p2), l2, P(p3), W(p4), l3, W(p6), l4, rows, cols, f, fs_dtype(e2), 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && !empty && rec::ln.rms, "rmsnorm sweep %d", i);
    before = rec::launches;
    st = fs_row_reduce(P(p1), l1, fs_dtype(e2), fs_row_op(e1), reinterpret_cast<float*>(W(p4)), rows, cols, 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && rows > 0 && rec::rd.rows == rows, "reduce sweep %d", i);
    before = rec::launches;
    st = fs_row_argmax(P(p1), l1, fs_dtype(e2), reinterpret_cast<int64_t*>(W(p4)), rows, cols, 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && rows > 0 && cols > 0 && rec::rd.out_i != nullptr, "argmax sweep %d", i);
    before = rec::launches;
    st = fs_gemm_epilogue_reduce(P(p1), l1, fs_dtype(e2), P(p2), fs_dtype(e3),
                                 reinterpret_cast<const float*>(P(p3)), fs_act(e1), fs_reduce(pick_enum()),
                                 reinterpret_cast<float*>(W(p4)), rows, cols, 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && rows > 0 && rec::ep.rows == rows, "epilogue sweep %d", i);
    before = rec::launches;
    const int64_t batch = pick_int();
    st = fs_copy_strided(P(p1), l1, l2, W(p4), l3, l4, rows, cols, batch, fs_dtype(e2), 0);
    if (rec::launches != before)
      EXPECT(st == FS_OK && !empty && batch > 0 && rec::cs.batch == batch, "strided copy sweep %d", i);
    before = rec::launches;
    st = fs_copy(P(p1), W(p4), rows, 0);
    if (rec::launches != before) EXPECT(st == FS_OK && rows > 0, "copy sweep %d", i);
  }
}

int main(int argc, char** argv) {
  const int n = argc > 1 ? std::atoi(argv[1]) : 20000;
  fixed_cases();
  sweep(n);
  std::printf("%d sweep iterations, %d launches recorded, %d failures\n", n, rec::launches, g_failures);
  return g_failures ? 1 : 0;
}
