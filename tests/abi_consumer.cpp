// A plain C++ consumer of the libfusedsub C ABI: device memory from
// hipMalloc, the null stream, no PyTorch and no Python in the process.
//
//   abi_consumer <case> <dir>
//
// reads the raw input arrays of <case> from <dir> (written by the GPU test
// from the seeded generators), runs the entry point on the GPU, and writes
// its outputs back to <dir> for the test to compare with the float64
// oracle.  <dir>/dims.txt holds the shape and scalars of the call.  Cases:
//   pointwise  x, bias, residual (f32)      -> y          fs_pointwise_chain, GELU
//   softmax    x, mask (bf16)               -> y          fs_row_softmax
//   layernorm  x, residual, gamma, beta     -> y, res_out fs_layernorm_residual
//   epilogue   c, bias (bf16), scale (f32)  -> out (f32)  fs_gemm_epilogue_reduce, sigmoid sum
//   program    x, bias, col, residual (bf16) -> y         fs_pointwise_program; the
//              operations come from <dir>/ops.txt, one "code a b" line each
//   softmax_u8 x (bf16), mask (u8)          -> y          fs_row_softmax, byte mask
//   logsumexp  x (bf16)                     -> out (f32)  fs_row_reduce, FS_ROW_LOGSUMEXP
// Exits 0 on success; on any failure prints the status and exits 1.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "fusedsub.h"

namespace {

std::string g_dir;

[[noreturn]] void die(const char* what) {
  std::fprintf(stderr, "abi_consumer: %s\n", what);
  std::exit(1);
}

void hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    std::fprintf(stderr, "abi_consumer: %s: %s\n", what, hipGetErrorString(e));
    std::exit(1);
  }
}

void fs_ok(fs_status s, const char* what) {
  if (s != FS_OK) {
    std::fprintf(stderr, "abi_consumer: %s: %s (%s)\n", what, fs_status_string(s),
                 fs_last_error_message());
    std::exit(1);
  }
}

std::vector<uint8_t> read_file(const char* name, size_t bytes) {
  const std::string path = g_dir + "/" + name;
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) die(("cannot open " + path).c_str());
  std::vector<uint8_t> v(bytes);
  const size_t got = bytes ? std::fread(v.data(), 1, bytes, f) : 0;
  std::fclose(f);
  if (got != bytes) die(("short read of " + path).c_str());
  return v;
}

void write_file(const char* name, const std::vector<uint8_t>& v) {
  const std::string path = g_dir + "/" + name;
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) die(("cannot create " + path).c_str());
  if (std::fwrite(v.data(), 1, v.size(), f) != v.size()) die(("short write of " + path).c_str());
  std::fclose(f);
}

// A device copy of a host array, freed at scope exit.
struct Dev {
  void* p = nullptr;
  size_t bytes = 0;
  explicit Dev(size_t n) : bytes(n) { hip_ok(hipMalloc(&p, n ? n : 16), "hipMalloc"); }
  explicit Dev(const std::vector<uint8_t>& h) : Dev(h.size()) {
    hip_ok(hipMemcpy(p, h.data(), h.size(), hipMemcpyHostToDevice), "hipMemcpy to device");
  }
  std::vector<uint8_t> host() const {
    std::vector<uint8_t> h(bytes);
    hip_ok(hipMemcpy(h.data(), p, bytes, hipMemcpyDeviceToHost), "hipMemcpy to host");
    return h;
  }
  ~Dev() { hipFree(p); }
  Dev(const Dev&) = delete;
  Dev& operator=(const Dev&) = delete;
};

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3)
    die("usage: abi_consumer <pointwise|softmax|layernorm|epilogue|program|softmax_u8|logsumexp>"
        " <dir>");
  const std::string kase = argv[1];
  g_dir = argv[2];
  int64_t rows = 0, cols = 0;
  double p1 = 0, p2 = 0;
  {
    const std::string path = g_dir + "/dims.txt";
    FILE* f = std::fopen(path.c_str(), "r");
    if (!f) die("cannot open dims.txt");
    long long r = 0, c = 0;
    const int n = std::fscanf(f, "%lld %lld %lf %lf", &r, &c, &p1, &p2);
    std::fclose(f);
    if (n != 4 || r < 0 || c < 0) die("bad dims.txt");
    rows = r;
    cols = c;
  }
  const size_t n = size_t(rows) * size_t(cols);
  hipStream_t null_stream = nullptr;
  if (kase == "pointwise") {
    Dev x(read_file("x.bin", n * 4)), b(read_file("bias.bin", size_t(cols) * 4)),
        r(read_file("residual.bin", n * 4)), y(n * 4);
    fs_ok(fs_pointwise_chain(x.p, cols, b.p, r.p, cols, y.p, cols, rows, cols, float(p1),
                             FS_ACT_GELU_ERF, FS_F32, null_stream),
          "fs_pointwise_chain");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("y.bin", y.host());
  } else if (kase == "softmax") {
    Dev x(read_file("x.bin", n * 2)), m(read_file("mask.bin", n * 2)), y(n * 2);
    fs_ok(fs_row_softmax(x.p, cols, m.p, cols, FS_BF16, y.p, cols, rows, cols, float(p1),
                         int64_t(p2), FS_BF16, null_stream),
          "fs_row_softmax");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("y.bin", y.host());
  } else if (kase == "layernorm") {
    Dev x(read_file("x.bin", n * 2)), r(read_file("residual.bin", n * 2)),
        g(read_file("gamma.bin", size_t(cols) * 2)), b(read_file("beta.bin", size_t(cols) * 2)),
        y(n * 2), ro(n * 2);
    fs_ok(fs_layernorm_residual(x.p, cols, r.p, cols, g.p, b.p, y.p, cols, ro.p, cols, rows,
                                cols, float(p1), FS_BF16, null_stream),
          "fs_layernorm_residual");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("y.bin", y.host());
    write_file("residual_out.bin", ro.host());
  } else if (kase == "epilogue") {
    Dev c(read_file("c.bin", n * 2)), b(read_file("bias.bin", size_t(cols) * 2)),
        s(read_file("scale.bin", size_t(cols) * 4)), out(size_t(rows) * 4);
    fs_ok(fs_gemm_epilogue_reduce(c.p, cols, FS_BF16, b.p, FS_BF16,
                                  static_cast<const float*>(s.p), FS_ACT_SIGMOID, FS_REDUCE_SUM,
                                  static_cast<float*>(out.p), rows, cols, null_stream),
          "fs_gemm_epilogue_reduce");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("out.bin", out.host());
  } else if (kase == "program") {
    std::vector<fs_op> ops;
    {
      const std::string path = g_dir + "/ops.txt";
      FILE* f = std::fopen(path.c_str(), "r");
      if (!f) die("cannot open ops.txt");
      int code = 0;
      double a = 0, b = 0;
      while (std::fscanf(f, "%d %lf %lf", &code, &a, &b) == 3)
        ops.push_back(fs_op{code, float(a), float(b)});
      std::fclose(f);
    }
    Dev x(read_file("x.bin", n * 2)), b(read_file("bias.bin", size_t(cols) * 2)),
        c(read_file("col.bin", size_t(cols) * 2)), r(read_file("residual.bin", n * 2)), y(n * 2);
    fs_ok(fs_pointwise_program(x.p, cols, ops.data(), int(ops.size()), b.p, c.p, r.p, cols, y.p,
                               cols, rows, cols, FS_BF16, null_stream),
          "fs_pointwise_program");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("y.bin", y.host());
  } else if (kase == "softmax_u8") {
    Dev x(read_file("x.bin", n * 2)), m(read_file("mask.bin", n)), y(n * 2);
    fs_ok(fs_row_softmax(x.p, cols, m.p, cols, FS_U8, y.p, cols, rows, cols, float(p1),
                         int64_t(p2), FS_BF16, null_stream),
          "fs_row_softmax");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("y.bin", y.host());
  } else if (kase == "logsumexp") {
    Dev x(read_file("x.bin", n * 2)), out(size_t(rows) * 4);
    fs_ok(fs_row_reduce(x.p, cols, FS_BF16, FS_ROW_LOGSUMEXP, static_cast<float*>(out.p), rows,
                        cols, null_stream),
          "fs_row_reduce");
    hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
    write_file("out.bin", out.host());
  } else {
    die("unknown case");
  }
  std::printf("abi_consumer %s: ok (%lld x %lld, ABI version %d)\n", kase.c_str(),
              static_cast<long long>(rows), static_cast<long long>(cols), fs_abi_version());
  return 0;
}
