"""Host-side tests of the C ABI: the libraries load, export every symbol
the headers declare, and reject bad arguments with the documented status
before any HIP call (so they run without a GPU).  No kernel is launched."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_30059_amd import _native as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NULL = None
A = 0x10000000          # fake, 16-byte aligned device addresses (never dereferenced:
B = 0x20000000          # every call below fails validation first)
C = 0x30000000


def declared(header, prefix):
    txt = open(os.path.join(ROOT, "include", header)).read()
    return sorted(set(re.findall(r"\b(" + prefix + r"[a-z0-9_]+)\s*\(", txt)))


def test_libraries_load_and_export_every_declared_symbol():
    lib = N.fusedsub()
    for name in declared("fusedsub.h", "fs_"):
        assert hasattr(lib, name), name
    g = N.fsgemm()
    for name in declared("fsgemm.h", "fsg_"):
        assert hasattr(g, name), name
    assert set(declared("fusedsub.h", "fs_")) == set(N.FUSEDSUB_SYMBOLS)
    assert set(declared("fsgemm.h", "fsg_")) == set(N.FSGEMM_SYMBOLS)


def test_only_declared_symbols_are_exported():
    for lib, pre in ((N.LIB_FUSEDSUB, "fs"), (N.LIB_FSGEMM, "fsg")):
        out = subprocess.run(["nm", "-D", "--defined-only", lib], capture_output=True,
                             text=True).stdout
        syms = {l.split()[-1] for l in out.splitlines() if " T " in l}
        ours = {s for s in syms if s.startswith(pre + "_")}
        assert ours == set(declared("fusedsub.h" if pre == "fs" else "fsgemm.h", pre + "_"))


def test_single_hip_runtime_in_process():
    N.fusedsub()
    N.fsgemm()
    libs = N.hip_runtimes_mapped()
    real = {os.path.realpath(p) for p in libs}
    assert len(real) <= 1, libs


def test_version_and_status_strings():
    assert N.fs_abi_version() == N.FS_ABI_VERSION
    for code, name in N.STATUS_NAMES.items():
        assert N.fs_status_string(code).startswith(name)
    assert "UNKNOWN" in N.fs_status_string(99)
    assert "UNKNOWN" in N.fs_status_string(-1)


# ---- pointwise ---------------------------------------------------------------
def pw(**kw):
    a = dict(x=A, ld_x=64, bias=NULL, residual=NULL, ld_r=64, y=B, ld_y=64, rows=4, cols=64,
             scale=1.0, act=0, dtype=0, stream=None)
    a.update(kw)
    return N.fs_pointwise_chain(**a)


def test_pointwise_validation():
    assert pw(x=NULL) == 1
    assert pw(y=NULL) == 1
    assert pw(rows=-1) == 2
    assert pw(cols=-5) == 2
    assert pw(ld_x=63) == 3
    assert pw(ld_y=10) == 3
    assert pw(residual=C, ld_r=3) == 3
    assert pw(dtype=7) == 4
    assert pw(act=9) == 6
    assert pw(scale=float("nan")) == 6
    assert pw(scale=float("inf")) == 6
    assert pw(x=A + 2) == 6                      # not aligned to 4 bytes for fp32
    assert pw(y=A + 4 * 64) == 5                 # y starts inside x (partial overlap)
    assert pw(y=A + 4, ld_y=64) == 5
    assert pw(bias=B + 16) == 5                  # bias inside y
    assert pw(residual=B + 64, ld_r=64) == 5     # residual partially overlaps y
    assert "overlap" in N.fs_last_error_message()


def test_pointwise_empty_problem_is_ok_without_pointers():
    assert pw(rows=0, x=NULL, y=NULL) == 0
    assert pw(cols=0, ld_x=0, ld_y=0, x=NULL, y=NULL) == 0
    assert N.fs_last_error_message() == ""


# ---- pointwise program ---------------------------------------------------------
def ops_array(*ops):
    arr = (N.FsOp * max(len(ops), 1))()
    for k, (code, a, b) in enumerate(ops):
        arr[k] = N.FsOp(code, a, b)
    return arr


def pp(**kw):
    a = dict(x=A, ld_x=64, ops=ops_array((2, 0.0, 0.0), (0, 0.5, 0.0), (6, -1.0, 1.0), (7, 0, 0)),
             n_ops=4, bias=C, col=NULL, residual=NULL, ld_r=64, y=B, ld_y=64, rows=4, cols=64,
             dtype=0, stream=None)
    a.update(kw)
    return N.fs_pointwise_program(**a)


def test_pointwise_program_validation():
    assert pp(dtype=2) == 4                                  # bytes are a mask dtype only
    assert pp(n_ops=N.FS_PROGRAM_MAX_OPS + 1) == 6
    assert pp(n_ops=-1) == 6
    assert pp(ops=None) == 1
    assert pp(ops=ops_array((13, 0, 0)), n_ops=1) == 6      # unknown code
    assert pp(ops=ops_array((0, float("nan"), 0)), n_ops=1) == 6
    assert pp(ops=ops_array((12, float("inf"), 0)), n_ops=1) == 6
    assert pp(ops=ops_array((6, 1.0, -1.0)), n_ops=1) == 6  # clamp bounds out of order
    assert pp(ops=ops_array((6, float("nan"), 1.0)), n_ops=1) == 6
    assert pp(bias=NULL) == 1                                # the program adds a bias
    assert pp(ops=ops_array((5, 0, 0)), n_ops=1) == 1       # it multiplies by a NULL residual
    assert pp(ops=ops_array((3, 0, 0)), n_ops=1, bias=NULL) == 1   # and a NULL column vector
    assert pp(ld_y=63) == 3
    assert pp(x=A + 2) == 6
    assert pp(bias=B + 64) == 5                              # bias inside y
    assert pp(y=A + 4) == 5                                  # y partly over x
    # checks that end before any HIP call: an empty problem, open clamp bounds
    assert pp(rows=0, x=NULL, y=NULL) == 0
    assert pp(ops=ops_array((6, float("-inf"), float("inf"))), n_ops=1, rows=0) == 0
    assert pp(ops=None, n_ops=0, rows=0) == 0
    # operations the program does not use leave their operands unread
    assert pp(ops=ops_array((7, 0, 0)), n_ops=1, bias=NULL, rows=0) == 0


def test_program_operation_table_matches_the_header():
    txt = open(os.path.join(ROOT, "include", "fusedsub.h")).read()
    codes = dict(re.findall(r"FS_OP_([A-Z_]+) = (\d+)", txt))
    assert {k.lower(): int(v) for k, v in codes.items()} == \
        {name: code for name, (code, _) in N.PROGRAM_OPS.items()}
    m = re.search(r"#define FS_PROGRAM_MAX_OPS (\d+)", txt)
    assert int(m.group(1)) == N.FS_PROGRAM_MAX_OPS


# ---- softmax -----------------------------------------------------------------
def sm(**kw):
    a = dict(x=A, ld_x=128, mask=NULL, ld_mask=128, mask_dtype=1, y=B, ld_y=128, rows=4,
             cols=128, scale=0.125, causal_q_len=0, dtype=1, stream=None)
    a.update(kw)
    return N.fs_row_softmax(**a)


def test_softmax_validation():
    assert sm(x=NULL) == 1
    assert sm(cols=N.FS_SOFTMAX_MAX_COLS + 1, ld_x=1 << 25, ld_y=1 << 25) == 2
    assert sm(rows=-1) == 2
    assert sm(ld_x=127) == 3
    assert sm(mask=C, ld_mask=100) == 3
    assert sm(dtype=3) == 4
    assert sm(mask=C, mask_dtype=5) == 4
    assert sm(causal_q_len=-1) == 6
    assert sm(scale=float("nan")) == 6
    assert sm(x=A + 1) == 6
    assert sm(mask=B + 256) == 5                 # mask overlaps y
    assert sm(y=A + 2) == 5                      # partial overlap with x
    assert sm(rows=0, x=NULL, y=NULL) == 0


# ---- layernorm ---------------------------------------------------------------
def ln(**kw):
    a = dict(x=A, ld_x=256, residual=NULL, ld_r=256, gamma=NULL, beta=NULL, y=B, ld_y=256,
             residual_out=NULL, ld_ro=256, rows=8, cols=256, eps=1e-5, dtype=1, stream=None)
    a.update(kw)
    return N.fs_layernorm_residual(**a)


def test_layernorm_validation():
    assert ln(y=NULL) == 1
    assert ln(cols=N.FS_LAYERNORM_MAX_COLS + 8, ld_x=1 << 25, ld_y=1 << 25) == 2
    assert ln(ld_y=255) == 3
    assert ln(residual=C, ld_r=1) == 3
    assert ln(residual_out=C, ld_ro=1) == 3
    assert ln(dtype=2) == 4
    assert ln(eps=-1.0) == 6
    assert ln(eps=float("inf")) == 6
    assert ln(gamma=A + 1) == 6
    assert ln(residual_out=B + 512) == 5          # residual_out overlaps y
    assert ln(gamma=B) == 5                       # gamma inside y
    assert ln(residual=C, residual_out=C + 2) == 5


def rms(**kw):
    a = dict(x=A, ld_x=256, residual=NULL, ld_r=256, gamma=NULL, y=B, ld_y=256,
             residual_out=NULL, ld_ro=256, rows=8, cols=256, eps=1e-6, dtype=1, stream=None)
    a.update(kw)
    return N.fs_rmsnorm_residual(**a)


def test_rmsnorm_validation():
    assert rms(x=NULL) == 1
    assert rms(cols=N.FS_LAYERNORM_MAX_COLS + 8, ld_x=1 << 25, ld_y=1 << 25) == 2
    assert rms(ld_x=7) == 3
    assert rms(dtype=5) == 4
    assert rms(eps=float("nan")) == 6
    assert rms(gamma=B + 64) == 5
    assert rms(residual=C, residual_out=B + 2) == 5
    assert rms(rows=0, x=NULL, y=NULL) == 0


def test_row_reduce_and_argmax_validation():
    red = lambda **kw: N.fs_row_reduce(**{**dict(x=A, ld_x=64, dtype=0, op=0, out=B, rows=4,  # noqa: E731
                                              cols=64, stream=None), **kw})
    arg = lambda **kw: N.fs_row_argmax(**{**dict(x=A, ld_x=64, dtype=0, out=B, rows=4,  # noqa: E731
                                              cols=64, stream=None), **kw})
    assert red(out=NULL) == 1
    assert red(rows=-1) == 2
    assert red(ld_x=3) == 3
    assert red(dtype=9) == 4
    assert red(op=7) == 6
    assert red(out=A + 8) == 5              # out inside x
    assert red(out=B + 2) == 6              # misaligned float*
    assert red(cols=0, op=1) == 2           # mean of nothing
    assert red(cols=0, op=2) == 2           # max of nothing
    assert red(cols=0, op=3) == 2           # log-sum-exp of nothing
    assert red(op=4) == 6                   # one past the last reduction
    assert red(rows=0, x=NULL, out=NULL) == 0
    assert arg(out=NULL) == 1
    assert arg(cols=0, ld_x=0) == 2
    assert arg(out=B + 4) == 6              # misaligned int64*
    assert arg(out=A) == 5
    assert arg(rows=0, out=NULL) == 0


# ---- epilogue ----------------------------------------------------------------
def ep(**kw):
    a = dict(c=A, ld_c=8192, c_dtype=1, bias=NULL, bias_dtype=1, col_scale=NULL, act=2,
             reduce=0, row_out=B, rows=16, cols=8192, stream=None)
    a.update(kw)
    return N.fs_gemm_epilogue_reduce(**a)


def test_epilogue_validation():
    assert ep(row_out=NULL) == 1
    assert ep(c=NULL) == 1
    assert ep(rows=-2) == 2
    assert ep(ld_c=100) == 3
    assert ep(c_dtype=4) == 4
    assert ep(bias=C, bias_dtype=9) == 4
    assert ep(act=11) == 6
    assert ep(reduce=4) == 6                      # one past log-sum-exp
    assert ep(reduce=-1) == 6
    assert ep(row_out=B + 2) == 6
    assert ep(row_out=A + 64) == 5                # row_out inside C
    assert ep(col_scale=B) == 5
    assert ep(rows=0, c=NULL, row_out=NULL) == 0
    assert ep(cols=0, reduce=1) == 2              # mean over zero columns
    assert ep(cols=0, reduce=2) == 2              # max over zero columns
    assert ep(cols=0, reduce=3) == 2              # log-sum-exp over zero columns


def test_copy_validation():
    assert N.fs_copy(A, B, -1, None) == 2
    assert N.fs_copy(NULL, B, 16, None) == 1
    assert N.fs_copy(A, A + 8, 16, None) == 5
    assert N.fs_copy(A, B, 0, None) == 0


# ---- gemm wrapper ------------------------------------------------------------
def gm(**kw):
    a = dict(a=A, lda=64, stride_a=0, b=B, ldb=32, stride_b=0, trans_b=0, c=C, ldc=32,
             stride_c=0, m=16, n=32, k=64, batch=1, alpha=1.0, bias=NULL, workspace=NULL,
             workspace_bytes=0, stream=None)
    a.update(kw)
    return N.fsg_gemm_bf16(**a)


def test_gemm_validation():
    assert gm(a=NULL) == 1
    assert gm(workspace_bytes=1024) == 1
    assert gm(m=-1) == 2
    assert gm(batch=0) == 2
    assert gm(lda=63) == 3
    assert gm(ldb=31) == 3
    assert gm(trans_b=1, ldb=63) == 3
    assert gm(ldc=31) == 3
    assert gm(trans_b=2) == 4
    assert gm(alpha=float("nan")) == 4
    assert gm(m=0, a=NULL, b=NULL, c=NULL) == 0
    assert "lda" in N.fsg_last_error_message() or N.fsg_last_error_message() == ""


def test_header_compiles_as_c():
    src = '#include "fusedsub.h"\n#include "fsgemm.h"\nint main(void){return fs_abi_version()!=FS_ABI_VERSION;}\n'
    p = "/tmp/_fs_hdr_test.c"
    with open(p, "w") as f:
        f.write(src)
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        f"-I{ROOT}/include", "-I/opt/rocm/include", "-c", p, "-o", "/tmp/_fs_hdr_test.o"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_copy_strided_validation():
    cs = lambda **kw: N.fs_copy_strided(**{**dict(src=A, ld_src=192, stride_src=64, dst=B,  # noqa: E731
                                             ld_dst=64, stride_dst=64 * 100, rows=100, cols=64,
                                             batch=3, dtype=1, stream=None), **kw})
    assert cs(src=NULL) == 1
    assert cs(rows=-1) == 2
    assert cs(batch=-2) == 2
    assert cs(batch=1 << 20, cols=1 << 11, ld_src=1 << 11, ld_dst=1 << 11) == 2   # batch*cols >= 2^30
    assert cs(ld_src=63) == 3
    assert cs(ld_dst=10) == 3
    assert cs(stride_src=-1) == 3
    assert cs(stride_dst=64) == 3          # destination batches overlap
    assert cs(dtype=5) == 4
    assert cs(dst=B + 1) == 6              # misaligned bf16 pointer
    assert cs(dst=A + 128) == 5            # spans overlap
    assert cs(rows=0, src=NULL, dst=NULL) == 0
    assert cs(batch=0, src=NULL, dst=NULL) == 0
    # interleaved destination (a head merge) is accepted by validation:
    # batches 64 apart inside rows of 192
    assert cs(ld_src=64, stride_src=6400, ld_dst=192, stride_dst=64, src=NULL) == 1


def test_gemm_ex_validation():
    ge = lambda **kw: N.fsg_gemm_bf16_ex(**{**dict(a=A, lda=64, stride_a=0, b=B, ldb=32,  # noqa: E731
                                              stride_b=0, trans_b=0, c=C, ldc=32, stride_c=0,
                                              m=16, n=32, k=64, batch=1, alpha=1.0,
                                              alpha_col=NULL, bias=NULL, bias_f32=0, act=0,
                                              c_in=NULL, ld_cin=32, stride_cin=0, beta=0.0,
                                              workspace=NULL, workspace_bytes=0,
                                              stream=None), **kw})
    assert ge(act=7) == 4
    assert ge(act=3) == 4                           # no sigmoid epilogue is offered
    assert ge(bias_f32=2) == 4
    assert ge(alpha=2.0, alpha_col=A + 4096) == 4     # a vector replaces the scalar
    assert ge(beta=float("nan")) == 4
    assert ge(beta=1.0) == 1                          # beta != 0 needs c_in
    assert ge(beta=1.0, c_in=A + 8192, ld_cin=31) == 3
    assert ge(m=-1) == 2
    assert ge(m=0, a=NULL, b=NULL, c=NULL) == 0


def test_causal_softmax_trimmed_validation():
    ct = lambda **kw: N.fs_causal_softmax_trimmed(**{**dict(x=A, ld_x=512, y=B, ld_y=512, rows=64,  # noqa: E731
                                                      cols=512, scale=0.125, causal_q_len=512,
                                                      block=128, dtype=1, stream=None), **kw})
    assert ct(x=NULL) == 1
    assert ct(block=96) == 6                 # not a power of two
    assert ct(block=0) == 6
    assert ct(causal_q_len=0) == 6           # the trimming needs a causal rule
    assert ct(scale=float("inf")) == 6
    assert ct(ld_y=100) == 3
    assert ct(dtype=9) == 4
    assert ct(y=A + 2) == 5
    assert ct(rows=0, x=NULL, y=NULL) == 0


def test_plain_cpp_consumer_is_built_against_the_in_tree_library():
    """tests/abi_consumer.cpp (run on the GPU by test_gpu_abi_consumer.py)
    links the in-tree libfusedsub.so and refuses a bad command line before
    any HIP call."""
    from paper_2609_30059_amd.build import ABI_CONSUMER
    assert os.access(ABI_CONSUMER, os.X_OK), "run python -m paper_2609_30059_amd.build"
    deps = subprocess.run(["ldd", ABI_CONSUMER], capture_output=True, text=True).stdout
    line = next(l for l in deps.splitlines() if "libfusedsub.so" in l)
    assert os.path.realpath(line.split("=>")[1].split()[0]) == os.path.realpath(N.LIB_FUSEDSUB)
    r = subprocess.run([ABI_CONSUMER], capture_output=True, text=True, timeout=60)
    assert r.returncode == 1 and "usage" in r.stderr
