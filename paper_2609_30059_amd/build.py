"""Build the native libraries in-tree for gfx950.

    python -m paper_2609_30059_amd.build

produces, next to this file,
  * libfusedsub.so -- the fused sub-kernels behind the C ABI of include/fusedsub.h
  * libfsgemm.so   -- the hipBLASLt GEMM wrapper of include/fsgemm.h
  * issue_rate     -- the issue-rate calibration program of tiers.py
  * libclockprobe.so -- the engine-clock probe of bench.py's clock-transient mode
  * libaccessfloor.so -- the access-shape floor kernels of bench.py's access-floors mode
  * abi_consumer   -- tests/abi_consumer.cpp, a plain C++ program that calls
                      libfusedsub.so through include/fusedsub.h (GPU test of the ABI)

Every HIP translation unit is compiled with the packed-FP32 target feature
switched off (ordinary fp32 code only).  Objects go to ``_build/`` (ignored
by git); the shared libraries are written atomically.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

FUSEDSUB_SOURCES = ["api.hip", "pointwise.hip", "program.hip", "softmax.hip", "layernorm.hip",
                    "epilogue.hip", "epilogue_maxlse.hip", "reduce.hip", "copy.hip"]
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]

LIB_FUSEDSUB = os.path.join(HERE, "libfusedsub.so")
LIB_FSGEMM = os.path.join(HERE, "libfsgemm.so")
ISSUE_RATE = os.path.join(HERE, "issue_rate")     # calibration program of tiers.py
LIB_CLOCK_PROBE = os.path.join(HERE, "libclockprobe.so")   # bench.py --clock-transient
LIB_ACCESS_FLOOR = os.path.join(HERE, "libaccessfloor.so")   # bench.py --access-floors
ABI_CONSUMER = os.path.join(HERE, "abi_consumer")   # tests/test_gpu_abi_consumer.py


def _hipcc() -> str:
    p = os.path.join(ROCM, "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def _compile(src, verbose, build_dir=BUILD, defines=()):
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    _run([_hipcc(), *HIP_FLAGS, *defines, f"-I{INCLUDE}", f"-I{CSRC}", "-c",
          os.path.join(CSRC, src), "-o", obj], verbose)
    return obj


def _link(objs, out, extra, verbose):
    tmp = out + ".tmp"
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp,
          f"-Wl,-rpath,{ROCM}/lib", *extra], verbose)
    os.replace(tmp, out)


def build(verbose: bool = False, jobs: int = 8) -> None:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), FUSEDSUB_SOURCES))
        gemm_obj = os.path.join(BUILD, "gemm_hipblaslt.o")
        fut = ex.submit(_run, ["g++", "-O2", "-std=c++17", "-fPIC", "-fvisibility=hidden",
                               "-D__HIP_PLATFORM_AMD__", f"-I{INCLUDE}", f"-I{ROCM}/include",
                               "-c", os.path.join(CSRC, "gemm_hipblaslt.cpp"), "-o", gemm_obj],
                        verbose)
        probe = ex.submit(_run, [_hipcc(), *HIP_FLAGS, os.path.join(CSRC, "issue_rate.hip"),
                                 "-o", ISSUE_RATE + ".tmp"], verbose)
        clock = ex.submit(_run, [_hipcc(), *HIP_FLAGS, "-shared",
                                 os.path.join(CSRC, "clock_probe.hip"), "-o",
                                 LIB_CLOCK_PROBE + ".tmp"], verbose)
        floor = ex.submit(_run, [_hipcc(), *HIP_FLAGS, "-shared",
                                 os.path.join(CSRC, "access_floor.hip"), "-o",
                                 LIB_ACCESS_FLOOR + ".tmp"], verbose)
        fut.result()
        probe.result()
        clock.result()
        floor.result()
    os.replace(ISSUE_RATE + ".tmp", ISSUE_RATE)
    os.replace(LIB_CLOCK_PROBE + ".tmp", LIB_CLOCK_PROBE)
    os.replace(LIB_ACCESS_FLOOR + ".tmp", LIB_ACCESS_FLOOR)
    _link(objs, LIB_FUSEDSUB, [], verbose)
    _run(["g++", "-shared", "-fPIC", gemm_obj, "-o", LIB_FSGEMM + ".tmp", f"-L{ROCM}/lib",
          f"-Wl,-rpath,{ROCM}/lib", "-lhipblaslt", "-lamdhip64"], verbose)
    os.replace(LIB_FSGEMM + ".tmp", LIB_FSGEMM)
    # a host-only C++ caller of the ABI, linked against the library just built
    # (found next to the program at run time)
    _run(["g++", "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__", f"-I{INCLUDE}",
          f"-I{ROCM}/include", os.path.join(ROOT, "tests", "abi_consumer.cpp"),
          "-o", ABI_CONSUMER + ".tmp", f"-L{HERE}", "-lfusedsub", f"-L{ROCM}/lib",
          "-lamdhip64", "-Wl,-rpath,$ORIGIN", f"-Wl,-rpath,{ROCM}/lib"], verbose)
    os.replace(ABI_CONSUMER + ".tmp", ABI_CONSUMER)


def build_variant(out_dir: str, defines=(), verbose: bool = False, jobs: int = 8) -> str:
    """Build libfusedsub.so into ``out_dir`` with extra ``-D`` build-time
    tuning parameters (see the FS_* macros in csrc/); returns its path."""
    os.makedirs(out_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, out_dir, defines), FUSEDSUB_SOURCES))
    out = os.path.join(out_dir, "libfusedsub.so")
    _link(objs, out, [], verbose)
    return out


def clean() -> None:
    shutil.rmtree(BUILD, ignore_errors=True)
    for p in (LIB_FUSEDSUB, LIB_FSGEMM, ISSUE_RATE, LIB_CLOCK_PROBE, LIB_ACCESS_FLOOR,
              ABI_CONSUMER):
        if os.path.exists(p):
            os.remove(p)


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print("built", LIB_FUSEDSUB, LIB_FSGEMM)
