"""The C-ABI layer (csrc/api.hip: argument validation, overflow guards, alias
checks, path choice) built for the host with AddressSanitizer and
UndefinedBehaviorSanitizer and driven by tests/abi_sanitize_check.cpp: fixed
cases with known statuses, then a deterministic sweep of extreme integers and
odd pointers over every entry point.  The HIP runtime calls and the kernel
launchers are stand-ins, so no GPU is needed and no kernel runs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build_command(out):
    return ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
            "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
            "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include",
            f"-I{ROOT}/paper_2609_30059_amd/csrc",
            "-x", "c++", f"{ROOT}/paper_2609_30059_amd/csrc/api.hip",
            "-x", "none", f"{ROOT}/tests/abi_sanitize_check.cpp", "-o", out]


def test_abi_layer_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if shutil.which("g++") is None or not os.path.isdir(os.path.join(ROCM, "include", "hip")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path / "abi_sanitize_check")
    b = subprocess.run(build_command(exe), capture_output=True, text=True)
    assert b.returncode == 0, b.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, "20000"], capture_output=True, text=True, env=env, timeout=300)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "runtime error" not in report and "AddressSanitizer" not in report, report[-4000:]
    assert "0 failures" in r.stdout
