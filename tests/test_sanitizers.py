"""The fp64 oracle and the library's host code (argument validation, plan
bookkeeping, the ternary packing) built with AddressSanitizer and
UndefinedBehaviorSanitizer, running the oracle's pins and the host-side ABI
tests on the CPU in a child process. Any memory error or undefined behaviour
aborts the child (halt_on_error); the parent checks its exit status and output.
The GPU code of the library is not instrumented (the host build only)."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "cd_oracle.c")
CSRC = os.path.join(ROOT, "paper_2505_17701_amd", "csrc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _preload(lib):
    """The sanitizer runtime first, then whatever the environment preloads already."""
    cur = os.environ.get("LD_PRELOAD")
    return lib if not cur else f"{lib}:{cur}"


def _run_child(tests, extra_env):
    env = dict(os.environ)
    env.update(SAN_ENV)
    env.update(extra_env)
    res = subprocess.run([sys.executable, "-m", "pytest", *tests, "-x", "-q", "-m", "not gpu",
                          "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True,
                         text=True, timeout=900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    for marker in ("AddressSanitizer", "runtime error:", "LeakSanitizer"):
        assert marker not in out, out[-4000:]
    return out


def test_oracle_pins_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc missing")
    lib = str(tmp_path / "libcdoracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                    "-Wall", "-Wextra", "-o", lib, ORACLE_SRC, "-lm"], check=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                          check=True).stdout.strip()
    out = _run_child(["tests/test_oracle_pins.py", "tests/test_traffic.py"],
                     {"CD_ORACLE_LIB": lib, "LD_PRELOAD": _preload(asan)})
    assert " passed" in out


def test_host_abi_under_asan_ubsan(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    rts = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not os.path.exists(hipcc) or not rts:
        pytest.skip("hipcc or the clang sanitizer runtime missing")
    lib = str(tmp_path / "libcountdown_san.so")
    # the device code is compiled as usual; only the host code is instrumented
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                    "-shared", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-shared-libsan",
                    "-I", os.path.join(ROOT, "include"), "-o", lib,
                    os.path.join(CSRC, "cd_api.hip"), os.path.join(CSRC, "cd_kernels.hip")],
                   check=True, capture_output=True)
    out = _run_child(["tests/test_abi_host.py"],
                     {"CD_LIBRARY": lib, "LD_PRELOAD": _preload(sorted(rts)[-1])})
    assert " passed" in out
