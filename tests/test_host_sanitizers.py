"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU needed).

The planner (``planner.cpp``) and the C-ABI layer (``abi.cpp``) parse caller
descriptors with 32/64-bit index arithmetic.  Here they are built with g++
``-fsanitize=address,undefined`` (kernel launchers replaced by stand-ins that
report hipErrorNotSupported), and

* a seeded random-descriptor fuzzer drives ``build_host_plan`` with valid and
  rule-breaking batches, checking the invariants of every accepted plan;
* the host-side test files (plans, items, launch orders, error paths, the
  asynchronous planner) run against the sanitizer build through
  ``MSTAR_ATTN_LIB`` with the ASan runtime preloaded into Python.

Any sanitizer report makes the run fail.  A planted heap overflow built with
the same flags checks that the sanitizer is really active."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_12688_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
FLAGS = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
         "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
       "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}


def _gxx():
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    asan = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("libasan not available")
    return gxx, asan


def _build(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr


@pytest.fixture(scope="module")
def built(tmp_path_factory):
    gxx, asan = _gxx()
    d = tmp_path_factory.mktemp("sanitize")
    lib = str(d / "libmstar_attn_sanitized.so")
    fuzz = str(d / "planner_fuzz")
    _build([gxx, *FLAGS, "-fPIC", "-shared", os.path.join(CSRC, "abi.cpp"), os.path.join(CSRC, "planner.cpp"),
            os.path.join(SAN, "kernels_stub.cpp"), "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
            "-o", lib])
    _build([gxx, *FLAGS, os.path.join(CSRC, "planner.cpp"), os.path.join(SAN, "planner_fuzz.cpp"), "-o", fuzz])
    return {"gxx": gxx, "asan": asan, "lib": lib, "fuzz": fuzz, "dir": str(d)}


def test_sanitizer_is_active(built):
    src = os.path.join(built["dir"], "overflow.cpp")
    with open(src, "w") as f:
        f.write("#include <vector>\nint main(int c, char**) { std::vector<int> v(4); return v.data()[4 + c]; }\n")
    exe = os.path.join(built["dir"], "overflow")
    _build([built["gxx"], *FLAGS, src, "-o", exe])
    res = subprocess.run([exe], capture_output=True, text=True, env={**os.environ, **ENV})
    assert res.returncode != 0 and "AddressSanitizer" in res.stderr


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_planner_fuzz(built, seed):
    res = subprocess.run([built["fuzz"], str(seed), "3000"], capture_output=True, text=True,
                         env={**os.environ, **ENV}, timeout=600)
    print(res.stdout + res.stderr[-4000:])
    assert res.returncode == 0
    assert "Sanitizer" not in res.stderr and "runtime error" not in res.stderr
    assert " 0 failures" in res.stdout


def test_host_tests_against_the_sanitized_library(built):
    env = {**os.environ, **ENV, "MSTAR_ATTN_LIB": built["lib"], "LD_PRELOAD": built["asan"]}
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                          os.path.join(ROOT, "tests", "test_abi_host.py"),
                          os.path.join(ROOT, "tests", "test_async_planner.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    print(res.stdout[-3000:] + res.stderr[-4000:])
    assert res.returncode == 0
    assert "Sanitizer" not in res.stderr and "runtime error" not in res.stderr
    assert " passed" in res.stdout and "failed" not in res.stdout
