"""Sanitizer builds of the host code (no GPU): the CPU oracle and the C-ABI
layer of the library (argument checks, workspace layout, shape queries),
each compiled with AddressSanitizer and UndefinedBehaviorSanitizer and run
over many shapes by a small C driver (tests/asan_oracle_main.c,
tests/asan_abi_main.c).  Device code is not instrumented: the sanitizer
flags reach only the host half of the HIP compile."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = os.path.join(ROOT, "tests")
SAN_ENV = {"ASAN_OPTIONS": "halt_on_error=1:detect_leaks=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def run_clean(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env={**os.environ, **SAN_ENV},
                       timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "Sanitizer" not in out and "runtime error" not in out, out[-4000:]
    return r.stdout


def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-omit-frame-pointer", "-fopenmp", "-I", os.path.join(ROOT, "oracle"),
                    os.path.join(ROOT, "oracle", "oracle.c"),
                    os.path.join(TESTS, "asan_oracle_main.c"), "-lm", "-o", exe], check=True)
    assert "oracle ok" in run_clean(exe)


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    from paper_2403_17607_amd import build
    clangxx = "/opt/rocm/llvm/bin/clang++"
    clang = "/opt/rocm/llvm/bin/clang"
    if not (os.path.exists(clangxx) and shutil.which(build.HIPCC)):
        pytest.skip("ROCm clang not found")
    objs = [os.path.join(build.BUILD, os.path.splitext(s)[0] + ".o") for s in build.SOURCES
            if s != "api.hip"]
    if not all(os.path.exists(o) for o in objs):
        build.build()
    api_o = str(tmp_path / "api_san.o")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in build.FLAGS if f != "-O3"]
    subprocess.run([build.HIPCC, *flags, "-O1", "-g", *san, "-c",
                    os.path.join(build.CSRC, "api.hip"), "-o", api_o], check=True,
                   capture_output=True)
    main_o = str(tmp_path / "abi_main.o")
    subprocess.run([clang, "-std=c11", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(TESTS, "asan_abi_main.c"), "-o", main_o], check=True)
    exe = str(tmp_path / "abi_asan")
    subprocess.run([clangxx, "-fsanitize=address,undefined", main_o, api_o, *objs,
                    "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe],
                   check=True)
    assert "abi ok" in run_clean(exe)
