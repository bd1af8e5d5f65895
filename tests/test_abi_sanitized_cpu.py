"""The C ABI's host layer (csrc/rf_abi.cpp: all argument validation, id-list
copies, overlap arithmetic and the rolling cache's bookkeeping) built with
AddressSanitizer and UndefinedBehaviorSanitizer by g++ (host code only; the
kernel launchers come from the built library and are never reached), driven
through every entry point's rejection paths and host-only successes by
tests/c/abi_errors.c in a fresh process that stops at the first report.
Skipped when g++ or the built library is missing."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_06309_amd")
LIB = os.path.join(PKG, "librhymeflow.so")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    gxx, gcc = shutil.which("g++"), shutil.which("gcc")
    if not gxx or not gcc:
        pytest.skip("no g++/gcc")
    if not os.path.exists(LIB):
        pytest.skip("library not built")
    d = tmp_path_factory.mktemp("asan")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"), "-I", "/opt/rocm/include",
           "-D__HIP_PLATFORM_AMD__"]
    abi_o, main_o, out = str(d / "rf_abi.o"), str(d / "abi_errors.o"), str(d / "abi_errors")
    subprocess.run([gxx, "-std=c++17", *SAN, *inc, "-c", os.path.join(PKG, "csrc", "rf_abi.cpp"), "-o", abi_o],
                   check=True)
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", *SAN, "-I", os.path.join(ROOT, "include"),
                    "-c", os.path.join(ROOT, "tests", "c", "abi_errors.c"), "-o", main_o], check=True)
    # the sanitized host layer first; the kernel launchers it calls come from the library
    subprocess.run([gxx, *SAN, main_o, abi_o, "-L", PKG, "-lrhymeflow", f"-Wl,-rpath,{PKG}",
                    "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-lm", "-o", out], check=True)
    return out


def test_abi_error_paths_are_clean_under_asan_and_ubsan(exe):
    env = dict(os.environ)
    # leaks of the HIP runtime's own start-up are not this layer's
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    last = r.stdout.strip().splitlines()[-1]
    assert last.startswith("ok ") and int(last.split()[1]) >= 100, r.stdout[-2000:]
