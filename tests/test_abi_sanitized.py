"""The host side of the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

librlsim.so's host code (argument checks, configuration validation, message
strings, the kernel-selection logic) is rebuilt with -fsanitize=address,undefined
on the host pass only (the device code is compiled as usual), and a C program
(tests/sanitize/abi_host_checks.c, built with the same sanitizers) drives every
call that fails or succeeds before any device work.  A memory error or an
undefined operation in that code aborts the program with a sanitizer report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")

pytestmark = pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="needs hipcc and clang")


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    import importlib.util
    spec = importlib.util.spec_from_file_location("rlsim_build", os.path.join(ROOT, "paper_2207_07736_amd", "build.py"))
    bld = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bld)
    lib = tmp_path / "librlsim.so"
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-Xarch_host", "-g"]
    flags = [f for f in bld.FLAGS if f != "-O3"] + ["-O1"]
    subprocess.run([HIPCC, *flags, *san, "-I", bld.INCLUDE, "-o", str(lib), bld.SRC], check=True,
                   capture_output=True, text=True)
    nm = subprocess.run(["nm", "-D", str(lib)], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in nm and "__ubsan_handle" in nm          # the host code is instrumented
    exe = tmp_path / "abi_host_checks"
    subprocess.run([CLANG, "-std=c11", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "sanitize", "abi_host_checks.c"),
                    "-L", str(tmp_path), "-lrlsim", f"-Wl,-rpath,{tmp_path}", "-L", os.path.join(ROCM, "lib"),
                    "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-lm", "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "abi host checks: OK" in res.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out
    shutil.rmtree(tmp_path, ignore_errors=True)
