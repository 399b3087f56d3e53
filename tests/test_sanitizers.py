"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU).  Each builds a small C driver
(tests/sanitize/) against a sanitizer build and runs it in a child process;
sanitizers act on host code only."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr
    return r.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", exe,
                    os.path.join(HERE, "sanitize", "oracle_driver.c"),
                    os.path.join(ROOT, "oracle", "vdo_oracle.c"), "-lm"], check=True)
    assert "all checks passed" in _run(exe)


HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm toolchain")
def test_host_abi_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libvdecode_san.so")
    exe = str(tmp_path / "abi_san")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all"]
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared", "-O1", "-g",
                        *host_san, "-I", os.path.join(ROOT, "include"), "-o", lib,
                        os.path.join(ROOT, "paper_2509_04827_amd", "csrc", "vdecode.hip"),
                        os.path.join(ROOT, "paper_2509_04827_amd", "csrc", "gemm.hip")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    subprocess.run([CLANG, "-O1", "-g", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-o", exe,
                    os.path.join(HERE, "sanitize", "abi_driver.c"), lib,
                    "-Wl,-rpath," + str(tmp_path), "-L/opt/rocm/lib", "-lamdhip64"], check=True)
    assert "all checks passed" in _run(exe)
