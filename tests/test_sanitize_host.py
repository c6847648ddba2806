"""Host sanitizer runs (CPU only, no GPU needed), with AddressSanitizer,
UndefinedBehaviorSanitizer and leak checking:
- the oracle runs small cases through every one of its entry points, with
  checks of properties the method fixes exactly (tests/sanitize/oracle_checks.c);
- the library's C ABI, its host code sanitized, answers every query and
  rejects invalid calls on the host (tests/sanitize/abi_checks.c); nothing is
  launched."""
import os
import shutil
import subprocess

import pytest

from paper_1907_01729_amd import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "sanitize", "oracle_checks.c")
ORACLE = os.path.join(ROOT, "oracle", "sinkhorn_oracle.c")


def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not installed")
    exe = str(tmp_path / "oracle_checks")
    build = subprocess.run([gcc, "-std=c11", "-O1", "-g", "-fopenmp", "-fno-omit-frame-pointer",
                            "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", exe, DRIVER, ORACLE,
                            "-lm"], capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert run.stdout.strip() == "ok"


def test_abi_host_paths_under_address_and_ub_sanitizers(tmp_path):
    """Builds the library with sanitized host code (about a minute) and runs the
    ABI driver against it."""
    lib = libbuild.build_host_sanitized()
    clang = os.path.join(os.path.dirname(os.path.realpath(libbuild.hipcc())), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    exe = str(tmp_path / "abi_checks")
    libdir = os.path.dirname(lib)
    build = subprocess.run([clang, "-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                            "-fno-sanitize-recover=all", "-shared-libsan", "-I", os.path.join(ROOT, "include"),
                            "-o", exe, os.path.join(ROOT, "tests", "sanitize", "abi_checks.c"), lib,
                            "-Wl,-rpath," + libdir], capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    rt = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1",
               LD_LIBRARY_PATH=os.pathsep.join(filter(None, [os.path.dirname(rt), libdir,
                                                             os.environ.get("LD_LIBRARY_PATH", "")])))
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert run.stdout.strip() == "ok"
