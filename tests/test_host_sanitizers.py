"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is rebuilt with its host code instrumented (device code as usual)
and the CPU tests of the ABI run against it in a child process with the
sanitizer runtime preloaded: argument validation of every entry point, the
closed-form row counts, and the host position lists against the oracle's
selection in every retention mode.  Any sanitizer report aborts the child."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    r = subprocess.run(["/opt/rocm/lib/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True, check=True)
    path = r.stdout.strip()
    assert os.path.isabs(path) and os.path.exists(path), path
    return path


def test_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2608_23167_amd.build import build_hostsan
    lib = build_hostsan(str(tmp_path))
    env = dict(os.environ)
    env.update(LD_PRELOAD=_asan_runtime(), SSM_HOSTSAN_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "tests._hostsan_plugin",
                        "-m", "not gpu", "tests/test_abi.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
    # the instrumented library really was the one loaded
    maps = subprocess.run(["ldd", lib], capture_output=True, text=True).stdout
    assert "libclang_rt.asan" in maps
