"""The oracle and the library's host-side code built with AddressSanitizer and
UndefinedBehaviorSanitizer, and the CPU tests that exercise them rerun in child
processes against those builds: the oracle's pins (every oracle function on
hand-worked, brute-force and edge-case inputs) and the C ABI's host checks
(argument validation and sizing; no kernel runs)."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_OPTIONS = "detect_leaks=0:abort_on_error=1:allocator_may_return_null=1"


def _run(test_file, env_extra, preload):
    env = dict(os.environ, ASAN_OPTIONS=ASAN_OPTIONS, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               LD_PRELOAD=preload, PYTHONDONTWRITEBYTECODE="1", **env_extra)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", test_file)], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    return out


def test_oracle_pins_under_asan_ubsan(tmp_path):
    from oracle import build
    lib = build.build(sanitize=True, out=str(tmp_path / "libsg_oracle_san.so"))
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    out = _run("test_oracle_pins.py", {"SG_ORACLE_LIB": lib}, asan)
    assert "passed" in out


def test_library_host_checks_under_asan_ubsan(tmp_path):
    from paper_2607_28150_amd import build
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        pytest.skip("the clang ASan runtime is not installed")
    lib = build.build_host_sanitized(str(tmp_path / "libsmartgen_san.so"))
    out = _run("test_abi.py", {"SG_LIB_PATH": lib}, rt[-1])
    assert "passed" in out
