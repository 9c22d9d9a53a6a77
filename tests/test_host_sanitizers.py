"""The host validation layer of libavtp.so under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only): tests/test_abi.py is run against a
build whose avtp_api.cpp is instrumented, with the ASan runtime preloaded
into that child process; any sanitizer report fails the test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"


def _asan_runtime():
    if not os.path.exists(CLANG):
        return None
    r = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_abi_validation_is_clean_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None or shutil.which("/opt/rocm/bin/hipcc") is None:
        pytest.skip("clang ASan runtime or hipcc not available")
    from paper_2608_26806_amd import build as B
    lib = B.build_host_sanitized(str(tmp_path / "libavtp_san.so"))
    env = dict(os.environ)
    # the ASan runtime must come first; anything the environment already
    # preloads stays loaded after it
    pre = env.get("LD_PRELOAD", "")
    env.update(LD_PRELOAD=rt + (":" + pre if pre else ""), AVTP_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-s", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
