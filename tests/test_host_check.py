"""The C ABI's validation and state machine on the CPU under AddressSanitizer and
UndefinedBehaviorSanitizer (sbd_host_check): sbd_api.cpp built with g++ against host-only
stand-ins for the HIP runtime and the kernel launchers, driven through every forced error
(paper_2509_04185_amd/csrc/host_check/host_check.cpp).  No GPU is needed."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2509_04185_amd", "csrc")
FLAGS = ["-std=c++17", "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def build(out, sources):
    cmd = ["g++"] + FLAGS + ["-I", os.path.join(CSRC, "host_check"), "-I", os.path.join(ROOT, "include"),
                             "-I", CSRC] + sources + ["-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)


def run(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    return subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)


def test_host_check_under_sanitizers(tmp_path):
    exe = str(tmp_path / "sbd_host_check")
    build(exe, [os.path.join(CSRC, "sbd_api.cpp"), os.path.join(CSRC, "host_check", "hip_stub.cpp"),
                os.path.join(CSRC, "host_check", "host_check.cpp")])
    p = run(exe)
    assert p.returncode == 0, p.stdout + p.stderr
    assert "host checks passed" in p.stdout and "FAILED" not in p.stdout + p.stderr
    assert "ERROR: AddressSanitizer" not in p.stderr and "runtime error" not in p.stderr


def test_sanitizer_build_catches_a_planted_overflow(tmp_path):
    """The same flags on a planted heap overflow: the run must fail with a sanitizer's report
    (UBSan's object-size check or ASan, whichever sees it first)."""
    src = tmp_path / "overflow.cpp"
    src.write_text("#include <cstdlib>\nint main(int c, char**) { int* p = (int*)std::malloc(8 * sizeof(int));"
                   " p[8 + c - 1] = 1; int r = p[0]; std::free(p); return r; }\n")
    exe = str(tmp_path / "overflow")
    build(exe, [str(src)])
    p = run(exe)
    assert p.returncode != 0 and ("heap-buffer-overflow" in p.stderr or "runtime error" in p.stderr)
