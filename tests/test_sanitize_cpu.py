"""The library's host-side logic under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: tests/sanitize/host_checks.cpp includes
the host source of libssd and exercises configuration validation, argument
checks of every entry point, GEMM launch plans and their workspace sizes, the
image pass plans (against the printed pass-count formula) and the session
workspace sizing.  Only host code is instrumented (-Xarch_host); no GPU is
touched.  Any sanitizer report or failed check fails the test."""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_20543_amd", "csrc")
SOURCES = [os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp")] + [
    os.path.join(CSRC, f + ".hip") for f in ("kernels_gemm", "kernels_attn", "kernels_misc", "kernels_fwd")]
FLAGS = ["-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-Xarch_host", "-fno-sanitize-recover=undefined"]


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not available")
def test_host_logic_under_sanitizers(tmp_path):
    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        r = subprocess.run(["hipcc", *FLAGS, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-4000:]
        return obj

    with cf.ThreadPoolExecutor(max_workers=5) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    exe = str(tmp_path / "host_checks")
    link = ["hipcc", "--offload-arch=gfx950", "-fsanitize=address", "-fsanitize=undefined", "-fno-gpu-sanitize",
            *objs, "-o", exe]
    r = subprocess.run(link, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "host checks passed" in r.stdout, (r.stdout[-2000:], r.stderr[-6000:])
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr[-6000:]
