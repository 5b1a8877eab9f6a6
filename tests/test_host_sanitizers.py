"""The host code of the library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The planner, the launch-table builder and checker and the split cost model run
inside every jorge_create, and jorge_plan / jorge_plan_stages run them without
a GPU. This test builds the library a second time with the host half
instrumented (the GPU half is compiled as usual and never runs), then runs
tests/test_abi_host.py against that build in a child process with the ASan
runtime preloaded, stopping at the first report of either sanitizer. Leak
detection is off: the Python interpreter itself holds allocations at exit.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _asan_runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


@pytest.mark.skipif(not os.path.exists(HIPCC) or _asan_runtime() is None,
                    reason="needs hipcc and the clang ASan runtime")
def test_host_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    lib = str(tmp_path / "libjorge_sanitized.so")
    # Each sanitizer flag applies to the host compilation only (-Xarch_host).
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-shared-libasan", "-fno-omit-frame-pointer",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2310_12298_amd", "csrc", "jorge.hip"), "-o", lib]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    nm = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in nm and "__ubsan_handle" in nm, "the host code is not instrumented"
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    child = ("import sys; sys.path[:0] = [{root!r}, {tests!r}]\n"
             "import paper_2310_12298_amd.jorge as J\n"
             "J.LIB_PATH = {lib!r}\n"
             "import pytest\n"
             "sys.exit(pytest.main([{abi!r}, '-q', '-p', 'no:cacheprovider']))\n").format(
        root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib, abi=os.path.join(ROOT, "tests", "test_abi_host.py"))
    res = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, env=env, cwd=ROOT,
                         timeout=900)
    out = res.stdout + res.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert res.returncode == 0, out[-6000:]
    assert " passed" in res.stdout and " failed" not in res.stdout, res.stdout[-3000:]
