"""Host-side AddressSanitizer run of the C ABI checks.

Builds a second copy of libloglinear whose host code is instrumented with AddressSanitizer
(build.py --asan; the device code is unchanged), then runs the host-only ABI tests against it
in a child process with the sanitizer runtime preloaded.  Any heap or stack overrun in the
argument checks, the workspace-size arithmetic or the status strings aborts the child."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"


def _asan_runtime():
    if not os.path.exists(CLANG):
        return None
    res = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    path = res.stdout.strip()
    return path if res.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(600)
def test_abi_checks_are_clean_under_host_asan(tmp_path):
    runtime = _asan_runtime()
    if shutil.which(HIPCC) is None or runtime is None:
        pytest.skip("hipcc or the clang ASan runtime is not installed")
    sys.path.insert(0, os.path.join(ROOT, "paper_2506_04761_amd"))
    try:
        import build as build_mod
    finally:
        sys.path.pop(0)
    lib = build_mod.build(asan=True, out=str(tmp_path / "libloglinear_asan.so"))
    assert b"__asan_report" in open(lib, "rb").read()

    env = dict(os.environ)
    env["LIBLOGLINEAR_PATH"] = lib
    env["LD_PRELOAD"] = runtime + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    check = ("import os, paper_2506_04761_amd._lib as m; "
             "assert m.LIB_PATH == os.environ['LIBLOGLINEAR_PATH'], m.LIB_PATH")
    res = subprocess.run([sys.executable, "-c", check], cwd=ROOT, env=env,
                         capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    out = res.stdout + res.stderr
    assert res.returncode == 0 and "AddressSanitizer" not in out, out[-4000:]
