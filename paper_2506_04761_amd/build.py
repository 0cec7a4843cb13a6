"""Builds libloglinear.so in-tree with hipcc for gfx950.

Usage: python paper_2506_04761_amd/build.py [-v] [--asan OUT]   (or call build()).
Every call recompiles; the sources are compiled in parallel, one hipcc process each, then linked.
Run it as a file, not as a package module: importing the package loads the library.

--asan OUT builds a second copy at OUT whose host code (argument checks, workspace layout,
launch bookkeeping) is instrumented with AddressSanitizer; the device code is built as usual.
Load it by setting LIBLOGLINEAR_PATH=OUT and preloading the compiler's ASan runtime.
"""

import concurrent.futures
import glob
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libloglinear.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # never emit packed-fp32 VALU ops (v_pk_fma_f32 and friends)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]

# Host-only sanitizer: each option applies to the host compilation alone.
ASAN_HOST_FLAGS = "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer".split()


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), flush=True)


def build(verbose: bool = False, asan: bool = False, out: str = None) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    out = out or LIB
    flags = list(HIPCC_FLAGS)
    if asan:
        flags = [f for f in flags if f != "-O3"] + ["-O1", "-g"] + ASAN_HOST_FLAGS
    srcs = sources()
    jobs = max(1, min(len(srcs), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1)), 16))
    with tempfile.TemporaryDirectory(prefix="ll_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in srcs]
        with concurrent.futures.ThreadPoolExecutor(jobs) as pool:
            for f in [pool.submit(_run, [hipcc] + flags + ["-c", s, "-o", o], verbose)
                      for s, o in zip(srcs, objs)]:
                f.result()
        tmp = out + ".tmp"
        _run([hipcc] + flags + ["-shared"] + objs + ["-o", tmp], verbose)
        os.replace(tmp, out)
    return out


if __name__ == "__main__":
    args = sys.argv[1:]
    asan_out = args[args.index("--asan") + 1] if "--asan" in args else None
    print(build(verbose="-v" in args, asan=asan_out is not None, out=asan_out))
