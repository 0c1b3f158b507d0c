"""Build libfabft.so (HIP kernels for gfx950 + the C ABI) in-tree.

    python -m paper_2507_16676_amd.build [-v]
    python -m paper_2507_16676_amd.build --host-sanitize OUT.so

The second form builds a copy with AddressSanitizer and UndefinedBehavior-
Sanitizer on the host code only (argument validation, launch set-up; the
device code is built as usual) into OUT.so, leaving the in-tree library
alone. Load it with FABFT_LIB=OUT.so and the ASan runtime preloaded, e.g.

    ASAN_OPTIONS=detect_leaks=0 LD_PRELOAD=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so) \
        FABFT_LIB=OUT.so python -m pytest tests/test_abi.py

Compiles with hipcc for gfx950 only. Packed fp32 VALU instructions are
switched off for device code (``-packed-fp32-ops``); the host pass warns that
it does not know that feature, which is harmless.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libfabft.so")
SOURCES = [os.path.join(CSRC, "fabft_kernels.hip"), os.path.join(CSRC, "fabft_api.cpp")]
ARCH = "gfx950"


def hipcc_path() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libfabft.so)")


COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# Kernels only: IEEE mode off, so max/min need no NaN-quieting of their inputs
# (needs relaxed NaN rules; the kernels test non-finite values on the bits and
# a NaN score still reaches exp2 and propagates into o, l and c).
KERNEL_FLAGS = ["-mno-amdgpu-ieee", "-fno-honor-nans",
                # the two-pass kernels unroll their loop over the two passes
                # (each pass then has constant branches); the injection forms
                # of that loop exceed LLVM's default size limit for a requested
                # unroll, and rolled up they spill. No other kernel changes.
                "-mllvm", "-pragma-unroll-threshold=100000"]


# The kernel source is compiled twice (FABFT_PART 0 and 1, see its head): the
# second part, the d = 128 forward kernels without the weighted check, with
# LLVM's iterative ILP scheduler.
PART1_FLAGS = ["-DFABFT_PART=1", "-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]


def build_cmds(out: str, objdir: str, extra=()) -> list[list[str]]:
    inc = ["-I", os.path.join(ROOT, "include")]
    hipcc = hipcc_path()
    k_obj = os.path.join(objdir, "fabft_kernels.o")
    k1_obj = os.path.join(objdir, "fabft_kernels_part1.o")
    a_obj = os.path.join(objdir, "fabft_api.o")
    return [
        [hipcc, "-x", "hip", *COMMON, *KERNEL_FLAGS, *inc, *extra, "-c", SOURCES[0], "-o", k_obj],
        [hipcc, "-x", "hip", *COMMON, *KERNEL_FLAGS, *PART1_FLAGS, *inc, *extra, "-c", SOURCES[0],
         "-o", k1_obj],
        [hipcc, "-x", "hip", *COMMON, *inc, *extra, "-c", SOURCES[1], "-o", a_obj],
        [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", k_obj, k1_obj, a_obj, "-o", out],
    ]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in line)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)


# every sanitizer flag is bound to the host pass (-Xarch_host): the device code
# is built exactly as in the product library
SANITIZERS = ("address", "undefined")
HOST_SANITIZE = [f for s in SANITIZERS for f in ("-Xarch_host", "-fsanitize=" + s)] + [
    "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def _run_all(cmds, verbose):
    """The compile steps (all but the last command) run side by side; the
    link runs after them."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=len(cmds) - 1) as ex:
        for f in [ex.submit(_run, c, verbose) for c in cmds[:-1]]:
            f.result()
    _run(cmds[-1], verbose)


def build_host_sanitized(out: str, verbose: bool = False) -> str:
    """libfabft.so with ASan and UBSan on the host code, written to `out`."""
    import tempfile
    with tempfile.TemporaryDirectory(prefix="fabft_build_") as objdir:
        cmds = build_cmds(out, objdir, HOST_SANITIZE)
        link = cmds[-1]
        cmds[-1] = (link[:-2] + [f for s in SANITIZERS for f in ("-Xarch_host", "-fsanitize=" + s)]
                    + ["-shared-libsan"] + link[-2:])
        _run_all(cmds, verbose)
    return out


def build(verbose: bool = False, extra=()) -> str:
    import tempfile
    tmp = LIB + f".tmp{os.getpid()}"
    with tempfile.TemporaryDirectory(prefix="fabft_build_") as objdir:
        try:
            _run_all(build_cmds(tmp, objdir, extra), verbose)
        except Exception:
            if os.path.exists(tmp):
                os.unlink(tmp)
            raise
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    v = "-v" in sys.argv
    if "--host-sanitize" in sys.argv:
        print(build_host_sanitized(sys.argv[sys.argv.index("--host-sanitize") + 1], verbose=v))
        sys.exit(0)
    extra = ["-Rpass-analysis=kernel-resource-usage"] if "--usage" in sys.argv else []
    print(build(verbose=v or bool(extra), extra=extra))
