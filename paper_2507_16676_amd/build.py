"""Build libfabft.so (HIP kernels for gfx950 + the C ABI) in-tree.

    python -m paper_2507_16676_amd.build [-v]

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


def build_cmd(out: str, extra=()) -> list[str]:
    return [hipcc_path(), f"--offload-arch={ARCH}", "-O3", "-std=c++17",
            "-shared", "-fPIC", "-x", "hip",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), *extra, "-o", out, *SOURCES]


def build(verbose: bool = False, extra=()) -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = build_cmd(tmp, extra)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in line)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.unlink(tmp)
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    v = "-v" in sys.argv
    extra = ["-Rpass-analysis=kernel-resource-usage"] if "--usage" in sys.argv else []
    print(build(verbose=v or bool(extra), extra=extra))
