"""Compile the rlcs HIP library in-tree for gfx950.

    python -m paper_2608_17641_amd.build

produces ``paper_2608_17641_amd/librlcs.so`` from ``csrc/rlcs.hip`` (kernels in
``csrc/rlcs_*.h``) against the public header ``include/rlcs.h``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librlcs.so")
SOURCES = [os.path.join(CSRC, "rlcs.hip")]
HEADERS = [os.path.join(CSRC, f) for f in ("rlcs_device.h", "rlcs_estimators.h", "rlcs_kernels.h")]
HEADERS.append(os.path.join(INCLUDE, "rlcs.h"))

ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the rlcs library)")


def command(out: str = LIB):
    return [
        hipcc(), "-O3", f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-shared",
        # packed fp32 instructions are kept out of the generated code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function",
        f"-I{INCLUDE}", f"-I{CSRC}",
        "-o", out, *SOURCES,
    ]


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


def build(force: bool = True, verbose: bool = False) -> str:
    """Compile librlcs.so: always when force, else only if it does not exist yet."""
    if not force and os.path.exists(LIB):
        return LIB
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = command(tmp)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l and "(ignoring feature)" not in l)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force=True, verbose=True))
