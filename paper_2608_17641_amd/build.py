"""Compile the rlcs HIP library in-tree for gfx950.

    python -m paper_2608_17641_amd.build

produces ``paper_2608_17641_amd/librlcs.so`` from the translation units ``csrc/rlcs_*.hip``
(one per group of entry points, compiled in parallel; kernels in ``csrc/rlcs_*.h``) against
the public header ``include/rlcs.h``, and ``paper_2608_17641_amd/libprobe.so`` from
``csrc/probe_stream.hip``: reference kernels that bench.py times beside the library (a streaming
copy with GAE's byte split, an empty launch), not part of the library.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librlcs.so")
PROBE_LIB = os.path.join(PKG, "libprobe.so")
PROBE_SOURCE = os.path.join(CSRC, "probe_stream.hip")
SOURCES = sorted(glob.glob(os.path.join(CSRC, "rlcs_*.hip")))
HEADERS = sorted(glob.glob(os.path.join(CSRC, "rlcs_*.h"))) + [os.path.join(INCLUDE, "rlcs.h")]

ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the rlcs library)")


FLAGS = [
    "-O3", f"--offload-arch={ARCH}", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no sinking of the stores that end two branches into one store through a selected address:
    # where the element-wise and vector load paths of a chunk last wrote different arrays (the
    # truncation continuation of its last step in one, its bootstrap in the other), that store
    # kept both arrays in private memory, 12 bytes per lane written through to HBM (masked GAE
    # 4096 x 256: 25 % more bytes written, 6.08 -> 5.20 us without; discounted returns on rows
    # of 255 steps 5.85 -> 4.92 us)
    "-mllvm", "-simplifycfg-sink-common=false",
    "-Wall", "-Wno-unused-function",
]


def compile_command(src: str, obj: str):
    return [hipcc(), *FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c", "-o", obj, src]


def link_command(objs, out: str = LIB):
    return [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out, *objs]


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


_NOISE = ("is not a recognized feature for this target", "(ignoring feature)")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if not any(n in l for n in _NOISE))
    return res.returncode, err


def build(force: bool = True, verbose: bool = False) -> str:
    """Compile librlcs.so and libprobe.so: always when force, else only what does not exist
    yet."""
    if not force and os.path.exists(LIB) and os.path.exists(PROBE_LIB):
        return LIB
    with tempfile.TemporaryDirectory(prefix="rlcs_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.basename(src) + ".o") for src in SOURCES]
        probe_obj = os.path.join(tmpdir, "probe_stream.o")
        jobs = min(len(SOURCES) + 1, max(1, min(8, os.cpu_count() or 1)))
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            results = list(pool.map(lambda so: (so[0], _run(compile_command(*so))),
                                    list(zip(SOURCES, objs)) + [(PROBE_SOURCE, probe_obj)]))
        for src, (rc, err) in results:
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {src} ({rc}):\n{err}")
            if verbose and err.strip():
                print(err, file=sys.stderr)
        for objects, out in ((objs, LIB), ([probe_obj], PROBE_LIB)):
            tmp = out + f".tmp{os.getpid()}"
            rc, err = _run(link_command(objects, tmp))
            if rc != 0:
                if os.path.exists(tmp):
                    os.remove(tmp)
                raise RuntimeError(f"link of {os.path.basename(out)} failed ({rc}):\n{err}")
            os.replace(tmp, out)
    return LIB


if __name__ == "__main__":
    print(build(force=True, verbose=True))
