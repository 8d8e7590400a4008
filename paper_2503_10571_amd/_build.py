"""Compile the HIP library (libradar.so) in-tree for gfx950.

The library is built from several translation units compiled in parallel:
csrc/radar.hip (host logic, C ABI), csrc/build.hip (index build),
csrc/split.hip (the split path's kernels) and csrc/fused.hip once per
feature count n (-DRADAR_FUSED_N=n), then linked into one shared object.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libradar.so")
INCLUDE = os.path.join(ROOT, "include")
OBJ_DIR = os.path.join(HERE, "_build")
FEATURE_COUNTS = (64, 128, 256, 512, 1024, 2048)

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 ops are kept out of the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results land in ordinary VGPRs, so the exp2 epilogue of the index
    # build reads them without an accumulator-register copy per element
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def units():
    """(object name, source, extra flags) of every translation unit."""
    out = [("radar.o", "radar.hip", []), ("build.o", "build.hip", []),
           ("split.o", "split.hip", [])]
    out += [(f"fused_n{n}.o", "fused.hip", [f"-DRADAR_FUSED_N={n}"])
            for n in FEATURE_COUNTS]
    return out


def sources():
    """Every file the library is built from (for hashes of the source)."""
    names = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".h")))
    return [os.path.join(CSRC, f) for f in names] + [os.path.join(INCLUDE, "radar.h")]


def _stale(obj, src):
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    deps = [src, os.path.join(CSRC, "radar_impl.h"), os.path.join(INCLUDE, "radar.h"),
            os.path.abspath(__file__)]
    return any(os.path.getmtime(d) > t for d in deps)


def _compile(obj, src, extra):
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-c", src, "-o", obj + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)} {extra}:\n"
                           + res.stdout + res.stderr)
    os.replace(obj + ".tmp", obj)
    return " ".join(cmd)


def build_library(verbose: bool = False, force: bool = True, jobs: int | None = None) -> str:
    """Compile the units (all of them, or with force=False only those whose
    sources changed) and link libradar.so next to this file."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    todo, objs = [], []
    for name, src, extra in units():
        obj = os.path.join(OBJ_DIR, name)
        objs.append(obj)
        path = os.path.join(CSRC, src)
        if force or _stale(obj, path):
            todo.append((obj, path, extra))
    jobs = jobs or min(len(todo) or 1, os.cpu_count() or 1, 16)
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        for cmd in ex.map(lambda a: _compile(*a), todo):
            if verbose:
                print(cmd)
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("link failed:\n" + res.stdout + res.stderr)
    if verbose:
        print(" ".join(cmd))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build_library(verbose=True, force="--changed" not in sys.argv))
