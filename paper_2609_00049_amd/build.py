"""Build librealq.so (the gfx950 HIP library behind include/realq.h) in-tree with hipcc.

    python -m paper_2609_00049_amd.build          # or: python paper_2609_00049_amd/build.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
LIB = PKG / "librealq.so"
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]
OBJ = PKG / "_build"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and Path(cand).exists():
            return cand
    raise RuntimeError("hipcc not found (ROCm required to build the HIP library)")


def sources():
    """HIP sources plus the host-only C++ units (launch planning)."""
    return sorted(str(p) for p in CSRC.glob("*.hip")) + sorted(str(p) for p in CSRC.glob("*.cpp"))


def _compile(src: str, verbose: bool) -> Path:
    obj = OBJ / (Path(src).name + ".o")
    cmd = [hipcc(), *HIPCC_FLAGS, f"-I{ROOT / 'include'}", "-c", src, "-o", str(obj)]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass warns that it does not know the packed-fp32 feature; only errors matter
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed on {src} with exit code {res.returncode}")
    return obj


def build(verbose: bool = False) -> Path:
    """Compile every source into librealq.so (always recompiles; one hipcc per source, in parallel)."""
    from concurrent.futures import ThreadPoolExecutor
    OBJ.mkdir(exist_ok=True)
    srcs = sources()
    workers = max(1, min(len(srcs), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(lambda p: _compile(p, verbose), srcs))
    tmp = LIB.with_suffix(".so.tmp")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *[str(o) for o in objs],
           "-lrocprofiler-sdk-roctx", "-o", str(tmp)]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"link failed with exit code {res.returncode}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
