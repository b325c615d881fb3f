"""Compile the HIP library (libgorio.so) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
LIB = PKG / "libgorio.so"
INCLUDE = PKG.parent / "include"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off", "-fno-gpu-rdc", "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(CSRC.glob("*.hip")) + sorted(CSRC.glob("*.cpp"))


def build(verbose: bool = False, extra: list[str] | None = None, jobs: int | None = None) -> Path:
    """Always recompiles (the caller asked for a build): every source to an
    object file in parallel, then one link."""
    from concurrent.futures import ThreadPoolExecutor

    objdir = PKG / "_build"
    objdir.mkdir(exist_ok=True)
    tag = os.getpid()

    def compile_one(src: Path) -> Path:
        obj = objdir / f"{src.name}.{tag}.o"
        cmd = [HIPCC, *FLAGS, *(extra or []), f"-I{INCLUDE}", "-c", "-o", str(obj), str(src)]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        return obj

    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 2) // 2))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = LIB.with_name(LIB.name + f".{tag}.tmp")
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-fno-gpu-rdc", "-o", str(tmp),
           *map(str, objs), "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    try:
        subprocess.run(cmd, check=True)
    finally:
        for o in objs:
            o.unlink(missing_ok=True)
    os.replace(tmp, LIB)
    build_microbench(verbose)
    return LIB


MICROBENCH = PKG / "microbench"
GATHER_CEILING = MICROBENCH / "gather_ceiling"


def build_microbench(verbose: bool = False) -> Path:
    """The random-gather ceiling probe (a standalone HIP program bench.py runs)."""
    src = MICROBENCH / "gather_ceiling.hip"
    tmp = GATHER_CEILING.with_name(GATHER_CEILING.name + f".{os.getpid()}.tmp")
    cmd = [HIPCC, *FLAGS, "-o", str(tmp), str(src)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, GATHER_CEILING)
    return GATHER_CEILING


if __name__ == "__main__":
    print(build(verbose=True))
