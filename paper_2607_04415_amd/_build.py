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
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off", "-fno-gpu-rdc", "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(CSRC.glob("*.hip")) + sorted(CSRC.glob("*.cpp"))


def build(verbose: bool = False, extra: list[str] | None = None) -> Path:
    """Always recompiles (the caller asked for a build)."""
    tmp = LIB.with_name(LIB.name + f".{os.getpid()}.tmp")
    cmd = [HIPCC, *FLAGS, *(extra or []), f"-I{INCLUDE}", "-o", str(tmp),
           *map(str, sources()), "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
