"""Build the C-ABI consumer check (tests/c_abi/relaysum_abi_check) against
the in-tree librelaysum.so and the HIP runtime, host code only."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "relaysum_abi_check.cpp")
BIN = os.path.join(HERE, "relaysum_abi_check")
PKG = os.path.join(ROOT, "paper_2110_04175_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False) -> str:
    tmp = BIN + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17", "-Wall",
           "-I", os.path.join(ROOT, "include"), SRC,
           "-L", PKG, "-lrelaysum", f"-Wl,-rpath,{PKG}", "-Wl,-rpath,$ORIGIN/../../paper_2110_04175_amd",
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True, cwd=HERE)
    os.replace(tmp, BIN)
    return BIN


if __name__ == "__main__":
    build(verbose=True)
