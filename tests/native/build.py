"""Builds tests/native/abi_driver: a plain C++ program that uses libdisdp.so
through include/disdp.h with the system HIP runtime and no PyTorch.  Test
infrastructure; __graft_entry__.build() calls build() after the library."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_driver.cpp")
EXE = os.path.join(HERE, "abi_driver")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
PKG = os.path.join(ROOT, "paper_2409_00918_amd")


def build(verbose: bool = False) -> str:
    tmp = EXE + ".tmp"
    cmd = [HIPCC, "-O2", "-std=c++17", "-Wall", "-Wno-unused-command-line-argument",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-o", tmp, SRC,
           "-L", PKG, "-ldisdp", "-Wl,-rpath,$ORIGIN/../../paper_2409_00918_amd", "-ldl"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
