"""Builds the native test programs (test infrastructure; __graft_entry__.build()
calls build() after the library):

  abi_driver  a plain C++ program that uses libdisdp.so through
              include/disdp.h with the system HIP runtime and no PyTorch;
  api_fuzz    the C-ABI front end (disdp_api.cpp) compiled with g++ under
              AddressSanitizer and UndefinedBehaviorSanitizer, host code
              only, with stub HIP calls, fuzzed without a GPU."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_driver.cpp")
EXE = os.path.join(HERE, "abi_driver")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
PKG = os.path.join(ROOT, "paper_2409_00918_amd")


FUZZ_SRC = os.path.join(HERE, "api_fuzz.cpp")
FUZZ_EXE = os.path.join(HERE, "api_fuzz")
API_SRC = os.path.join(PKG, "csrc", "disdp_api.cpp")


def build_fuzz(verbose: bool = False) -> str:
    """g++ (host code only, no HIP device code) with both sanitizers."""
    tmp = FUZZ_EXE + ".tmp"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
           "-o", tmp, FUZZ_SRC, API_SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, FUZZ_EXE)
    return FUZZ_EXE


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
    build_fuzz(verbose)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
