"""Builds libdisdp.so in-tree with hipcc for gfx950.

    python -m paper_2409_00918_amd.build

Flags:
  --offload-arch=gfx950     MI355X only; no other target, no host fallback.
  -ffp-contract=off         one rounding per operation (no FMA contraction);
                            the kernels also say so with a pragma.
  -Xclang -target-feature -Xclang -packed-fp32-ops
                            keep the compiler from emitting packed fp32
                            arithmetic (v_pk_*_f32); the host pass warns that
                            it does not know the feature, which is harmless.
HIP's defaults give correctly rounded fp32 division and square root and keep
fp32 denormals; nothing here overrides them.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdisdp.so")
# measurement helper for bench.py (a plain copy kernel); not part of the ABI
PROBE_LIB = os.path.join(PKG, "libdisdp_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "hbm_probe.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = [os.path.join(CSRC, "disdp_api.cpp"),
           os.path.join(CSRC, "disdp_kernels.hip")]

FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
         "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-command-line-argument",
         "-I", INCLUDE, "-I", CSRC]


def _compile(out: str, sources, verbose: bool) -> None:
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    _compile(LIB, SOURCES, verbose)
    _compile(PROBE_LIB, PROBE_SOURCES, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
