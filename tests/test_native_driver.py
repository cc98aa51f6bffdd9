"""The C ABI from a plain C++ program (tests/native/abi_driver.cpp): no
PyTorch, the system HIP runtime, hipMalloc / hipHostMalloc buffers, a
created stream, the error codes a C caller sees, and bit parity with the
CPU oracle for the fused call in both modes and in both launch shapes
(DISDP_LAUNCH_SHAPE set from C), the int32-contribution path,
a slab placed by disdp_shard_layout, and a shard in memory from the
virtual-memory API (hipMemCreate / hipMemMap, as VMM-based allocators hand
it out)."""
import os
import subprocess

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "native", "abi_driver")
PKG_LIB = os.path.join(os.path.dirname(HERE), "paper_2409_00918_amd", "libdisdp.so")
FUZZ = os.path.join(HERE, "native", "api_fuzz")


def _exe():
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built (python tests/native/build.py, or __graft_entry__.build())")
    return EXE


def test_driver_links_the_in_tree_library():
    """CPU: the program starts, resolves libdisdp.so from this tree and
    prints its usage without touching a GPU."""
    r = subprocess.run([_exe()], capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "usage" in r.stderr
    ldd = subprocess.run(["ldd", EXE], capture_output=True, text=True, timeout=60).stdout
    line = next(ln for ln in ldd.splitlines() if "libdisdp.so" in ln)
    assert os.path.realpath(line.split("=>")[1].split("(")[0].strip()) == os.path.realpath(PKG_LIB)


@pytest.mark.gpu
def test_c_abi_from_a_plain_cpp_program_matches_the_oracle():
    lib = oracle.build(force=False)
    r = subprocess.run([_exe(), lib], capture_output=True, text=True, timeout=300)
    print(r.stdout)
    print(r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_driver: all ok" in r.stdout


def test_api_front_end_fuzz_under_sanitizers():
    """CPU: the front end's argument checks, the layout planner and the
    choice of kernel, head and advanced pointers, over 500,000 random calls
    with AddressSanitizer and UndefinedBehaviorSanitizer (any finding
    aborts)."""
    if not os.path.exists(FUZZ):
        pytest.fail(f"{FUZZ} is not built (python tests/native/build.py)")
    r = subprocess.run([FUZZ], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "api_fuzz: ok" in r.stdout
