"""CPU oracle for the DisDP parameter-server hot path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product (``paper_2409_00918_amd``)
never imports it and shares no code with it: the oracle is plain C built by
gcc (``disdp_oracle.c``), loaded here through ctypes and fed numpy arrays.

What it computes (arXiv 2409.00918):
  * ``aggregate_f32``   -- the switch's W-way gradient sum in worker order
                          (Section III-A overall architecture; Section III-C).
  * ``aggregate_fixed`` -- the same sum in the integer format of the SmartNIC
                          format-conversion unit (Section III-B), bit-exact;
                          contributions may be float32, bf16 or int32 that is
                          already in that format.
  * ``quantize_array``  -- that format conversion over a buffer.
  * ``adamw``           -- the parameter server's mixed-precision Adam step,
                          step 5 of the backward stage (Section III-D, Table III).
  * ``fused``           -- the two composed, element by element
                          (``fused_inplace``: the same on caller arrays).
  * ``bf16_rne``        -- the 2-byte parameter copy written by step 5.

All floating-point work happens in the C file in IEEE binary32 with the
operation order documented there.  Every function is pinned by
``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "disdp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

DT_F32, DT_BF16, DT_I32 = 0, 1, 2
AGG_FP32, AGG_FIXED = 0, 1

# gcc flags: IEEE binary32 with no contraction and no fast-math shortcuts.
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-frounding-math", "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile ``disdp_oracle.c`` with gcc into ``liboracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def load_library(path: str) -> ctypes.CDLL:
    """Load an oracle build from `path` and declare its signatures."""
    L = ctypes.CDLL(path)
    vp, i64, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float
    ci = ctypes.c_int
    L.oracle_bf16_rne.restype = ctypes.c_uint16
    L.oracle_bf16_rne.argtypes = [f32]
    L.oracle_bf16_to_f32.restype = f32
    L.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
    L.oracle_quantize.restype = ctypes.c_int32
    L.oracle_quantize.argtypes = [f32, ci]
    L.oracle_quantize_array.restype = None
    L.oracle_quantize_array.argtypes = [vp, ci, i64, ci, vp]
    L.oracle_aggregate_f32.restype = None
    L.oracle_aggregate_f32.argtypes = [vp, ci, ci, i64, vp]
    L.oracle_aggregate_fixed.restype = None
    L.oracle_aggregate_fixed.argtypes = [vp, ci, ci, i64, ci, vp, vp]
    L.oracle_scalars.restype = None
    L.oracle_scalars.argtypes = [f32, f32, f32, f32, i64, vp]
    L.oracle_adamw.restype = None
    L.oracle_adamw.argtypes = [vp, vp, vp, vp, vp, i64,
                               f32, f32, f32, f32, f32, i64, f32]
    L.oracle_fused.restype = None
    L.oracle_fused.argtypes = [vp, ci, ci, i64, ci, ci, vp, vp, vp, vp,
                               vp, vp, f32, f32, f32, f32, f32, i64, f32]
    L.oracle_mxcsr_ftz_daz.restype = ctypes.c_uint
    L.oracle_mxcsr_ftz_daz.argtypes = []
    return L


def lib() -> ctypes.CDLL:
    """The loaded oracle library (built on first use if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


@contextlib.contextmanager
def using(library: ctypes.CDLL):
    """Run the wrappers below against another build (the mutation tests)."""
    global _lib
    saved = lib()
    _lib = library
    try:
        yield
    finally:
        _lib = saved


def build_source(src_text: str, out_path: str) -> str:
    """Compile C source text with the oracle's flags into `out_path`."""
    src = out_path + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", *CFLAGS, "-o", out_path, src, "-lm"])
    return out_path


def source() -> str:
    with open(_SRC) as f:
        return f.read()


# ---------------------------------------------------------------- helpers --
def _ptr(a: Optional[np.ndarray]) -> Optional[int]:
    return None if a is None else a.ctypes.data


def _grad_dtype(gs: Sequence[np.ndarray]) -> int:
    dt = {g.dtype for g in gs}
    if len(dt) != 1:
        raise TypeError("all contributions must share one dtype")
    d = dt.pop()
    if d == np.float32:
        return DT_F32
    if d == np.uint16:        # bf16 carried as raw bits
        return DT_BF16
    if d == np.int32:         # contributions already in the integer format
        return DT_I32
    raise TypeError(f"unsupported gradient dtype {d}")


def _ptr_array(gs: Sequence[np.ndarray]):
    for g in gs:
        if not g.flags.c_contiguous:
            raise ValueError("contributions must be contiguous")
    arr = (ctypes.c_void_p * len(gs))(*[g.ctypes.data for g in gs])
    return arr


def _check_n(gs: Sequence[np.ndarray]) -> int:
    if not 1 <= len(gs) <= 64:
        raise ValueError("W must be in [1, 64]")
    n = gs[0].size
    if any(g.size != n for g in gs):
        raise ValueError("contributions differ in length")
    return n


def bf16_rne(x) -> np.ndarray:
    """fp32 -> bf16 bits (uint16), round to nearest even, elementwise."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    L = lib()
    return np.fromiter((L.oracle_bf16_rne(float(v)) for v in x),
                       dtype=np.uint16, count=x.size)


def bf16_to_f32(h) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16).ravel()
    L = lib()
    return np.fromiter((L.oracle_bf16_to_f32(int(v)) for v in h),
                       dtype=np.float32, count=h.size)


def quantize(x, k: int) -> np.ndarray:
    """Element by element through oracle_quantize (float32 input)."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    L = lib()
    return np.fromiter((L.oracle_quantize(float(v), k) for v in x),
                       dtype=np.int32, count=x.size)


def quantize_array(g: np.ndarray, k: int) -> np.ndarray:
    """oracle_quantize_array over a float32 or bf16 (uint16 bits) buffer."""
    g = np.ascontiguousarray(g)
    out = np.empty(g.size, dtype=np.int32)
    lib().oracle_quantize_array(g.ctypes.data, _grad_dtype([g]), g.size, k,
                                out.ctypes.data)
    return out


def scalars(lr, beta1, beta2, wd, t) -> np.ndarray:
    """[beta1, 1-beta1, beta2, 1-beta2, 1-beta1^t, 1-beta2^t, 1-lr*wd] as fp32."""
    out = np.zeros(7, dtype=np.float32)
    lib().oracle_scalars(lr, beta1, beta2, wd, t, out.ctypes.data)
    return out


def aggregate_f32(gs: Sequence[np.ndarray]) -> np.ndarray:
    n = _check_n(gs)
    out = np.empty(n, dtype=np.float32)
    lib().oracle_aggregate_f32(_ptr_array(gs), len(gs), _grad_dtype(gs), n,
                               out.ctypes.data)
    return out


def aggregate_fixed(gs: Sequence[np.ndarray], k: int):
    """Returns (int32 aggregate, fp32 dequantised aggregate)."""
    n = _check_n(gs)
    ai = np.empty(n, dtype=np.int32)
    af = np.empty(n, dtype=np.float32)
    lib().oracle_aggregate_fixed(_ptr_array(gs), len(gs), _grad_dtype(gs), n,
                                 k, ai.ctypes.data, af.ctypes.data)
    return ai, af


def adamw(agg, p, m, v, *, lr, beta1, beta2, eps, wd, t, grad_scale=1.0,
          want_bf16=True):
    """One step on copies of p, m, v.  Returns (p, m, v, p16 or None)."""
    agg = np.ascontiguousarray(agg, dtype=np.float32)
    p = np.array(p, dtype=np.float32, copy=True)
    m = np.array(m, dtype=np.float32, copy=True)
    v = np.array(v, dtype=np.float32, copy=True)
    n = agg.size
    assert p.size == m.size == v.size == n
    p16 = np.empty(n, dtype=np.uint16) if want_bf16 else None
    lib().oracle_adamw(agg.ctypes.data, p.ctypes.data, m.ctypes.data,
                       v.ctypes.data, _ptr(p16), n, lr, beta1, beta2, eps, wd,
                       t, grad_scale)
    return p, m, v, p16


def fused(gs: Sequence[np.ndarray], p, m, v, *, mode=AGG_FP32, frac_bits=0,
          lr, beta1, beta2, eps, wd, t, grad_scale=1.0, want_bf16=True,
          want_agg_f32=False, want_agg_i32=False):
    """Aggregate + AdamW on copies of p, m, v.

    Returns a dict with keys p, m, v and, when requested, p16, agg_f32,
    agg_i32."""
    n = _check_n(gs)
    p = np.array(p, dtype=np.float32, copy=True)
    m = np.array(m, dtype=np.float32, copy=True)
    v = np.array(v, dtype=np.float32, copy=True)
    assert p.size == m.size == v.size == n
    p16 = np.empty(n, dtype=np.uint16) if want_bf16 else None
    af = np.empty(n, dtype=np.float32) if want_agg_f32 else None
    ai = np.empty(n, dtype=np.int32) if want_agg_i32 else None
    lib().oracle_fused(_ptr_array(gs), len(gs), _grad_dtype(gs), n, mode,
                       frac_bits, p.ctypes.data, m.ctypes.data, v.ctypes.data,
                       _ptr(p16), _ptr(af), _ptr(ai), lr, beta1, beta2, eps,
                       wd, t, grad_scale)
    out = {"p": p, "m": m, "v": v}
    if want_bf16:
        out["p16"] = p16
    if want_agg_f32:
        out["agg_f32"] = af
    if want_agg_i32:
        out["agg_i32"] = ai
    return out


def fused_inplace(gs: Sequence[np.ndarray], p: np.ndarray, m: np.ndarray, v: np.ndarray,
                  p16: Optional[np.ndarray], *, mode=AGG_FP32, frac_bits=0, lr, beta1,
                  beta2, eps, wd, t, grad_scale=1.0) -> None:
    """The same step as ``fused`` on caller-owned arrays, updated in place:
    p, m, v float32 and p16 uint16 (or None), all contiguous, nothing
    allocated or copied -- for timing the oracle itself."""
    n = _check_n(gs)
    for a in (p, m, v) + (() if p16 is None else (p16,)):
        if a.size != n or not a.flags.c_contiguous:
            raise ValueError("state arrays must be contiguous and of the shard's length")
    if p.dtype != np.float32 or m.dtype != np.float32 or v.dtype != np.float32 or \
            (p16 is not None and p16.dtype != np.uint16):
        raise TypeError("p, m, v must be float32 and p16 uint16")
    lib().oracle_fused(_ptr_array(gs), len(gs), _grad_dtype(gs), n, mode, frac_bits,
                       p.ctypes.data, m.ctypes.data, v.ctypes.data, _ptr(p16), None, None,
                       lr, beta1, beta2, eps, wd, t, grad_scale)


def fp_env_ok() -> bool:
    """True when the host FPU keeps denormals (no FTZ/DAZ)."""
    return lib().oracle_mxcsr_ftz_daz() == 0
