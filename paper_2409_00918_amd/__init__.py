"""Python binding of libdisdp: the DisDP parameter-server hot path on MI355X.

Thin ctypes marshalling over the C ABI declared in ``include/disdp.h``: the
functions below turn torch device tensors into pointers, lengths and the
current HIP stream and call the library.  Every step of the path -- the W-way
reduction of the gradient contributions (the SmartSwitch's aggregation,
Sections III-A and III-C of arXiv 2409.00918, in fp32 or in the integer format
of Section III-B), the Adam step with decoupled weight decay and the bf16
parameter copy (Section III-D, step 5) -- runs in the library's HIP kernels.
There is no other implementation here: if ``libdisdp.so`` is missing, every
call raises.

``aggregate``       -- the reduction alone            (disdp_aggregate)
``adam_step``       -- the optimizer step alone       (disdp_adam_step)
``aggregate_adam``  -- both in one pass               (disdp_aggregate_adam)
``quantize``        -- a worker's float -> int32 conversion (disdp_quantize)
``allocate_shard``  -- one device allocation holding a shard's arrays, placed
                       by disdp_shard_layout (``contiguous_bytes``: such an
                       allocation, physically contiguous)
``aggregate_adam_dev``, ``step_scalars``
                    -- the fused call with the step's constants read from
                       device memory (one HIP graph for every step)
``aggregate_adam_multi`` -- the fused call over many tensors in separate
                       buffers (a batch of tensors per launch)
``MultiTensorStep`` -- the same over a fixed list of tensors, checked and
                       packed once, one step per call
"""
from __future__ import annotations

import ctypes
import os
import sys
import threading
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdisdp.so")

# Status codes, dtypes and modes (values fixed by include/disdp.h).
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_ALIAS, ERR_HIP = 0, 1, 2, 3, 4
DT_F32, DT_BF16, DT_I32 = 0, 1, 2
AGG_FP32, AGG_FIXED = 0, 1
MAX_W = 64

EXPORTS = ("disdp_aggregate", "disdp_adam_step", "disdp_aggregate_adam",
           "disdp_quantize", "disdp_shard_layout", "disdp_step_scalars",
           "disdp_aggregate_adam_dev", "disdp_aggregate_adam_multi",
           "disdp_status_string")
LAYOUT_BF16_COPY, LAYOUT_AGG_F32, LAYOUT_AGG_I32 = 1, 2, 4


class AdamWHParams(ctypes.Structure):
    """disdp_adamw_hparams_t."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("step", ctypes.c_int64),
                ("grad_scale", ctypes.c_float)]


class StepScalars(ctypes.Structure):
    """disdp_step_scalars_t: the per-step constants of the optimizer."""
    _fields_ = [("beta1", ctypes.c_float), ("one_minus_beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("one_minus_beta2", ctypes.c_float),
                ("bias_correction1", ctypes.c_float), ("bias_correction2", ctypes.c_float),
                ("decay", ctypes.c_float), ("lr", ctypes.c_float), ("eps", ctypes.c_float),
                ("grad_scale", ctypes.c_float)]


class DisdpError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


_lib = None


def hip_runtimes_mapped() -> list:
    """Paths of every HIP runtime library mapped into this process."""
    with open("/proc/self/maps") as f:
        return sorted({line.split()[-1] for line in f
                       if "libamdhip64" in line.rsplit("/", 1)[-1]})


def lib() -> ctypes.CDLL:
    """The loaded libdisdp.so.  Raises if it has not been built.

    torch ships its own HIP runtime under the same soname as the system one
    (libamdhip64.so.7).  torch is imported first so that the library's
    dependency binds to that already-loaded runtime: loaded the other way
    round, the process would hold two HIP runtimes and the library's launches
    would go to one that does not own torch's memory and streams."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2409_00918_amd.build` (hipcc, gfx950)")
        import torch  # noqa: F401  (binds libamdhip64.so.7 to torch's runtime)
        L = ctypes.CDLL(LIB_PATH)
        runtimes = hip_runtimes_mapped()
        if len(runtimes) > 1:
            raise RuntimeError(
                "two HIP runtimes are loaded in this process "
                f"({', '.join(runtimes)}); load libdisdp through this module "
                "after importing torch, not before")
        vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.disdp_aggregate.restype = ci
        L.disdp_aggregate.argtypes = [vp, ci, ci, i64, ci, ci, vp, vp, vp]
        L.disdp_adam_step.restype = ci
        L.disdp_adam_step.argtypes = [vp, vp, vp, vp, vp, i64,
                                      ctypes.POINTER(AdamWHParams), vp]
        L.disdp_aggregate_adam.restype = ci
        L.disdp_aggregate_adam.argtypes = [vp, ci, ci, i64, ci, ci, vp, vp, vp,
                                           vp, vp, vp,
                                           ctypes.POINTER(AdamWHParams), vp]
        L.disdp_quantize.restype = ci
        L.disdp_quantize.argtypes = [vp, ci, i64, ci, vp, vp]
        L.disdp_shard_layout.restype = ci
        L.disdp_shard_layout.argtypes = [i64, ci, ci, ctypes.c_uint, vp, vp]
        L.disdp_step_scalars.restype = ci
        L.disdp_step_scalars.argtypes = [ctypes.POINTER(AdamWHParams), ctypes.POINTER(StepScalars)]
        L.disdp_aggregate_adam_dev.restype = ci
        L.disdp_aggregate_adam_dev.argtypes = [vp, ci, ci, i64, ci, ci, vp, vp, vp, vp, vp, vp,
                                               vp, vp]
        L.disdp_aggregate_adam_multi.restype = ci
        L.disdp_aggregate_adam_multi.argtypes = [vp, ci, ci, ci, vp, ci, ci, vp, vp, vp, vp,
                                                 ctypes.POINTER(AdamWHParams), vp, vp]
        L.disdp_status_string.restype = ctypes.c_char_p
        L.disdp_status_string.argtypes = [ci]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().disdp_status_string(int(status)).decode()


# ------------------------------------------------------------ raw calls --
# Integer pointers and sizes exactly as the C ABI takes them; used by the
# tensor wrappers below and by the ABI tests.
def _ptr_array(ptrs: Sequence[int]):
    return (ctypes.c_void_p * max(1, len(ptrs)))(*[p or None for p in ptrs])


def raw_aggregate(grad_ptrs, W, gdtype, n, mode, frac_bits, agg_f32, agg_i32,
                  stream) -> int:
    arr = None if grad_ptrs is None else _ptr_array(grad_ptrs)
    return lib().disdp_aggregate(arr, W, gdtype, n, mode, frac_bits,
                                 agg_f32 or None, agg_i32 or None,
                                 stream or None)


def raw_quantize(grad, gdtype, n, frac_bits, out, stream) -> int:
    return lib().disdp_quantize(grad or None, gdtype, n, frac_bits, out or None,
                                stream or None)


def raw_adam_step(grad, param, m, v, p16, n, hp: Optional[AdamWHParams],
                  stream) -> int:
    return lib().disdp_adam_step(grad or None, param or None, m or None,
                                 v or None, p16 or None, n,
                                 None if hp is None else ctypes.byref(hp),
                                 stream or None)


def raw_aggregate_adam(grad_ptrs, W, gdtype, n, mode, frac_bits, param, m, v,
                       p16, agg_f32, agg_i32, hp: Optional[AdamWHParams],
                       stream) -> int:
    arr = None if grad_ptrs is None else _ptr_array(grad_ptrs)
    return lib().disdp_aggregate_adam(
        arr, W, gdtype, n, mode, frac_bits, param or None, m or None,
        v or None, p16 or None, agg_f32 or None, agg_i32 or None,
        None if hp is None else ctypes.byref(hp), stream or None)


def raw_aggregate_adam_dev(grad_ptrs, W, gdtype, n, mode, frac_bits, param, m, v,
                           p16, agg_f32, agg_i32, scalars, stream) -> int:
    arr = None if grad_ptrs is None else _ptr_array(grad_ptrs)
    return lib().disdp_aggregate_adam_dev(
        arr, W, gdtype, n, mode, frac_bits, param or None, m or None,
        v or None, p16 or None, agg_f32 or None, agg_i32 or None, scalars or None,
        stream or None)


def host_array(xs, ctype=ctypes.c_void_p):
    """A ctypes host array of `xs` (pointers as integers, 0 = NULL; or sizes
    with ctype=c_int64); None stays None and a ctypes array passes through,
    so a caller repeating a call can build its arrays once."""
    if xs is None or isinstance(xs, ctypes.Array):
        return xs
    return (ctype * max(1, len(xs)))(*[(x or None) if ctype is ctypes.c_void_p else x
                                       for x in xs])


def raw_aggregate_adam_multi(grad_ptrs, W, gdtype, T, ns, mode, frac_bits, params, ms, vs,
                             p16s, hp: Optional[AdamWHParams], stream, scalars=0) -> int:
    """Host arrays from Python lists of integers or from `host_array`
    (None = a NULL array)."""
    return lib().disdp_aggregate_adam_multi(
        host_array(grad_ptrs), W, gdtype, T, host_array(ns, ctypes.c_int64), mode, frac_bits,
        host_array(params), host_array(ms), host_array(vs), host_array(p16s),
        None if hp is None else ctypes.byref(hp), scalars or None, stream or None)


# --------------------------------------------------------- torch tensors --
def _torch():
    import torch
    return torch


def _mode(mode) -> int:
    if mode in (AGG_FP32, "fp32"):
        return AGG_FP32
    if mode in (AGG_FIXED, "fixed"):
        return AGG_FIXED
    raise ValueError(f"unknown aggregation mode {mode!r}")


def _grad_dtype(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return DT_F32
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return DT_BF16
    if t.dtype == torch.int32:
        return DT_I32
    raise TypeError(f"unsupported gradient dtype {t.dtype}")


def _dev_ptr(t, name: str, n: int, dtypes) -> int:
    """Pointer of a device tensor, or of a pinned host tensor (which the
    library streams over the host link; it checks the mapping itself)."""
    if t is None:
        return 0
    if not (t.is_cuda or t.is_pinned()):
        raise ValueError(f"{name} must be a device tensor or pinned host memory")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() != n:
        raise ValueError(f"{name} has {t.numel()} elements, expected {n}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}")
    return t.data_ptr()


def _device_index(tensors) -> int:
    """Index of the one GPU the device tensors among `tensors` live on (-1
    when all are pinned host memory); a call never spans devices."""
    idx = -1
    for t in tensors:
        if t is None:
            continue
        d = t.get_device()           # -1 for host tensors
        if d < 0:
            continue
        if idx < 0:
            idx = d
        elif d != idx:
            raise ValueError(f"all device tensors of one call must be on one GPU, got "
                             f"cuda:{idx} and cuda:{d}")
    return idx


_raw_stream = None


def _current_stream_handle(idx: int) -> int:
    """torch's current HIP stream of device `idx`, as a raw handle (the
    C-level query when this torch has it: the public one builds a Stream
    object per call)."""
    global _raw_stream
    if _raw_stream is None:
        torch = _torch()
        _raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None) or \
            (lambda i: torch.cuda.current_stream(i).cuda_stream)
    return _raw_stream(idx)


def _launch(fn, tensors, stream, *args):
    """Call `fn(*args, hip_stream)` with the tensors' GPU current: the
    library launches on the current device.  The stream is the one given,
    else torch's current stream of that device."""
    return _launch_on(_device_index(tensors), stream, fn, *args)


def _launch_on(idx, stream, fn, *args):
    """_launch for tensors known to live on GPU `idx` (-1: none does)."""
    torch = _torch()
    cur = torch.cuda.current_device()
    if idx < 0:
        idx = cur
    s = _current_stream_handle(idx) if stream is None else getattr(stream, "cuda_stream", stream)
    if idx == cur:
        return fn(*args, s)
    with torch.cuda.device(idx):
        return fn(*args, s)


def _hparams(lr, beta1, beta2, eps, weight_decay, step, grad_scale):
    return AdamWHParams(lr, beta1, beta2, eps, weight_decay, int(step),
                        grad_scale)


def _check(status: int, what: str) -> None:
    if status != OK:
        raise DisdpError(status, what)


def _grads(grads):
    torch = _torch()
    grads = list(grads)
    if not grads:
        raise ValueError("at least one contribution is needed")
    n = grads[0].numel()
    gdt = _grad_dtype(grads[0])
    allowed = {DT_F32: (torch.float32,), DT_I32: (torch.int32,)}.get(
        gdt, (torch.bfloat16, torch.int16, torch.uint16))
    ptrs = [_dev_ptr(g, f"grads[{i}]", n, allowed) for i, g in enumerate(grads)]
    return grads, ptrs, gdt, n


def aggregate(grads, *, mode="fp32", frac_bits: int = 0, agg_out_f32=None,
              agg_out_i32=None, stream=None) -> None:
    """W-way reduction of `grads` (float32 or bf16 device tensors of one
    length) into `agg_out_f32` and/or `agg_out_i32` (int32, fixed mode)."""
    torch = _torch()
    grads, ptrs, gdt, n = _grads(grads)
    st = _launch(raw_aggregate, grads + [agg_out_f32, agg_out_i32], stream,
                 ptrs, len(grads), gdt, n, _mode(mode), frac_bits,
                 _dev_ptr(agg_out_f32, "agg_out_f32", n, (torch.float32,)),
                 _dev_ptr(agg_out_i32, "agg_out_i32", n, (torch.int32,)))
    _check(st, "disdp_aggregate")


def adam_step(grad, param, m, v, param_bf16_out=None, *, lr, beta1, beta2,
              eps, weight_decay, step, grad_scale=1.0, stream=None) -> None:
    """One AdamW step on (param, m, v) in place from the fp32 aggregate."""
    torch = _torch()
    n = param.numel()
    f32 = (torch.float32,)
    st = _launch(
        raw_adam_step, [grad, param, m, v, param_bf16_out], stream,
        _dev_ptr(grad, "grad", n, f32), _dev_ptr(param, "param", n, f32),
        _dev_ptr(m, "m", n, f32), _dev_ptr(v, "v", n, f32),
        _dev_ptr(param_bf16_out, "param_bf16_out", n,
                 (torch.bfloat16, torch.int16, torch.uint16)),
        n, _hparams(lr, beta1, beta2, eps, weight_decay, step, grad_scale))
    _check(st, "disdp_adam_step")


def aggregate_adam(grads, param, m, v, param_bf16_out=None, *, lr, beta1,
                   beta2, eps, weight_decay, step, grad_scale=1.0,
                   mode="fp32", frac_bits: int = 0, agg_out_f32=None,
                   agg_out_i32=None, stream=None) -> None:
    """Aggregate `grads` and take one AdamW step, in one pass."""
    torch = _torch()
    grads, ptrs, gdt, n = _grads(grads)
    f32 = (torch.float32,)
    st = _launch(
        raw_aggregate_adam,
        grads + [param, m, v, param_bf16_out, agg_out_f32, agg_out_i32], stream,
        ptrs, len(grads), gdt, n, _mode(mode), frac_bits,
        _dev_ptr(param, "param", n, f32), _dev_ptr(m, "m", n, f32),
        _dev_ptr(v, "v", n, f32),
        _dev_ptr(param_bf16_out, "param_bf16_out", n,
                 (torch.bfloat16, torch.int16, torch.uint16)),
        _dev_ptr(agg_out_f32, "agg_out_f32", n, f32),
        _dev_ptr(agg_out_i32, "agg_out_i32", n, (torch.int32,)),
        _hparams(lr, beta1, beta2, eps, weight_decay, step, grad_scale))
    _check(st, "disdp_aggregate_adam")


def step_scalars(*, lr, beta1, beta2, eps, weight_decay, step, grad_scale=1.0) -> StepScalars:
    """The constants disdp_aggregate_adam derives for this step (host)."""
    out = StepScalars()
    st = lib().disdp_step_scalars(
        ctypes.byref(_hparams(lr, beta1, beta2, eps, weight_decay, step, grad_scale)),
        ctypes.byref(out))
    _check(st, "disdp_step_scalars")
    return out


def aggregate_adam_dev(grads, param, m, v, param_bf16_out=None, *, scalars,
                       mode="fp32", frac_bits: int = 0, agg_out_f32=None,
                       agg_out_i32=None, stream=None) -> None:
    """aggregate_adam with the step constants read when the kernel runs from
    `scalars`: a float32 tensor of 10 elements (a StepScalars image, e.g.
    filled by copying step_scalars(...)), on the device or pinned host
    memory.  Lets one captured HIP graph serve every step."""
    torch = _torch()
    grads, ptrs, gdt, n = _grads(grads)
    f32 = (torch.float32,)
    st = _launch(
        raw_aggregate_adam_dev,
        grads + [param, m, v, param_bf16_out, agg_out_f32, agg_out_i32, scalars], stream,
        ptrs, len(grads), gdt, n, _mode(mode), frac_bits,
        _dev_ptr(param, "param", n, f32), _dev_ptr(m, "m", n, f32),
        _dev_ptr(v, "v", n, f32),
        _dev_ptr(param_bf16_out, "param_bf16_out", n,
                 (torch.bfloat16, torch.int16, torch.uint16)),
        _dev_ptr(agg_out_f32, "agg_out_f32", n, f32),
        _dev_ptr(agg_out_i32, "agg_out_i32", n, (torch.int32,)),
        _dev_ptr(scalars, "scalars", ctypes.sizeof(StepScalars) // 4, f32))
    _check(st, "disdp_aggregate_adam_dev")


class MultiTensorStep:
    """disdp_aggregate_adam_multi over a fixed list of tensors, for a caller
    that steps the same tensors again and again: the tensors are checked
    and their pointers packed into host arrays once, and each call takes
    one step.  `tensors`: a sequence of (grads, param, m, v, param_bf16_out)
    with grads a list of W contributions of that tensor's length and
    param_bf16_out possibly None.  The object keeps the tensors alive."""

    def __init__(self, tensors, *, mode="fp32", frac_bits: int = 0):
        torch = _torch()
        self._tensors = list(tensors)
        self._mode = _mode(mode)
        self._frac_bits = frac_bits
        self.T = len(self._tensors)
        if not self._tensors:
            return
        W = len(self._tensors[0][0])
        gdt = _grad_dtype(self._tensors[0][0][0])
        allowed = {DT_F32: (torch.float32,), DT_I32: (torch.int32,)}.get(
            gdt, (torch.bfloat16, torch.int16, torch.uint16))
        f32 = (torch.float32,)
        p16t = (torch.bfloat16, torch.int16, torch.uint16)
        gp, ns, ps, ms_, vs, cs, every = [], [], [], [], [], [], []
        for j, (grads, p, m, v, c) in enumerate(self._tensors):
            if len(grads) != W:
                raise ValueError(f"tensor {j} has {len(grads)} contributions, expected {W}")
            n = p.numel()
            gp += [_dev_ptr(g, f"tensors[{j}] grads[{w}]", n, allowed)
                   for w, g in enumerate(grads)]
            ns.append(n)
            ps.append(_dev_ptr(p, f"tensors[{j}] param", n, f32))
            ms_.append(_dev_ptr(m, f"tensors[{j}] m", n, f32))
            vs.append(_dev_ptr(v, f"tensors[{j}] v", n, f32))
            cs.append(_dev_ptr(c, f"tensors[{j}] param_bf16_out", n, p16t))
            every += list(grads) + [p, m, v, c]
        self.W = W
        self._gdt = gdt
        self._device = _device_index(every)
        self._arrays = (host_array(gp), host_array(ns, ctypes.c_int64), host_array(ps),
                        host_array(ms_), host_array(vs), host_array(cs) if any(cs) else None)

    def __call__(self, *, lr=None, beta1=None, beta2=None, eps=None, weight_decay=None,
                 step=None, grad_scale=1.0, scalars=None, stream=None) -> None:
        """One step of every tensor: the hyperparameters, or `scalars` (as
        for aggregate_adam_dev) instead."""
        if not self.T:
            return
        hp = None if scalars is not None else \
            _hparams(lr, beta1, beta2, eps, weight_decay, step, grad_scale)
        sc = _dev_ptr(scalars, "scalars", ctypes.sizeof(StepScalars) // 4, (_torch().float32,))
        idx = self._device
        if scalars is not None:
            d = _device_index([scalars])
            if idx >= 0 and d >= 0 and d != idx:
                raise ValueError(f"scalars on cuda:{d}, tensors on cuda:{idx}")
            idx = d if idx < 0 else idx
        gp, ns, ps, ms_, vs, cs = self._arrays
        st = _launch_on(idx, stream, lambda *a: raw_aggregate_adam_multi(
            *a[:-1], stream=a[-1], scalars=sc),
            gp, self.W, self._gdt, self.T, ns, self._mode, self._frac_bits, ps, ms_, vs, cs, hp)
        _check(st, "disdp_aggregate_adam_multi")


def aggregate_adam_multi(tensors, *, lr=None, beta1=None, beta2=None, eps=None,
                         weight_decay=None, step=None, grad_scale=1.0, scalars=None,
                         mode="fp32", frac_bits: int = 0, stream=None) -> None:
    """aggregate_adam over many tensors at once (a batch of tensors per
    launch); the tensors as for MultiTensorStep, which a caller stepping
    the same tensors repeatedly should keep instead.  Every tensor takes
    the same step: the hyperparameters, or `scalars` instead."""
    MultiTensorStep(tensors, mode=mode, frac_bits=frac_bits)(
        lr=lr, beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay, step=step,
        grad_scale=grad_scale, scalars=scalars, stream=stream)


def quantize(grad, out, *, frac_bits: int, stream=None) -> None:
    """out (int32) = the switch's integer format of `grad` (float32 or bf16)
    at scale 2^frac_bits, saturating."""
    torch = _torch()
    n = grad.numel()
    gdt = _grad_dtype(grad)
    if gdt == DT_I32:
        raise TypeError("quantize takes float32 or bf16 input")
    allowed = (torch.float32,) if gdt == DT_F32 else \
        (torch.bfloat16, torch.int16, torch.uint16)
    st = _launch(raw_quantize, [grad, out], stream,
                 _dev_ptr(grad, "grad", n, allowed), gdt, n, frac_bits,
                 _dev_ptr(out, "out", n, (torch.int32,)))
    _check(st, "disdp_quantize")


_GDT = {"f32": DT_F32, "bf16": DT_BF16, "i32": DT_I32}


def shard_layout(n: int, W: int, gdtype="f32", *, bf16_copy=True, agg_f32=False,
                 agg_i32=False):
    """(byte offsets, total bytes) of a shard's arrays in one allocation, as
    disdp_shard_layout places them.  Offsets are listed as contributions
    0..W-1, param, m, v, param_bf16, agg_f32, agg_i32 (-1 = not included)."""
    flags = ((LAYOUT_BF16_COPY if bf16_copy else 0) | (LAYOUT_AGG_F32 if agg_f32 else 0)
             | (LAYOUT_AGG_I32 if agg_i32 else 0))
    offs = (ctypes.c_int64 * (W + 6))()
    total = ctypes.c_int64()
    st = lib().disdp_shard_layout(n, W, _GDT.get(gdtype, gdtype), flags, offs,
                                  ctypes.byref(total))
    _check(st, "disdp_shard_layout")
    return list(offs), total.value


_HIP_DEVICE_MALLOC_CONTIGUOUS = 0x4    # hipDeviceMallocContiguous
_hip = None


def _hip_runtime() -> ctypes.CDLL:
    """torch's HIP runtime: with torch imported, the soname resolves to the
    copy already loaded (the one that owns torch's memory and streams)."""
    global _hip
    if _hip is None:
        _torch()
        L = ctypes.CDLL("libamdhip64.so.7")
        L.hipExtMallocWithFlags.restype = ctypes.c_int
        L.hipExtMallocWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t,
                                            ctypes.c_uint]
        L.hipGetLastError.restype = ctypes.c_int
        L.hipPeekAtLastError.restype = ctypes.c_int
        _hip = L
    return _hip


class _ContiguousBlock:
    """One physically contiguous device allocation (hipExtMallocWithFlags
    with hipDeviceMallocContiguous).  Blocks are never freed while the
    process runs: on MI355X, memory that torch's caching allocator later
    placed in the address range of a freed contiguous block was read back
    stale or zero by kernels that ran after a synchronised copy into it.
    A released block returns to the pool and serves the next request that
    fits."""

    def __init__(self, nbytes: int, device_index: int):
        torch = _torch()
        hip = _hip_runtime()
        ptr = ctypes.c_void_p()
        with torch.cuda.device(device_index):
            pending = hip.hipPeekAtLastError()
            rc = hip.hipExtMallocWithFlags(ctypes.byref(ptr), nbytes,
                                           _HIP_DEVICE_MALLOC_CONTIGUOUS)
        self.ptr = ptr.value or 0
        if rc != 0 or not self.ptr:
            if pending == 0:                # clear the error this call recorded,
                hip.hipGetLastError()       # never one that was already pending
            raise MemoryError(f"no physically contiguous block of {nbytes} bytes "
                              f"(HIP error {rc})")
        self.nbytes = nbytes
        self.device_index = device_index
        self.leased = False


_blocks = []                       # every contiguous block of this process
_blocks_lock = threading.RLock()   # reentrant: a lease may be collected while held


class _Lease:
    """The owner torch holds for a tensor over (a prefix of) one block,
    through __cuda_array_interface__: torch keeps it alive while any view
    exists, and collecting it hands the block back to the pool."""

    def __init__(self, block: _ContiguousBlock, nbytes: int):
        self.block = block
        self.__cuda_array_interface__ = {"shape": (nbytes,), "typestr": "|u1",
                                         "data": (block.ptr, False), "version": 2}

    def __del__(self):
        self.block.leased = False


def _lease_block(nbytes: int, device_index: int):
    """The smallest free pooled block of at least `nbytes` on the device,
    else a new block; None when the runtime has none.  A pooled block is
    handed out again only once the device has finished the work already
    queued on it, from any stream (the wait hipFree would have made)."""
    with _blocks_lock:
        fits = [b for b in _blocks if not b.leased and b.device_index == device_index
                and b.nbytes >= nbytes]
        if fits:
            block = min(fits, key=lambda b: b.nbytes)
            _torch().cuda.synchronize(device_index)
        else:
            try:
                block = _ContiguousBlock(nbytes, device_index)
            except MemoryError:
                return None
            _blocks.append(block)
        block.leased = True
        return block


def contiguous_pool(device="cuda"):
    """(bytes held, bytes leased, largest idle block) of the contiguous-block
    pool on a device."""
    torch = _torch()
    dev = torch.device(device)
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    with _blocks_lock:
        mine = [b for b in _blocks if b.device_index == idx]
        return (sum(b.nbytes for b in mine), sum(b.nbytes for b in mine if b.leased),
                max((b.nbytes for b in mine if not b.leased), default=0))


def contiguous_bytes(nbytes: int, device="cuda"):
    """A uint8 device tensor of `nbytes` over one physically contiguous
    block (pooled for the life of the process, back in the pool when the
    last view goes), or None when the runtime has no such block (or torch
    cannot wrap it)."""
    torch = _torch()
    dev = torch.device(device)
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    block = _lease_block(nbytes, idx)
    if block is None:
        return None
    owner = _Lease(block, nbytes)
    refs = sys.getrefcount(owner)
    try:
        t = torch.as_tensor(owner, device=torch.device("cuda", idx))
    except (TypeError, RuntimeError, ValueError):
        return None                 # the lease goes with `owner`
    # the tensor must hold the lease (which returns the block when collected)
    if sys.getrefcount(owner) <= refs:
        return None
    if t.data_ptr() != block.ptr or t.numel() != nbytes or t.dtype != torch.uint8:
        return None
    return t


CONTIGUOUS_MIN_BYTES = 1 << 30   # smallest shard slab given a contiguous block


class Shard:
    """A shard's arrays as torch views of one device allocation (`slab`):
    grads (W tensors), param, m, v, and when requested param_bf16 (int16
    bits), agg_f32, agg_i32.  Contents are uninitialised.

    With `contiguous` (the default) a slab of at least CONTIGUOUS_MIN_BYTES
    is one physically contiguous block of device memory (`self.contiguous`
    says whether the runtime had one; otherwise, and for smaller slabs,
    torch's caching allocator provides it: a pooled block is kept for the
    life of the process, which only large shards are worth).  On MI355X
    the fused kernel streams such a slab at 6.50-6.56 TB/s in every fresh
    process tried, against 6.34-6.55 for ordinary allocations, whose
    physical pages vary from process to process."""

    def __init__(self, n: int, W: int, gdtype="f32", *, bf16_copy=True, agg_f32=False,
                 agg_i32=False, device="cuda", contiguous=True):
        torch = _torch()
        offs, total = shard_layout(n, W, gdtype, bf16_copy=bf16_copy, agg_f32=agg_f32,
                                   agg_i32=agg_i32)
        slab = contiguous_bytes(total, device) \
            if contiguous and total >= CONTIGUOUS_MIN_BYTES else None
        self.contiguous = slab is not None
        self.slab = slab if slab is not None else \
            torch.empty(total, dtype=torch.uint8, device=device)

        def view(i, dtype, esize):
            if offs[i] < 0:
                return None
            return self.slab[offs[i]: offs[i] + n * esize].view(dtype)

        gt, gsz = {"f32": (torch.float32, 4), "bf16": (torch.int16, 2),
                   "i32": (torch.int32, 4)}[gdtype]
        self.grads = [view(w, gt, gsz) for w in range(W)]
        self.param = view(W, torch.float32, 4)
        self.m = view(W + 1, torch.float32, 4)
        self.v = view(W + 2, torch.float32, 4)
        self.param_bf16 = view(W + 3, torch.int16, 2)
        self.agg_f32 = view(W + 4, torch.float32, 4)
        self.agg_i32 = view(W + 5, torch.int32, 4)


def allocate_shard(n: int, W: int, gdtype="f32", **kw) -> Shard:
    """A Shard of n elements with W contributions of `gdtype` ("f32", "bf16"
    or "i32"), placed by disdp_shard_layout in one physically contiguous
    allocation when the runtime has one; keyword arguments as for Shard."""
    return Shard(n, W, gdtype, **kw)


def algorithmic_bytes_per_element(W: int, grad_bytes: int, adam: bool = True,
                                  bf16_copy: bool = True, agg_f32: bool = False,
                                  agg_i32: bool = False) -> int:
    """Bytes one element moves through HBM in one call, each byte counted
    once: W contributions read; with the optimizer, p, m, v read and written
    (12 + 12) and the bf16 copy written (2); optional aggregates written."""
    b = W * grad_bytes
    if adam:
        b += 24 + (2 if bf16_copy else 0)
    b += (4 if agg_f32 else 0) + (4 if agg_i32 else 0)
    return b
