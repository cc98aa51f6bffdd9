"""The C ABI of libdisdp on the CPU (no GPU, no kernel launch).

Argument checking happens on the host before any HIP call, so every error
path is exercised here with made-up pointer values that are never
dereferenced.  Calls that would pass every check are not made: they would
launch a kernel.
"""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2409_00918_amd as dd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "disdp.h")

pytestmark = pytest.mark.skipif(not os.path.exists(dd.LIB_PATH),
                                reason="libdisdp.so not built")

# fake, well separated, 256-byte aligned "device" addresses
A = [0x10_0000_0000 + k * 0x1_0000_0000 for k in range(80)]
N = 1000
NULL_ARRAY = "null"      # pass a NULL `grads` array


def hp(**kw):
    base = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1,
                step=1, grad_scale=1.0)
    base.update(kw)
    return dd.AdamWHParams(**base)


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(disdp_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_exactly_the_exports():
    assert declared_functions() == sorted(dd.EXPORTS)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", dd.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (disdp_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(dd.lib(), name)


def test_header_compiles_as_c_and_cxx(tmp_path):
    src = tmp_path / "use.c"
    src.write_text('#include "disdp.h"\nint main(void){ disdp_adamw_hparams_t h;'
                   ' (void)h; return (int)DISDP_OK; }\n')
    for compiler, lang in (("gcc", "c"), ("g++", "c++")):
        subprocess.run([compiler, "-x", lang, "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                        "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                        str(src)], check=True)


def test_hparams_struct_layout_matches_c():
    # lr, beta1, beta2, eps, wd: 5 floats; int64 step aligned to 8; float
    assert dd.AdamWHParams.step.offset == 24
    assert dd.AdamWHParams.grad_scale.offset == 32
    assert ctypes.sizeof(dd.AdamWHParams) == 40


def test_status_strings():
    assert dd.status_string(dd.OK) == "ok"
    names = {dd.status_string(s) for s in range(5)}
    assert len(names) == 5
    assert dd.status_string(99) == "unknown status"
    assert dd.status_string(-1) == "unknown status"


# ---------------------------------------------------------------- aggregate --
def agg(ptrs=None, W=4, gdtype=dd.DT_F32, n=N, mode=dd.AGG_FP32, k=24,
        f32=A[70], i32=0):
    if ptrs is None:
        ptrs = A[:W]
    elif ptrs is NULL_ARRAY:
        ptrs = None
    return dd.raw_aggregate(ptrs, W, gdtype, n, mode, k, f32, i32, 0)


@pytest.mark.parametrize("W", [0, -1, 65, 1000])
def test_aggregate_rejects_W_out_of_range(W):
    assert agg(ptrs=A[:4], W=W) == dd.ERR_INVALID_ARG


def test_aggregate_rejects_negative_n():
    assert agg(n=-1) == dd.ERR_INVALID_ARG
    assert agg(n=-(2**62)) == dd.ERR_INVALID_ARG


def test_aggregate_rejects_huge_n():
    assert agg(n=2**60) == dd.ERR_INVALID_ARG


@pytest.mark.parametrize("gdtype", [2, -1, 7])
def test_aggregate_unknown_dtype(gdtype):
    assert agg(gdtype=gdtype) == dd.ERR_UNSUPPORTED


@pytest.mark.parametrize("mode", [2, -1])
def test_aggregate_unknown_mode(mode):
    assert agg(mode=mode) == dd.ERR_UNSUPPORTED


@pytest.mark.parametrize("k", [-1, 31, 64])
def test_aggregate_frac_bits_range_in_fixed_mode(k):
    assert agg(mode=dd.AGG_FIXED, k=k) == dd.ERR_INVALID_ARG


def test_aggregate_int32_output_only_in_fixed_mode():
    assert agg(mode=dd.AGG_FP32, i32=A[71]) == dd.ERR_INVALID_ARG


def test_aggregate_null_pointers():
    assert agg(ptrs=NULL_ARRAY) == dd.ERR_INVALID_ARG
    assert agg(ptrs=[A[0], 0, A[2], A[3]]) == dd.ERR_INVALID_ARG
    assert agg(f32=0) == dd.ERR_INVALID_ARG                       # fp32 mode needs it
    assert agg(mode=dd.AGG_FIXED, f32=0, i32=0) == dd.ERR_INVALID_ARG


def test_aggregate_empty_shard_is_ok_without_pointers():
    assert agg(ptrs=NULL_ARRAY, n=0, f32=0) == dd.OK
    assert dd.raw_aggregate(None, 3, dd.DT_BF16, 0, dd.AGG_FIXED, 24, 0, 0, 0) == dd.OK


def test_aggregate_checks_counts_before_empty_shortcut():
    assert agg(ptrs=NULL_ARRAY, W=0, n=0) == dd.ERR_INVALID_ARG
    assert agg(ptrs=NULL_ARRAY, n=0, gdtype=5) == dd.ERR_UNSUPPORTED


def test_aggregate_output_overlapping_input_is_alias():
    assert agg(f32=A[2]) == dd.ERR_ALIAS
    # partial overlap: output starts inside contribution 1
    assert agg(f32=A[1] + 4 * (N - 1)) == dd.ERR_ALIAS
    # just past the end of contribution 1 is fine for the check (it would launch,
    # so only verify the overlap predicate through a neighbouring violation)
    assert agg(f32=A[1] + 4 * N, mode=dd.AGG_FIXED, i32=A[1] + 4 * N) == dd.ERR_ALIAS


def test_aggregate_two_outputs_overlapping_is_alias():
    assert agg(mode=dd.AGG_FIXED, f32=A[70], i32=A[70]) == dd.ERR_ALIAS
    assert agg(mode=dd.AGG_FIXED, f32=A[70], i32=A[70] + 8) == dd.ERR_ALIAS


def test_aggregate_bf16_spans_are_two_bytes():
    # bf16 contribution of N elements spans 2N bytes: an output starting at
    # byte 2N - 2 overlaps, one at 2N would not
    assert agg(gdtype=dd.DT_BF16, f32=A[0] + 2 * N - 2) == dd.ERR_ALIAS


# ----------------------------------------------------------------- adam step --
def adam(grad=A[0], p=A[1], m=A[2], v=A[3], p16=A[4], n=N, h="default"):
    if h == "default":
        h = hp()
    return dd.raw_adam_step(grad, p, m, v, p16, n, h, 0)


@pytest.mark.parametrize("bad", [
    dict(step=0), dict(step=-5), dict(beta1=1.0), dict(beta1=-0.1),
    dict(beta2=1.0), dict(beta2=float("nan")), dict(beta1=float("nan")),
    dict(eps=-1e-8), dict(eps=float("inf")), dict(eps=float("nan")),
    dict(lr=float("nan")), dict(lr=float("inf")),
    dict(weight_decay=float("inf")), dict(grad_scale=float("nan"))])
def test_adam_rejects_bad_hyperparameters(bad):
    assert adam(h=hp(**bad)) == dd.ERR_INVALID_ARG


def test_adam_rejects_missing_hparams():
    assert adam(h=None) == dd.ERR_INVALID_ARG


def test_adam_checks_hparams_even_for_empty_shard():
    assert adam(n=0, h=hp(step=0)) == dd.ERR_INVALID_ARG
    assert adam(grad=0, p=0, m=0, v=0, p16=0, n=0) == dd.OK


@pytest.mark.parametrize("which", ["grad", "p", "m", "v"])
def test_adam_null_required_pointer(which):
    kw = {which: 0}
    assert adam(**kw) == dd.ERR_INVALID_ARG


@pytest.mark.parametrize("a,b", [("p", "m"), ("p", "v"), ("m", "v"), ("p16", "p"),
                                 ("grad", "p"), ("grad", "m"), ("grad", "v"),
                                 ("grad", "p16")])
def test_adam_aliasing(a, b):
    base = dict(grad=A[0], p=A[1], m=A[2], v=A[3], p16=A[4])
    base[a] = base[b]
    assert adam(**base) == dd.ERR_ALIAS


def test_adam_bf16_copy_overlapping_state_tail():
    # the bf16 copy (2N bytes) starting in the last element of m
    assert adam(p16=A[2] + 4 * (N - 1)) == dd.ERR_ALIAS


# ------------------------------------------------------------------- fused --
def fused(ptrs=None, W=8, gdtype=dd.DT_F32, n=N, mode=dd.AGG_FP32, k=24,
          p=A[70], m=A[71], v=A[72], p16=A[73], f32=0, i32=0, h="default"):
    if ptrs is None:
        ptrs = A[:W]
    elif ptrs is NULL_ARRAY:
        ptrs = None
    if h == "default":
        h = hp()
    return dd.raw_aggregate_adam(ptrs, W, gdtype, n, mode, k, p, m, v, p16,
                                 f32, i32, h, 0)


def test_fused_argument_checks():
    assert fused(W=0) == dd.ERR_INVALID_ARG
    assert fused(W=65, ptrs=A[:65]) == dd.ERR_INVALID_ARG
    assert fused(n=-3) == dd.ERR_INVALID_ARG
    assert fused(gdtype=9) == dd.ERR_UNSUPPORTED
    assert fused(mode=4) == dd.ERR_UNSUPPORTED
    assert fused(mode=dd.AGG_FIXED, k=31) == dd.ERR_INVALID_ARG
    assert fused(h=hp(step=0)) == dd.ERR_INVALID_ARG
    assert fused(h=None) == dd.ERR_INVALID_ARG
    assert fused(i32=A[74]) == dd.ERR_INVALID_ARG        # int32 aggregate in fp32 mode
    assert fused(p=0) == dd.ERR_INVALID_ARG
    assert fused(ptrs=A[:7] + [0]) == dd.ERR_INVALID_ARG
    assert fused(ptrs=NULL_ARRAY, p=0, m=0, v=0, p16=0, n=0) == dd.OK


def test_fused_aliasing():
    assert fused(p=A[3]) == dd.ERR_ALIAS                 # state onto a contribution
    assert fused(p16=A[70]) == dd.ERR_ALIAS              # copy onto the weight
    assert fused(f32=A[71]) == dd.ERR_ALIAS              # aggregate onto m
    assert fused(mode=dd.AGG_FIXED, f32=A[74], i32=A[74]) == dd.ERR_ALIAS
    assert fused(mode=dd.AGG_FIXED, i32=A[5] + 16) == dd.ERR_ALIAS


def test_fused_accepts_repeated_contributions_for_checks():
    # the same contribution buffer twice is legal (inputs may overlap); with
    # a bad step the call still fails on the step, not on aliasing
    assert fused(ptrs=[A[0]] * 8, h=hp(step=0)) == dd.ERR_INVALID_ARG


def test_binding_raises_without_device_tensors():
    torch = pytest.importorskip("torch")
    g = torch.zeros(8)
    with pytest.raises(ValueError):
        dd.aggregate([g, g], agg_out_f32=torch.zeros(8))


def test_library_binds_to_the_same_hip_runtime_as_torch():
    # run in a fresh interpreter: load the library through the binding first,
    # then use torch; exactly one HIP runtime may be mapped
    code = ("import paper_2409_00918_amd as dd; dd.lib(); import torch; "
            "torch.zeros(1); print(len(dd.hip_runtimes_mapped()))")
    out = subprocess.run([__import__("sys").executable, "-c", code], cwd=ROOT,
                         capture_output=True, text=True, check=True).stdout
    assert out.strip().splitlines()[-1] == "1"


# ---------------------------------------------------------------- quantize --
def test_quantize_argument_checks():
    q = lambda g=A[0], dt=dd.DT_F32, n=N, k=24, out=A[1]: dd.raw_quantize(g, dt, n, k, out, 0)
    assert q(n=-1) == dd.ERR_INVALID_ARG
    assert q(dt=dd.DT_I32) == dd.ERR_UNSUPPORTED
    assert q(dt=7) == dd.ERR_UNSUPPORTED
    assert q(k=31) == dd.ERR_INVALID_ARG and q(k=-1) == dd.ERR_INVALID_ARG
    assert q(g=0) == dd.ERR_INVALID_ARG and q(out=0) == dd.ERR_INVALID_ARG
    assert q(g=0, out=0, n=0) == dd.OK
    assert q(out=A[0]) == dd.ERR_ALIAS
    assert q(out=A[0] + 4 * (N - 1)) == dd.ERR_ALIAS
    assert q(dt=dd.DT_BF16, out=A[0] + 2 * N - 2) == dd.ERR_ALIAS


def test_int32_contributions_only_in_fixed_mode():
    assert agg(gdtype=dd.DT_I32, mode=dd.AGG_FP32) == dd.ERR_UNSUPPORTED
    assert fused(gdtype=dd.DT_I32, mode=dd.AGG_FP32) == dd.ERR_UNSUPPORTED
    # in fixed mode the combination passes the enumeration checks (and then
    # fails here only on the planted aliasing, so nothing launches)
    assert agg(gdtype=dd.DT_I32, mode=dd.AGG_FIXED, f32=A[2]) == dd.ERR_ALIAS


# -------------------------------------------------------------- shard layout --
PAGE = 1 << 21


ALIGN = 16 * PAGE          # every array starts on a 32 MiB boundary
GAP = 17 * PAGE            # at least this far past the end of the previous one


@pytest.mark.parametrize("n,W,gdt", [(875_000_000, 8, "f32"), (812_500_000, 16, "bf16"),
                                     (2_734_375_000, 8, "i32"), (1, 1, "f32"), (0, 3, "bf16"),
                                     (3_000_001, 64, "f32"), (64 << 20, 8, "f32")])
@pytest.mark.parametrize("opts", [dict(), dict(bf16_copy=False), dict(agg_f32=True, agg_i32=True)])
def test_shard_layout_places_every_array_on_32MiB_boundaries(n, W, gdt, opts):
    offs, total = dd.shard_layout(n, W, gdt, **opts)
    esize = {"f32": 4, "bf16": 2, "i32": 4}[gdt]
    want = [n * esize] * W + [4 * n] * 3 + [
        2 * n if opts.get("bf16_copy", True) else 0,
        4 * n if opts.get("agg_f32") else 0, 4 * n if opts.get("agg_i32") else 0]
    requested = [True] * (W + 3) + [opts.get("bf16_copy", True), bool(opts.get("agg_f32")),
                                    bool(opts.get("agg_i32"))]
    assert [o >= 0 for o in offs] == requested
    if n == 0:
        assert total == 0 and all(o == 0 for o in offs if o >= 0)
        return
    placed = [(o, sz) for o, sz in zip(offs, want) if o >= 0]
    prev_end = None
    for o, sz in placed:
        assert o % ALIGN == 0
        if prev_end is None:
            assert o == 0
        else:
            # the first 32 MiB boundary at least 17 pages past the previous end
            assert o >= prev_end + GAP and o - ALIGN < prev_end + GAP
        prev_end = o + -(-sz // PAGE) * PAGE
    assert total == prev_end


def test_shard_layout_argument_checks():
    L = dd.lib()
    offs = (ctypes.c_int64 * 70)()
    tot = ctypes.c_int64()
    assert L.disdp_shard_layout(-1, 8, 0, 1, offs, ctypes.byref(tot)) == dd.ERR_INVALID_ARG
    assert L.disdp_shard_layout(10, 0, 0, 1, offs, ctypes.byref(tot)) == dd.ERR_INVALID_ARG
    assert L.disdp_shard_layout(10, 65, 0, 1, offs, ctypes.byref(tot)) == dd.ERR_INVALID_ARG
    assert L.disdp_shard_layout(10, 8, 5, 1, offs, ctypes.byref(tot)) == dd.ERR_UNSUPPORTED
    assert L.disdp_shard_layout(10, 8, 0, 1, None, ctypes.byref(tot)) == dd.ERR_INVALID_ARG
    assert L.disdp_shard_layout(10, 8, 0, 1, offs, None) == dd.ERR_INVALID_ARG


def test_binding_refuses_a_call_spanning_two_gpus():
    """The library launches on one device; the binding checks that every
    device tensor of a call lives on the same GPU (stand-in objects: no GPU
    is touched)."""
    import types
    import paper_2409_00918_amd as dd
    g0 = types.SimpleNamespace(get_device=lambda: 0)
    g1 = types.SimpleNamespace(get_device=lambda: 1)
    host = types.SimpleNamespace(get_device=lambda: -1)
    assert dd._device_index([g0, None, host, g0]) == 0
    assert dd._device_index([host, None]) == -1
    with pytest.raises(ValueError, match="one GPU"):
        dd._device_index([g0, host, g1])


def test_shard_layout_refuses_a_total_beyond_int64():
    """n may be as large as 2^56, but with many contributions the layout's
    total would not fit in int64: refused rather than wrapped."""
    import paper_2409_00918_amd as dd
    with pytest.raises(dd.DisdpError) as ei:
        dd.shard_layout(1 << 56, 64, "f32")
    assert ei.value.status == dd.ERR_INVALID_ARG
    offs, total = dd.shard_layout(1 << 56, 1, "bf16")
    assert 0 < total < 2 ** 63 and offs[1] >= (1 << 57)


# ------------------------------------------------- step scalars in memory --
def test_step_scalars_struct_layout_matches_c():
    assert ctypes.sizeof(dd.StepScalars) == 40
    assert dd.StepScalars.decay.offset == 24
    assert dd.StepScalars.grad_scale.offset == 36


@pytest.mark.parametrize("b1,b2,lr,wd", [(0.9, 0.95, 1e-4, 0.1), (0.9, 0.999, 3e-4, 0.0),
                                         (0.5, 0.5, 1.0, 0.25), (0.0, 0.0, 1e-3, 0.01),
                                         (0.99, 0.9999, 6e-5, 1.0)])
@pytest.mark.parametrize("t", [1, 2, 3, 17, 1000, 10**6, 2**40])
def test_step_scalars_equal_the_oracles(b1, b2, lr, wd, t):
    np = pytest.importorskip("numpy")
    import oracle
    f = np.float32
    got = dd.step_scalars(lr=f(lr), beta1=f(b1), beta2=f(b2), eps=f(1e-8),
                          weight_decay=f(wd), step=t, grad_scale=f(0.5))
    want = oracle.scalars(f(lr), f(b1), f(b2), f(wd), t)
    bits = np.array([got.beta1, got.one_minus_beta1, got.beta2, got.one_minus_beta2,
                     got.bias_correction1, got.bias_correction2, got.decay], dtype=np.float32)
    assert np.array_equal(bits.view(np.uint32), want.view(np.uint32))
    assert (got.lr, got.eps, got.grad_scale) == (f(lr), f(1e-8), f(0.5))


def test_step_scalars_argument_checks():
    out = dd.StepScalars()
    L = dd.lib()
    assert L.disdp_step_scalars(None, ctypes.byref(out)) == dd.ERR_INVALID_ARG
    assert L.disdp_step_scalars(ctypes.byref(hp()), None) == dd.ERR_INVALID_ARG
    assert L.disdp_step_scalars(ctypes.byref(hp(step=0)), ctypes.byref(out)) == dd.ERR_INVALID_ARG
    assert L.disdp_step_scalars(ctypes.byref(hp(beta1=1.0)), ctypes.byref(out)) == \
        dd.ERR_INVALID_ARG
    with pytest.raises(dd.DisdpError):
        dd.step_scalars(lr=1e-4, beta1=0.9, beta2=0.95, eps=-1.0, weight_decay=0.0, step=1)


def fused_dev(ptrs=None, W=8, gdtype=dd.DT_F32, n=N, mode=dd.AGG_FP32, k=24,
              p=A[70], m=A[71], v=A[72], p16=A[73], f32=0, i32=0, s=A[75]):
    if ptrs is None:
        ptrs = A[:W]
    elif ptrs is NULL_ARRAY:
        ptrs = None
    return dd.raw_aggregate_adam_dev(ptrs, W, gdtype, n, mode, k, p, m, v, p16,
                                     f32, i32, s, 0)


def test_fused_dev_argument_checks():
    assert fused_dev(W=0) == dd.ERR_INVALID_ARG
    assert fused_dev(n=-1) == dd.ERR_INVALID_ARG
    assert fused_dev(gdtype=9) == dd.ERR_UNSUPPORTED
    assert fused_dev(mode=dd.AGG_FIXED, k=31) == dd.ERR_INVALID_ARG
    assert fused_dev(i32=A[74]) == dd.ERR_INVALID_ARG    # int32 aggregate in fp32 mode
    assert fused_dev(s=0) == dd.ERR_INVALID_ARG          # no scalars
    assert fused_dev(s=A[75] + 2) == dd.ERR_INVALID_ARG  # misaligned scalars
    assert fused_dev(v=0) == dd.ERR_INVALID_ARG
    assert fused_dev(ptrs=NULL_ARRAY, p=0, m=0, v=0, p16=0, s=0, n=0) == dd.OK


def test_fused_dev_aliasing():
    assert fused_dev(s=A[70] + 4 * (N - 4)) == dd.ERR_ALIAS   # scalars inside the weights
    assert fused_dev(s=A[70] + 4 * N - 36) == dd.ERR_ALIAS    # straddling their end
    assert fused_dev(s=A[73] + 2 * N - 4) == dd.ERR_ALIAS     # end of the bf16 copy
    assert fused_dev(p=A[3]) == dd.ERR_ALIAS
    # scalars overlapping a contribution are legal (both are read only); the
    # call then fails later on the fake, unmapped addresses
    assert fused_dev(s=A[2] + 8) == dd.ERR_INVALID_ARG


# ------------------------------------------------------------ many tensors --
def multi(T=3, W=4, gdtype=dd.DT_F32, ns=None, mode=dd.AGG_FP32, k=24, grads=None,
          params=None, ms=None, vs=None, p16s="default", h="default"):
    """Tensor j's buffers at A[...]-style fake addresses far apart."""
    base = lambda j, i: 0x20_0000_0000 + (j * 16 + i) * 0x1_0000_0000
    ns = [N] * T if ns is None else ns
    grads = [base(j, w) for j in range(T) for w in range(W)] if grads is None else grads
    params = [base(j, 12) for j in range(T)] if params is None else params
    ms = [base(j, 13) for j in range(T)] if ms is None else ms
    vs = [base(j, 14) for j in range(T)] if vs is None else vs
    p16s = [base(j, 15) for j in range(T)] if p16s == "default" else p16s
    h = hp() if h == "default" else h
    return dd.raw_aggregate_adam_multi(grads, W, gdtype, T, ns, mode, k, params, ms, vs, p16s,
                                       h, 0)


def test_multi_argument_checks():
    assert multi(T=-1, ns=[]) == dd.ERR_INVALID_ARG
    assert multi(T=65537, ns=[0] * 65537) == dd.ERR_INVALID_ARG
    assert multi(W=0, grads=[]) == dd.ERR_INVALID_ARG
    assert multi(gdtype=7) == dd.ERR_UNSUPPORTED
    assert multi(gdtype=dd.DT_I32) == dd.ERR_UNSUPPORTED           # int32 only in fixed mode
    assert multi(mode=dd.AGG_FIXED, k=31) == dd.ERR_INVALID_ARG
    assert multi(h=hp(step=0)) == dd.ERR_INVALID_ARG
    assert multi(h=None) == dd.ERR_INVALID_ARG
    assert multi(ns=[N, -1, N]) == dd.ERR_INVALID_ARG
    assert multi(ns=[N, 2**56 + 1, N]) == dd.ERR_INVALID_ARG
    g = [0x20_0000_0000 + i * 0x1_0000_0000 for i in range(12)]
    g[5] = 0
    assert multi(grads=g) == dd.ERR_INVALID_ARG                     # NULL contribution
    assert multi(vs=[0x50_0000_0000, 0, 0x51_0000_0000]) == dd.ERR_INVALID_ARG
    # empty lists and all-empty tensors need no pointers
    assert multi(T=0, ns=[], grads=[], params=[], ms=[], vs=[], p16s=None) == dd.OK
    assert dd.raw_aggregate_adam_multi(None, 4, dd.DT_F32, 2, [0, 0], dd.AGG_FP32, 0, None, None,
                                       None, None, hp(), 0) == dd.OK
    # a NULL entry is fine for an empty tensor; a NULL array is not for a full one
    assert multi(ns=[N, 0, N], vs=[0x50_0000_0000, 0, 0x51_0000_0000]) == dd.ERR_INVALID_ARG  # fake, unmapped


def test_multi_aliasing_across_tensors():
    T, W = 3, 4
    base = lambda j, i: 0x20_0000_0000 + (j * 16 + i) * 0x1_0000_0000
    # tensor 1's weight array inside tensor 2's third contribution
    assert multi(params=[base(0, 12), base(2, 2) + 64, base(2, 12)]) == dd.ERR_ALIAS
    # two tensors sharing one moment array
    assert multi(ms=[base(0, 13), base(0, 13), base(2, 13)]) == dd.ERR_ALIAS
    # a bf16 copy straddling the end of another tensor's v
    assert multi(p16s=[base(0, 15), base(0, 14) + 4 * N - 2, base(2, 15)]) == dd.ERR_ALIAS
    # contributions shared between tensors are legal (read only); the call
    # then fails later, on the fake unmapped addresses
    g = [base(j, w) for j in range(T) for w in range(W)]
    g[4] = g[0]
    assert multi(grads=g) == dd.ERR_INVALID_ARG


def test_multi_takes_exactly_one_source_of_step_constants():
    base = 0x70_0000_0000

    def call(h, sc):
        return dd.raw_aggregate_adam_multi(
            [0x20_0000_0000 + i * 0x1_0000_0000 for i in range(8)], 4, dd.DT_F32, 2, [N, N],
            dd.AGG_FP32, 0, [0x30_0000_0000, 0x31_0000_0000], [0x32_0000_0000, 0x33_0000_0000],
            [0x34_0000_0000, 0x35_0000_0000], None, h, 0, scalars=sc)
    assert call(hp(), base) == dd.ERR_INVALID_ARG        # both
    assert call(None, 0) == dd.ERR_INVALID_ARG           # neither
    assert call(None, base + 2) == dd.ERR_INVALID_ARG    # misaligned
    assert call(None, 0x34_0000_0000 + 8) == dd.ERR_ALIAS  # inside an output
    # a valid combination gets as far as the (fake, unmapped) addresses
    assert call(None, base) == dd.ERR_INVALID_ARG
    assert call(hp(), 0) == dd.ERR_INVALID_ARG


def test_multi_accepts_host_arrays_built_once():
    """host_array packs pointer and size lists once; the raw call takes the
    packed arrays as it takes lists, with the same checks."""
    T, W = 3, 4
    base = lambda j, i: 0x20_0000_0000 + (j * 16 + i) * 0x1_0000_0000
    grads = [base(j, w) for j in range(T) for w in range(W)]
    params = [base(0, 12), base(2, 2) + 64, base(2, 12)]       # tensor 1 inside a contribution
    ms = [base(j, 13) for j in range(T)]
    vs = [base(j, 14) for j in range(T)]
    assert dd.host_array(None) is None
    g = dd.host_array(grads)
    assert dd.host_array(g) is g and [x or 0 for x in g] == grads
    ns = dd.host_array([N] * T, ctypes.c_int64)
    assert list(ns) == [N] * T
    packed = (g, W, dd.DT_F32, T, ns, dd.AGG_FP32, 0, dd.host_array(params), dd.host_array(ms),
              dd.host_array(vs), None, hp(), 0)
    listed = (grads, W, dd.DT_F32, T, [N] * T, dd.AGG_FP32, 0, params, ms, vs, None, hp(), 0)
    assert dd.raw_aggregate_adam_multi(*packed) == dd.ERR_ALIAS
    assert dd.raw_aggregate_adam_multi(*listed) == dd.ERR_ALIAS
    # NULL entries survive packing (0 -> NULL)
    z = dd.host_array([0, base(0, 0)])
    assert z[0] is None and z[1] == base(0, 0)
