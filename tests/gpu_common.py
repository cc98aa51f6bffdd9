"""Shared helpers of the GPU parity tests (not a test module).

Inputs come from ``synth`` (seeded), are uploaded to the device, run through
the C ABI (via the thin binding) and the results are compared element by
element with the CPU oracle run on the same input bits.
"""
import numpy as np

import oracle
import synth

HP = dict(lr=np.float32(1e-4), beta1=np.float32(0.9), beta2=np.float32(0.95),
          eps=np.float32(1e-8), wd=np.float32(0.1))


def torch():
    import torch as _t
    return _t


def to_dev(a: np.ndarray, offset: int = 0):
    """Device copy of `a`; with offset > 0 the tensor starts `offset`
    elements into a larger allocation (an unaligned pointer)."""
    t = torch()
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    src = t.from_numpy(np.ascontiguousarray(a))
    if offset == 0:
        return src.cuda()
    big = t.zeros(a.size + offset + 8, dtype=src.dtype, device="cuda")
    big[offset:offset + a.size].copy_(src)
    return big[offset:offset + a.size]


def to_host(x) -> np.ndarray:
    t = torch()
    a = x.detach().cpu().numpy()
    if x.dtype == t.int16:
        a = a.view(np.uint16)
    return a


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def f32_same(a, b) -> bool:
    """Bit-identical, except that any NaN matches any NaN."""
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    na, nb = np.isnan(a), np.isnan(b)
    return bool(np.array_equal(na, nb) and np.array_equal(bits(a[~na]), bits(b[~nb])))


def bf16_same(a, b) -> bool:
    a = np.asarray(a, np.uint16)
    b = np.asarray(b, np.uint16)
    na = (a & 0x7FFF) > 0x7F80
    nb = (b & 0x7FFF) > 0x7F80
    return bool(np.array_equal(na, nb) and np.array_equal(a[~na], b[~nb]))


def max_rel_err(got, want) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    ok = np.isfinite(want) & np.isfinite(got)
    if not ok.any():
        return 0.0
    d = np.abs(got[ok] - want[ok])
    den = np.abs(want[ok])
    rel = np.where(den > 0, d / np.where(den > 0, den, 1.0), np.where(d > 0, np.inf, 0.0))
    return float(rel.max())


def bf16_ulp_diff(a, b) -> int:
    """Largest distance in bf16 units in the last place between finite
    patterns (ordered as sign-magnitude integers)."""
    def key(h):
        h = np.asarray(h, np.int64)
        return np.where(h & 0x8000, -(h & 0x7FFF), h & 0x7FFF)
    fin = ((np.asarray(a) & 0x7FFF) < 0x7F80) & ((np.asarray(b) & 0x7FFF) < 0x7F80)
    if not fin.any():
        return 0
    return int(np.max(np.abs(key(a)[fin] - key(b)[fin])))


def assert_parity(got: dict, want: dict, label: str) -> None:
    """Bit parity of every output present in both dicts, plus the stated
    tolerances (max relative error 1e-6 for fp32 state, 1 bf16 ulp)."""
    for k in ("agg_i32",):
        if k in want and k in got:
            assert np.array_equal(got[k], want[k]), f"{label}: {k} differs"
    for k in ("agg_f32", "p", "m", "v"):
        if k in want and k in got:
            assert max_rel_err(got[k], want[k]) <= 1e-6, f"{label}: {k} rel err"
            assert f32_same(got[k], want[k]), f"{label}: {k} not bit-identical"
    if "p16" in want and "p16" in got:
        assert bf16_ulp_diff(got["p16"], want["p16"]) <= 1, f"{label}: p16 ulp"
        assert bf16_same(got["p16"], want["p16"]), f"{label}: p16 not bit-identical"


def run_fused_case(W, gdtype, mode, n, t=3, frac_bits=24, offsets=(0, 0),
                   want_agg=True, want_p16=True, seed=0, sigma=1e-4, hp=None):
    """One disdp_aggregate_adam call against the oracle.  offsets[0] shifts
    the contributions, offsets[1] the state and outputs."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    hp = dict(HP if hp is None else hp)
    gs = synth.host_grads(100 + seed, t, W, n, sigma, gdtype=gdtype,
                          outlier_frac=0.01, outlier_scale=100.0)
    p, m, v = synth.host_state(100 + seed, n, mv_sigma=sigma)
    dg = [to_dev(g, offsets[0]) for g in gs]
    dp, dm, dv = (to_dev(x, offsets[1]) for x in (p, m, v))
    d16 = to_dev(np.zeros(n, np.uint16), offsets[1]) if want_p16 else None
    daf = to_dev(np.zeros(n, np.float32), offsets[1]) if want_agg else None
    dai = to_dev(np.zeros(n, np.int32), offsets[1]) if (want_agg and mode == "fixed") else None
    dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                      beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                      step=t, mode=mode, frac_bits=frac_bits, agg_out_f32=daf,
                      agg_out_i32=dai)
    t_.cuda.synchronize()
    got = {"p": to_host(dp), "m": to_host(dm), "v": to_host(dv)}
    if want_p16:
        got["p16"] = to_host(d16)
    if daf is not None:
        got["agg_f32"] = to_host(daf)
    if dai is not None:
        got["agg_i32"] = to_host(dai)
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32,
                        frac_bits=frac_bits, t=t, want_bf16=want_p16,
                        want_agg_f32=want_agg, want_agg_i32=(want_agg and mode == "fixed"),
                        **hp)
    return got, want


def cu_masked_stream(n_cus):
    """A default-priority stream restricted to the first n_cus CUs
    (hipExtStreamCreateWithCUMask on torch's HIP runtime): (torch stream,
    raw handle, runtime library).  A CU-masked stream has a hardware queue
    of its own.  The caller destroys the handle with hipStreamDestroy."""
    import ctypes
    t_ = torch()
    total = t_.cuda.get_device_properties(0).multi_processor_count
    hip = ctypes.CDLL("libamdhip64.so.7")          # torch's runtime, already loaded
    words = (total + 31) // 32
    mask = (ctypes.c_uint32 * words)()
    for cu in range(min(n_cus, total)):
        mask[cu // 32] |= 1 << (cu % 32)
    h = ctypes.c_void_p()
    assert hip.hipExtStreamCreateWithCUMask(ctypes.byref(h), ctypes.c_uint32(words), mask) == 0
    return t_.cuda.ExternalStream(h.value), h, hip


def host_threads() -> int:
    """Host threads a test may use (the CPU share of one GPU: at most 16)."""
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def whole_shard_mismatches(grads, pre, post, *, gdtype, mode, frac_bits, t, hp,
                           chunk=1 << 26, threads=None, label=""):
    """Every element of one fused step against the oracle.

    grads: the W contributions the step read (device tensors); pre: (p, m, v)
    before the step (device copies); post: dict of the step's outputs
    (device tensors) with keys p, m, v, p16 and optionally agg_i32.  The
    shard is read back in chunks of `chunk` elements into pinned host
    buffers; each chunk is split over `threads` host threads, each running
    the C oracle on its piece and counting the elements whose bits differ.
    Returns {output: mismatching elements}, plus "elements"."""
    import time
    from concurrent.futures import ThreadPoolExecutor
    t_ = torch()
    threads = threads or host_threads()
    n = post["p"].numel()
    keys = [k for k in ("p", "m", "v", "p16", "agg_i32") if k in post]
    arrays = {f"g{w}": g for w, g in enumerate(grads)}
    arrays.update({"p0": pre[0], "m0": pre[1], "v0": pre[2]})
    arrays.update(post)
    size = min(chunk, n)
    pin = t_.cuda.is_available()
    host = {k: t_.empty(size, dtype=a.dtype, pin_memory=pin) for k, a in arrays.items()}
    bad = {k: 0 for k in keys}
    oracle_mode = oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32
    W = len(grads)

    def piece(views, lo, hi):
        gs = [views[f"g{w}"][lo:hi] for w in range(W)]
        want = oracle.fused(gs, views["p0"][lo:hi], views["m0"][lo:hi], views["v0"][lo:hi],
                            mode=oracle_mode, frac_bits=frac_bits, t=t,
                            want_agg_i32="agg_i32" in keys, **hp)
        out = {}
        for k in keys:
            g = views[k][lo:hi]
            w_ = want[k]
            if g.dtype == np.float32:
                g, w_ = g.view(np.uint32), w_.view(np.uint32)
            out[k] = int(np.count_nonzero(g != w_))
        return out

    t_copy = t_orc = 0.0
    with ThreadPoolExecutor(max_workers=threads) as pool:
        for s in range(0, n, size):
            e = min(n, s + size)
            c0 = time.perf_counter()
            views = {}
            for k, a in arrays.items():
                h = host[k][:e - s]
                h.copy_(a[s:e])
                x = h.numpy()
                views[k] = x.view(np.uint16) if x.dtype == np.int16 else x
            c1 = time.perf_counter()
            cuts = [(e - s) * j // threads for j in range(threads + 1)]
            for res in pool.map(lambda j: piece(views, cuts[j], cuts[j + 1]), range(threads)):
                for k, c in res.items():
                    bad[k] += c
            c2 = time.perf_counter()
            t_copy += c1 - c0
            t_orc += c2 - c1
    print(f"[wholeshard] {label} {n} elements: read back {t_copy:.1f} s, oracle and "
          f"compare {t_orc:.1f} s on {threads} threads; mismatches {bad}", flush=True)
    bad["elements"] = n
    return bad
