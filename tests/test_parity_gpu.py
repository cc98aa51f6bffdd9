"""GPU parity of libdisdp against the CPU oracle, at sizes the oracle finishes
in seconds: every entry point, both gradient types, both aggregation modes,
compile-time and run-time worker counts, ragged lengths around the tile and
vector boundaries, unaligned pointers, special values, the tiny-shard
workload over 10 steps, and the equivalences the ABI promises.

The bar is bit parity with the oracle (integer aggregates, fp32 state and
the bf16 copy); the stated tolerances (fp32 relative error <= 1e-6, bf16
within 1 ulp) are asserted as well.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import (HP, assert_parity, bits, cu_masked_stream, f32_same, run_fused_case,
                        to_dev, to_host, torch)

pytestmark = pytest.mark.gpu

# lengths: empty-ish, below one vector group, around 4-element groups,
# around one tile (a one-wave block: 64 lanes x 4 elements = 256) and a few
# tiles, around 256-lane tiles (1024), and larger ragged shards spanning
# many tiles
LENGTHS = [1, 2, 3, 4, 5, 7, 8, 9, 63, 255, 256, 257, 511, 513, 1023, 1024, 1025,
           2047, 2048, 2049, 2051, 4099, 65541, 300_007]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import paper_2409_00918_amd as dd
    dd.lib()
    t = torch()
    assert t.cuda.is_available(), "GPU tests need a device"


def _label(**kw):
    return " ".join(f"{k}={v}" for k, v in kw.items())


@pytest.mark.parametrize("W", [1, 2, 3, 4, 8, 16])
@pytest.mark.parametrize("gdtype", ["f32", "bf16"])
@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_sweep_lengths(W, gdtype, mode):
    for i, n in enumerate(LENGTHS):
        got, want = run_fused_case(W, gdtype, mode, n, t=1 + i % 5, seed=i)
        assert_parity(got, want, _label(W=W, gdtype=gdtype, mode=mode, n=n))


# run-time worker counts: whole chunks (8 fp32 / 16 bf16 contributions) and
# every remainder piece of 8, 4, 2 and 1 after them or alone
@pytest.mark.parametrize("W", [5, 9, 10, 11, 13, 14, 15, 17, 23, 27, 31, 32, 33, 47, 63, 64])
@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fixed"),
                                         ("f32", "fixed"), ("bf16", "fp32")])
def test_fused_runtime_worker_counts(W, gdtype, mode):
    for i, n in enumerate([3, 1029, 70_001]):
        got, want = run_fused_case(W, gdtype, mode, n, t=2 + i, seed=50 + i)
        assert_parity(got, want, _label(W=W, gdtype=gdtype, mode=mode, n=n))


@pytest.mark.parametrize("offsets", [(1, 0), (0, 1), (2, 3), (3, 2)])
@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fixed")])
def test_fused_unaligned_pointers(offsets, gdtype, mode):
    for n in (1, 6, 1000, 40_001):
        got, want = run_fused_case(8, gdtype, mode, n, t=4, offsets=offsets, seed=7)
        assert_parity(got, want, _label(offsets=offsets, n=n))


@pytest.mark.parametrize("k", [1, 2, 3, 37, 63, 64, 130, 200, 255])
@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fixed"), ("bf16", "fp32"),
                                         ("f32", "fixed")])
def test_fused_common_misalignment(k, gdtype, mode):
    """Every array starts k elements past a 256-element boundary (a sub-range
    of aligned arrays): the library does the first 256 - k elements one by
    one (block 0 looping over its lanes) and runs the vector kernel on the
    rest.  Lengths shorter than that head included."""
    for n in (1, 2, 3, 4, 5, 26, 27, 28, 63, 64, 65, 125, 126, 127, 192, 193, 255, 256, 257,
              1027, 40_001, 262_147):
        got, want = run_fused_case(8, gdtype, mode, n, t=3, offsets=(k, k), seed=11 + k)
        assert_parity(got, want, _label(k=k, gdtype=gdtype, mode=mode, n=n))


def _offsets(rng, count, two_byte, even):
    """Element offsets in [0, 64) for `count` arrays; with `even`, the
    2-byte arrays (flags in `two_byte`) all get even offsets."""
    o = [int(x) for x in rng.integers(0, 64, count)]
    if even:
        o = [x & ~1 if tb else x for x, tb in zip(o, two_byte)]
    return o


@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fp32"), ("f32", "fixed"),
                                         ("bf16", "fixed")])
def test_fused_unrelated_misalignments(gdtype, mode):
    """Every array at its own element offset: the vector kernels with the
    first output on a 64-element boundary and the other arrays at
    4-byte-aligned addresses (bf16 arrays at offsets of one parity), or the
    element kernel (bf16 arrays of both parities).  Against the oracle over
    lengths from below one group to many tiles with a ragged tail."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(77 if gdtype == "f32" else 78)
    cases = [(1, 1), (3, 5), (8, 63), (8, 64), (5, 1027), (16, 40_001), (8, 262_147), (9, 70_001)]
    for i, (W, n) in enumerate(cases):
        for even in (True, False):
            bf = gdtype == "bf16"
            # contributions, p, m, v, bf16 copy, fp32 aggregate, int32 aggregate
            two = [bf] * W + [False, False, False, True, False, False]
            o = _offsets(rng, W + 6, two, even)
            gs = synth.host_grads(700 + i, 1, W, n, 1e-4, gdtype=gdtype,
                                  outlier_frac=0.01, outlier_scale=100.0)
            p, m, v = synth.host_state(700 + i, n, mv_sigma=1e-4)
            dg = [to_dev(g, o[w]) for w, g in enumerate(gs)]
            dp, dm, dv = to_dev(p, o[W]), to_dev(m, o[W + 1]), to_dev(v, o[W + 2])
            d16 = to_dev(np.zeros(n, np.uint16), o[W + 3])
            daf = to_dev(np.zeros(n, np.float32), o[W + 4])
            dai = to_dev(np.zeros(n, np.int32), o[W + 5]) if mode == "fixed" else None
            dd.aggregate_adam(dg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"],
                              beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                              step=2, mode=mode, frac_bits=24, agg_out_f32=daf,
                              agg_out_i32=dai)
            t_.cuda.synchronize()
            want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed"
                                else oracle.AGG_FP32, frac_bits=24, t=2,
                                want_agg_f32=True, want_agg_i32=mode == "fixed", **HP)
            got = {"p": to_host(dp), "m": to_host(dm), "v": to_host(dv),
                   "p16": to_host(d16), "agg_f32": to_host(daf)}
            if dai is not None:
                got["agg_i32"] = to_host(dai)
            assert_parity(got, want, _label(W=W, n=n, offsets=o))


def test_aggregate_adam_step_and_quantize_unrelated_misalignments():
    """The same for the single-purpose calls: disdp_aggregate (the first
    output is the fp32 or the int32 aggregate), disdp_adam_step and
    disdp_quantize, each array at its own offset."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(79)
    for i, n in enumerate([2, 255, 4099, 70_001]):
        for gdtype in ("f32", "bf16"):
            W = 5
            two = [gdtype == "bf16"] * W + [False, False]
            o = _offsets(rng, W + 2, two, True)
            gs = synth.host_grads(720 + i, 1, W, n, 1e-4, gdtype=gdtype,
                                  outlier_frac=0.01, outlier_scale=100.0)
            dg = [to_dev(g, o[w]) for w, g in enumerate(gs)]
            ai = to_dev(np.zeros(n, np.int32), o[W])
            af = to_dev(np.zeros(n, np.float32), o[W + 1])
            dd.aggregate(dg, mode="fixed", frac_bits=24, agg_out_i32=ai)
            dd.aggregate(dg, mode="fp32", agg_out_f32=af)
            t_.cuda.synchronize()
            lab = _label(n=n, gdtype=gdtype, offsets=o)
            assert np.array_equal(to_host(ai), oracle.aggregate_fixed(gs, 24)[0]), lab
            assert f32_same(to_host(af), oracle.aggregate_f32(gs)), lab
            q = to_dev(np.zeros(n, np.int32), (o[0] + 7) % 64)
            dd.quantize(dg[1], q, frac_bits=20)
            t_.cuda.synchronize()
            assert np.array_equal(to_host(q), oracle.quantize_array(gs[1], 20)), lab
        p, m, v = synth.host_state(730 + i, n, mv_sigma=1e-4)
        o = _offsets(rng, 5, [False, False, False, False, True], True)
        agg = oracle.aggregate_f32(synth.host_grads(731 + i, 1, 2, n, 1e-4))
        dagg = to_dev(agg, o[0])
        dp, dm, dv = to_dev(p, o[1]), to_dev(m, o[2]), to_dev(v, o[3])
        d16 = to_dev(np.zeros(n, np.uint16), o[4])
        dd.adam_step(dagg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                     eps=HP["eps"], weight_decay=HP["wd"], step=3)
        t_.cuda.synchronize()
        p1, m1, v1, p16 = oracle.adamw(agg, p, m, v, t=3, **HP)
        assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16)},
                      {"p": p1, "m": m1, "v": v1, "p16": p16}, f"adam_step n={n} offsets={o}")


@pytest.mark.parametrize("k", [1, 2, 3, 50, 130])
def test_aggregate_and_adam_step_common_misalignment(k):
    import paper_2409_00918_amd as dd
    t_ = torch()
    for n in (2, 7, 70_001):
        gs = synth.host_grads(360 + k, 1, 5, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
        dg = [to_dev(g, k) for g in gs]
        af = to_dev(np.zeros(n, np.float32), k)
        ai = to_dev(np.zeros(n, np.int32), k)
        dd.aggregate(dg, mode="fixed", frac_bits=24, agg_out_f32=af, agg_out_i32=ai)
        t_.cuda.synchronize()
        want_i, want_f = oracle.aggregate_fixed(gs, 24)
        assert np.array_equal(to_host(ai), want_i), (k, n)
        assert f32_same(to_host(af), want_f), (k, n)
        dd.aggregate(dg, mode="fp32", agg_out_f32=af)
        t_.cuda.synchronize()
        assert f32_same(to_host(af), oracle.aggregate_f32(gs)), (k, n)
        p, m, v = synth.host_state(360 + k, n, mv_sigma=1e-4)
        dp, dm, dv = to_dev(p, k), to_dev(m, k), to_dev(v, k)
        d16 = to_dev(np.zeros(n, np.uint16), k)
        dd.adam_step(af, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                     eps=HP["eps"], weight_decay=HP["wd"], step=2)
        t_.cuda.synchronize()
        p1, m1, v1, p16 = oracle.adamw(oracle.aggregate_f32(gs), p, m, v, t=2, **HP)
        assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16)},
                      {"p": p1, "m": m1, "v": v1, "p16": p16}, f"adam_step k={k} n={n}")


@pytest.mark.parametrize("want_agg,want_p16", [(False, False), (True, False), (False, True)])
def test_fused_optional_outputs(want_agg, want_p16):
    for mode in ("fp32", "fixed"):
        got, want = run_fused_case(4, "f32", mode, 10_007, t=5, want_agg=want_agg,
                                   want_p16=want_p16, seed=3)
        assert_parity(got, want, _label(mode=mode))


@pytest.mark.parametrize("frac_bits", [0, 8, 16, 30])
def test_fused_fixed_scales(frac_bits):
    # at 2^30 a 1e-4 * 100 outlier reaches ~1e8, and contributions of 3e1
    # saturate; at 2^0 most contributions quantise to 0
    got, want = run_fused_case(8, "f32", "fixed", 50_001, t=2, frac_bits=frac_bits,
                               sigma=3.0 if frac_bits == 30 else 1e-4, seed=9)
    assert_parity(got, want, _label(frac_bits=frac_bits))


def test_fused_hyperparameter_variants():
    variants = [dict(HP, lr=np.float32(3e-4)), dict(HP, wd=np.float32(0.0)),
                dict(HP, beta1=np.float32(0.0), beta2=np.float32(0.0)),
                dict(HP, beta2=np.float32(0.999), eps=np.float32(1e-6)),
                dict(HP, eps=np.float32(0.0))]
    for i, hp in enumerate(variants):
        for t in (1, 7, 1000):
            got, want = run_fused_case(3, "bf16", "fp32", 5003, t=t, hp=hp, seed=20 + i)
            assert_parity(got, want, _label(variant=i, t=t))


# ------------------------------------------------------------- special values --
def _special_contributions(n, W):
    rng = np.random.default_rng(5)
    pool = np.array([0.0, -0.0, 1e-45, -1e-45, 1e-40, -3e-39, 1.1754942e-38, 5e-8,
                     -5e-8, 2.0**-25, 3 * 2.0**-25, 1e3, -1e3, 65504.0, 3e38, -3e38,
                     np.inf, -np.inf, np.nan, 127.99999, -128.0, 128.0],
                    dtype=np.float32)
    return [pool[rng.integers(0, pool.size, n)] for _ in range(W)]


@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_special_values(mode):
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 4099, 4
    gs = _special_contributions(n, W)
    p, m, v = synth.host_state(77, n, mv_sigma=1e-3)
    p[:50] = np.float32(1e-42)          # denormal weights
    m[50:100] = np.float32(-1e-41)
    v[100:150] = np.float32(1e-44)      # denormal second moments
    dg = [to_dev(g) for g in gs]
    dp, dm, dv = to_dev(p), to_dev(m), to_dev(v)
    d16 = to_dev(np.zeros(n, np.uint16))
    daf = to_dev(np.zeros(n, np.float32))
    dai = to_dev(np.zeros(n, np.int32)) if mode == "fixed" else None
    dd.aggregate_adam(dg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"],
                      beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                      step=3, mode=mode, frac_bits=24, agg_out_f32=daf, agg_out_i32=dai)
    t_.cuda.synchronize()
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32,
                        frac_bits=24, t=3, want_agg_f32=True,
                        want_agg_i32=(mode == "fixed"), **HP)
    got = {"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16),
           "agg_f32": to_host(daf)}
    if dai is not None:
        got["agg_i32"] = to_host(dai)
    assert_parity(got, want, f"special values, {mode}")


def test_adam_step_division_and_sqrt_across_magnitudes():
    # gradients spread over the whole fp32 range (incl. denormals) stress the
    # correctly rounded divide and square root
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(123)
    n = 200_003
    e = rng.integers(-149, 60, n).astype(np.float64)
    g = (rng.choice([-1.0, 1.0], n) * rng.uniform(1, 2, n) * 2.0**e).astype(np.float32)
    p = rng.standard_normal(n).astype(np.float32)
    m = (rng.standard_normal(n) * 2.0**rng.integers(-140, 30, n)).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 2.0**rng.integers(-149, 60, n)).astype(np.float32)
    for t in (1, 2, 17):
        dg, dp, dm, dv = to_dev(g), to_dev(p), to_dev(m), to_dev(v)
        d16 = to_dev(np.zeros(n, np.uint16))
        dd.adam_step(dg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                     eps=HP["eps"], weight_decay=HP["wd"], step=t)
        t_.cuda.synchronize()
        p1, m1, v1, p16 = oracle.adamw(g, p, m, v, t=t, **HP)
        assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16)},
                      {"p": p1, "m": m1, "v": v1, "p16": p16}, f"t={t}")


# ----------------------------------------------------------- the three calls --
@pytest.mark.parametrize("W,gdtype,mode", [(8, "f32", "fp32"), (16, "bf16", "fp32"),
                                           (8, "f32", "fixed"), (5, "bf16", "fixed"),
                                           (1, "f32", "fp32"), (27, "bf16", "fp32"),
                                           (31, "f32", "fixed"), (40, "bf16", "fixed")])
def test_aggregate_matches_oracle(W, gdtype, mode):
    import paper_2409_00918_amd as dd
    t_ = torch()
    for n in (1, 5, 1027, 123_457):
        gs = synth.host_grads(300 + W, 1, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                              outlier_scale=1e4)
        dg = [to_dev(g) for g in gs]
        daf = to_dev(np.zeros(n, np.float32))
        dai = to_dev(np.zeros(n, np.int32)) if mode == "fixed" else None
        dd.aggregate(dg, mode=mode, frac_bits=24, agg_out_f32=daf, agg_out_i32=dai)
        t_.cuda.synchronize()
        if mode == "fixed":
            ai, af = oracle.aggregate_fixed(gs, 24)
            assert np.array_equal(to_host(dai), ai), n
        else:
            af = oracle.aggregate_f32(gs)
        assert f32_same(to_host(daf), af), n


def test_aggregate_fixed_int_only_output():
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 9001
    gs = synth.host_grads(310, 0, 3, n, 1e-4)
    dai = to_dev(np.zeros(n, np.int32))
    dd.aggregate([to_dev(g) for g in gs], mode="fixed", frac_bits=20, agg_out_i32=dai)
    t_.cuda.synchronize()
    assert np.array_equal(to_host(dai), oracle.aggregate_fixed(gs, 20)[0])


def test_aggregate_fixed_is_worker_order_independent_on_device():
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 33_333, 8
    gs = synth.host_grads(311, 0, W, n, 1e-3, outlier_frac=0.05, outlier_scale=1e6)
    dg = [to_dev(g) for g in gs]
    outs = []
    for perm in (list(range(W)), list(reversed(range(W))), [3, 1, 7, 0, 2, 6, 4, 5]):
        dai = to_dev(np.zeros(n, np.int32))
        daf = to_dev(np.zeros(n, np.float32))
        dd.aggregate([dg[j] for j in perm], mode="fixed", frac_bits=24,
                     agg_out_f32=daf, agg_out_i32=dai)
        t_.cuda.synchronize()
        outs.append((to_host(dai), bits(to_host(daf))))
    for o in outs[1:]:
        assert np.array_equal(o[0], outs[0][0]) and np.array_equal(o[1], outs[0][1])


def test_adam_step_matches_oracle():
    import paper_2409_00918_amd as dd
    t_ = torch()
    for n in (1, 3, 4, 1025, 250_001):
        g = synth.host_grads(320, 0, 1, n, 1e-3, outlier_frac=0.01, outlier_scale=100.0)[0]
        p, m, v = synth.host_state(320, n, mv_sigma=1e-3)
        dg, dp, dm, dv = to_dev(g), to_dev(p), to_dev(m), to_dev(v)
        d16 = to_dev(np.zeros(n, np.uint16))
        dd.adam_step(dg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                     eps=HP["eps"], weight_decay=HP["wd"], step=6)
        t_.cuda.synchronize()
        p1, m1, v1, p16 = oracle.adamw(g, p, m, v, t=6, **HP)
        assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16)},
                      {"p": p1, "m": m1, "v": v1, "p16": p16}, f"n={n}")


@pytest.mark.parametrize("W,gdtype,mode", [(8, "f32", "fp32"), (16, "bf16", "fp32"),
                                           (8, "f32", "fixed"), (7, "bf16", "fixed")])
def test_fused_equals_aggregate_then_adam_step(W, gdtype, mode):
    """The ABI promise: the fused call is bit-identical to the two-call path."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 100_003
    gs = synth.host_grads(330, 0, W, n, 1e-4, gdtype=gdtype)
    p, m, v = synth.host_state(330, n, mv_sigma=1e-4)
    dg = [to_dev(g) for g in gs]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=3)
    a = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    dd.aggregate_adam(dg, *a, mode=mode, frac_bits=24, **kw)
    b = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    agg = to_dev(np.zeros(n, np.float32))
    dd.aggregate(dg, mode=mode, frac_bits=24, agg_out_f32=agg)
    dd.adam_step(agg, *b, **kw)
    t_.cuda.synchronize()
    for x, y in zip(a, b):
        assert np.array_equal(to_host(x), to_host(y))


@pytest.mark.parametrize("W,gdtype,mode", [(8, "f32", "fp32"), (16, "bf16", "fixed"),
                                            (5, "f32", "fp32")])
def test_chunked_calls_equal_one_call(W, gdtype, mode):
    """Each element's result depends only on that element: the shard done in
    one call equals the shard done as several calls on sub-ranges, whatever
    the grid of each call and whether a sub-range starts on a vector
    boundary (aligned chunks take the vector kernel, the others the element
    kernel)."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 3 * 262_144 + 4_099
    gs = synth.host_grads(335, 2, W, n, 1e-4, gdtype=gdtype,
                          outlier_frac=0.01, outlier_scale=100.0)
    p, m, v = synth.host_state(335, n, mv_sigma=1e-4)
    dg = [to_dev(g) for g in gs]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=2, mode=mode, frac_bits=24)
    ai_whole = t_.zeros(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
    whole = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    dd.aggregate_adam(dg, *whole, agg_out_i32=ai_whole, **kw)
    # cuts: one tile, a few groups, an odd element count, then the rest
    cuts = [0, 1024, 1024 + 12, 1024 + 12 + 7, 262_144 + 5, n]
    ai_parts = t_.zeros(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
    parts = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    for lo, hi in zip(cuts[:-1], cuts[1:]):
        dd.aggregate_adam([g[lo:hi] for g in dg], *(x[lo:hi] for x in parts),
                          agg_out_i32=None if ai_parts is None else ai_parts[lo:hi], **kw)
    t_.cuda.synchronize()
    for x, y in zip(whole, parts):
        assert np.array_equal(to_host(x), to_host(y))
    if mode == "fixed":
        assert np.array_equal(to_host(ai_whole), to_host(ai_parts))


def test_empty_shard_writes_nothing():
    import paper_2409_00918_amd as dd
    t_ = torch()
    e = t_.empty(0, device="cuda")
    dd.aggregate([e, e], agg_out_f32=e)
    dd.adam_step(e, t_.empty(0, device="cuda"), t_.empty(0, device="cuda"),
                 t_.empty(0, device="cuda"), lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8,
                 weight_decay=0.1, step=1)
    t_.cuda.synchronize()


def test_errors_are_raised_by_the_binding_on_device():
    import paper_2409_00918_amd as dd
    t_ = torch()
    x = t_.zeros(16, device="cuda")
    with pytest.raises(dd.DisdpError) as ei:
        dd.aggregate([x, x], agg_out_f32=x)          # output is an input
    assert ei.value.status == dd.ERR_ALIAS
    with pytest.raises(dd.DisdpError) as ei:
        dd.adam_step(t_.zeros(16, device="cuda"), x, t_.zeros(16, device="cuda"),
                     t_.zeros(16, device="cuda"), lr=1e-4, beta1=1.0, beta2=0.95,
                     eps=1e-8, weight_decay=0.1, step=1)
    assert ei.value.status == dd.ERR_INVALID_ARG


# --------------------------------------------------------- streams and state --
def test_side_stream_and_determinism():
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 1_000_003, 8
    gs = synth.host_grads(340, 0, W, n, 1e-4)
    p, m, v = synth.host_state(340, n, mv_sigma=1e-4)
    dg = [to_dev(g) for g in gs]
    res = []
    s = t_.cuda.Stream()
    for use_side in (False, True):
        st = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
        t_.cuda.synchronize()
        if use_side:
            with t_.cuda.stream(s):
                dd.aggregate_adam(dg, *st, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                                  eps=HP["eps"], weight_decay=HP["wd"], step=2)
            s.synchronize()
        else:
            dd.aggregate_adam(dg, *st, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                              eps=HP["eps"], weight_decay=HP["wd"], step=2)
            t_.cuda.synchronize()
        res.append([to_host(x) for x in st])
    for x, y in zip(*res):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_call_captured_in_a_hip_graph(mode):
    """The entry points enqueue only kernel launches (no allocation, memset
    or synchronisation), so a caller can capture them in a HIP graph.  The
    step's hyperparameters are kernel arguments fixed at capture.  Each of
    three replays, with eager work and synchronisations between them, must
    equal the same call made eagerly on a copy of the state."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 1_000_003, 4
    gs = synth.host_grads(345, 0, W, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
    p, m, v = synth.host_state(345, n, mv_sigma=1e-4)
    dg = [to_dev(g) for g in gs]
    cap = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    ref = [x.clone() for x in cap]
    agg_cap = t_.zeros(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
    agg_ref = t_.zeros(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=4, mode=mode, frac_bits=24)
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    graph = t_.cuda.CUDAGraph()
    with t_.cuda.graph(graph, stream=side):
        dd.aggregate_adam(dg, *cap, agg_out_i32=agg_cap, **kw)
    t_.cuda.synchronize()
    # capture records the launch without running it
    assert all(t_.equal(a, b) for a, b in zip(cap, ref))
    other = t_.zeros(1 << 20, device="cuda")
    for r in range(3):
        graph.replay()
        dd.aggregate_adam(dg, *ref, agg_out_i32=agg_ref, **kw)
        t_.cuda.synchronize()
        other.add_(1.0)                       # unrelated eager work between replays
        t_.cuda.synchronize()
        for a, b in zip(cap, ref):
            assert t_.equal(a, b), f"replay {r}"
        if mode == "fixed":
            assert t_.equal(agg_cap, agg_ref), f"replay {r}: agg_i32"
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32,
                        frac_bits=24, t=4, **HP)
    # the first replay is one step from the initial state: check it against
    # the oracle through a fresh eager call from the same start
    fresh = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    dd.aggregate_adam(dg, *fresh, **kw)
    t_.cuda.synchronize()
    assert_parity({"p": to_host(fresh[0]), "m": to_host(fresh[1]), "v": to_host(fresh[2]),
                   "p16": to_host(fresh[3])}, want, f"graph {mode}")
    del graph


def _scalars_tensor(**kw):
    """The StepScalars image of one step as 10 float32 values (host)."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    return t_.frombuffer(bytearray(dd.step_scalars(**kw)), dtype=t_.float32).clone()


@pytest.mark.parametrize("gdtype", ["f32", "bf16"])
@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_dev_equals_fused(gdtype, mode):
    """disdp_aggregate_adam_dev, with the step's constants in device memory
    and in pinned host memory, gives the bits of disdp_aggregate_adam with
    the same hyperparameters, over ragged lengths, steps and settings."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    settings = [dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
                     weight_decay=HP["wd"], step=1),
                dict(lr=np.float32(3e-3), beta1=np.float32(0.8), beta2=np.float32(0.999),
                     eps=np.float32(1e-6), weight_decay=np.float32(0.0), step=7,
                     grad_scale=np.float32(0.125)),
                dict(lr=np.float32(1e-5), beta1=np.float32(0.9), beta2=np.float32(0.95),
                     eps=np.float32(1e-8), weight_decay=np.float32(1.0), step=123_456)]
    for i, n in enumerate([1, 5, 257, 4099, 300_007]):
        for j, kw in enumerate(settings):
            W = (3, 8, 5)[j]
            gs = synth.host_grads(900 + i, j, W, n, 1e-4, gdtype=gdtype,
                                  outlier_frac=0.01, outlier_scale=100.0)
            p, m, v = synth.host_state(900 + i, n, mv_sigma=1e-4)
            dg = [to_dev(g) for g in gs]
            ref = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
            dd.aggregate_adam(dg, *ref, mode=mode, frac_bits=20, **kw)
            for where in ("device", "pinned"):
                sc = _scalars_tensor(**kw)
                sc = sc.cuda() if where == "device" else sc.pin_memory()
                got = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
                dd.aggregate_adam_dev(dg, *got, scalars=sc, mode=mode, frac_bits=20)
                t_.cuda.synchronize()
                for a, b in zip(got, ref):
                    assert t_.equal(a, b), _label(n=n, setting=j, where=where)
            if n == 4099:
                want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed"
                                    else oracle.AGG_FP32, frac_bits=20, t=kw["step"],
                                    lr=kw["lr"], beta1=kw["beta1"], beta2=kw["beta2"],
                                    eps=kw["eps"], wd=kw["weight_decay"],
                                    grad_scale=kw.get("grad_scale", np.float32(1.0)))
                assert_parity({"p": to_host(ref[0]), "m": to_host(ref[1]),
                               "v": to_host(ref[2]), "p16": to_host(ref[3])}, want,
                              _label(n=n, setting=j))


@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_one_hip_graph_serves_every_optimizer_step(mode):
    """One capture, six optimizer steps: the graph holds a copy node that
    refreshes the step's constants in device memory from pinned host memory
    (rewritten before each replay) and the disdp_aggregate_adam_dev launch.
    Fresh contributions are written into the captured buffers between
    replays, with unrelated eager work and synchronisations in between; each
    step must equal the oracle's step t bit for bit."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 300_007, 4
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"])
    p, m, v = synth.host_state(910, n, mv_sigma=1e-4)
    dg = [t_.zeros(n, device="cuda") for _ in range(W)]
    st = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    agg = t_.zeros(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
    host = t_.zeros(10, dtype=t_.float32, pin_memory=True)
    dev = t_.zeros(10, dtype=t_.float32, device="cuda")
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    graph = t_.cuda.CUDAGraph()
    with t_.cuda.graph(graph, stream=side):
        dev.copy_(host, non_blocking=True)
        dd.aggregate_adam_dev(dg, *st, scalars=dev, mode=mode, frac_bits=24,
                              agg_out_i32=agg)
    t_.cuda.synchronize()
    assert t_.equal(st[0].cpu(), t_.from_numpy(p))     # capture ran nothing
    other = t_.zeros(1 << 20, device="cuda")
    for t in range(1, 7):
        gs = synth.host_grads(910, t, W, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
        for d, g in zip(dg, gs):
            d.copy_(t_.from_numpy(g))
        host.copy_(_scalars_tensor(step=t, **kw))
        t_.cuda.synchronize()
        graph.replay()
        t_.cuda.synchronize()
        other.add_(1.0)
        t_.cuda.synchronize()
        want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed"
                            else oracle.AGG_FP32, frac_bits=24, t=t,
                            want_agg_i32=mode == "fixed", **HP)
        assert_parity({"p": to_host(st[0]), "m": to_host(st[1]), "v": to_host(st[2]),
                       "p16": to_host(st[3])}, want, f"graph step {t} {mode}")
        if mode == "fixed":
            assert np.array_equal(to_host(agg), want["agg_i32"]), f"step {t} agg_i32"
        p, m, v = want["p"], want["m"], want["v"]
    del graph



@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_on_cu_masked_streams(mode):
    """On a CU-masked stream the library raises its per-CU occupancy cap
    (a different launch configuration); results stay identical to the
    default stream's and to the oracle."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 2_000_003, 8
    gs = synth.host_grads(346, 0, W, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
    p, m, v = synth.host_state(346, n, mv_sigma=1e-4)
    dg = [to_dev(g) for g in gs]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=2, mode=mode, frac_bits=24)
    base = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    dd.aggregate_adam(dg, *base, **kw)
    t_.cuda.synchronize()
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32,
                        frac_bits=24, t=2, **HP)
    assert_parity({"p": to_host(base[0]), "m": to_host(base[1]), "v": to_host(base[2]),
                   "p16": to_host(base[3])}, want, f"default stream {mode}")
    for n_cus in (32, 200):
        s, h, hip = cu_masked_stream(n_cus)
        try:
            st = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
            t_.cuda.synchronize()
            dd.aggregate_adam(dg, *st, stream=s, **kw)
            s.synchronize()
            for a, b in zip(base, st):
                assert t_.equal(a, b), f"{n_cus} CUs, {mode}"
        finally:
            t_.cuda.synchronize()
            hip.hipStreamDestroy(h)


def test_concurrent_calls_from_two_threads():
    """The library keeps no per-call state and is re-entrant: two host
    threads (the ctypes calls release the interpreter lock) each enqueue 12
    steps on their own stream and shard at the same time, with different
    worker counts, modes and sizes; every result equals the same steps run
    alone, one thread after the other."""
    import threading
    import paper_2409_00918_amd as dd
    t_ = torch()
    cases = [(8, "f32", "fp32", 1_000_003), (5, "bf16", "fixed", 777_777)]
    inputs = []
    for i, (W, gdtype, mode, n) in enumerate(cases):
        gs = synth.host_grads(350 + i, 0, W, n, 1e-4, gdtype=gdtype)
        p, m, v = synth.host_state(350 + i, n, mv_sigma=1e-4)
        inputs.append(([to_dev(g) for g in gs], (p, m, v)))

    def run(i, state, stream, barrier=None):
        W, gdtype, mode, n = cases[i]
        dg = inputs[i][0]
        if barrier is not None:
            barrier.wait()
        with t_.cuda.stream(stream):
            for step in range(1, 13):
                dd.aggregate_adam(dg, *state, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                                  eps=HP["eps"], weight_decay=HP["wd"], step=step, mode=mode,
                                  frac_bits=24)
        stream.synchronize()

    def fresh(i):
        n = cases[i][3]
        return [to_dev(x) for x in inputs[i][1]] + [to_dev(np.zeros(n, np.uint16))]

    streams = [t_.cuda.Stream(), t_.cuda.Stream()]
    alone = []
    for i in range(2):
        st = fresh(i)
        t_.cuda.synchronize()
        run(i, st, streams[i])
        alone.append(st)
    together = [fresh(0), fresh(1)]
    t_.cuda.synchronize()
    barrier = threading.Barrier(2)
    errors = []

    def worker(i):
        try:
            run(i, together[i], streams[i], barrier)
        except Exception as e:          # reported below, in the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    assert not any(th.is_alive() for th in threads)
    t_.cuda.synchronize()
    for i in range(2):
        for a, b in zip(alone[i], together[i]):
            assert t_.equal(a, b), f"case {i}"


def test_resume_from_saved_state_is_bit_identical():
    """5 steps straight equal 2 steps, a save/restore of (p, m, v, t), and 3
    more steps: all optimizer state is the caller's."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 20_011, 4
    p, m, v = synth.host_state(350, n)
    grads = [[to_dev(g) for g in synth.host_grads(350, t, W, n, 1e-3)] for t in range(1, 6)]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"])

    def steps(state, ts):
        for t in ts:
            dd.aggregate_adam(grads[t - 1], *state, step=t, **kw)
        t_.cuda.synchronize()

    a = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    steps(a, range(1, 6))
    b = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    steps(b, range(1, 3))
    saved = [to_host(x) for x in b]
    c = [to_dev(x) for x in saved]
    steps(c, range(3, 6))
    for x, y in zip(a, c):
        assert np.array_equal(to_host(x), to_host(y))


# -------------------------------------------------- tiny shard, 10 steps ------
def test_tiny_shard_ten_steps_against_oracle():
    """N = 1,048,576, W = 4 fp32 contributions ~ N(0, 1e-3), weights
    ~ N(0, 0.02), m = v = 0, AdamW(1e-4, 0.9, 0.95, 1e-8, 0.1), fresh seeded
    gradients each of 10 steps, bf16 copy out; every element every step."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["tiny_n1M_w4_f32"]
    n, W = wl.n, wl.W
    p, m, v = synth.host_state(wl.wid, n, wl.p_sigma)
    dp, dm, dv = to_dev(p), to_dev(m), to_dev(v)
    d16 = to_dev(np.zeros(n, np.uint16))
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    for t in range(1, wl.steps + 1):
        gs = synth.host_grads(wl.wid, t, W, n, wl.sigma)
        dd.aggregate_adam([to_dev(g) for g in gs], dp, dm, dv, d16, lr=hp["lr"],
                          beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
                          weight_decay=hp["wd"], step=t)
        t_.cuda.synchronize()
        want = oracle.fused(gs, p, m, v, t=t, **hp)
        got = {"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16)}
        assert_parity(got, want, f"step {t}")
        p, m, v = want["p"], want["m"], want["v"]


# ------------------------------------- format conversion and int32 contributions --
@pytest.mark.parametrize("gdtype", ["f32", "bf16"])
@pytest.mark.parametrize("k", [0, 16, 24, 30])
def test_quantize_matches_oracle(gdtype, k):
    import paper_2409_00918_amd as dd
    t_ = torch()
    for i, n in enumerate((1, 3, 4, 5, 1023, 1025, 65541, 300_007)):
        g = synth.host_grads(400 + k, i, 1, n, 1e-3, gdtype=gdtype, outlier_frac=0.02,
                             outlier_scale=1e6)[0]
        if gdtype == "f32" and n > 8:
            g[:6] = np.array([np.inf, -np.inf, np.nan, 3e38, -3e38, 1e-45], np.float32)
        for off in ((0, 0), (1, 3), (1, 1), (2, 2), (3, 3), (5, 1), (45, 45), (200, 200),
                    (7, 130)) if n > 4 else ((0, 0), (2, 2), (45, 45), (200, 200)):
            out = to_dev(np.zeros(n, np.int32), off[1])
            dd.quantize(to_dev(g, off[0]), out, frac_bits=k)
            t_.cuda.synchronize()
            assert np.array_equal(to_host(out), oracle.quantize_array(g, k)), (n, off)


def _quantize_edge_values(k):
    """Inputs at the edges of the integer format at scale 2^k: the largest
    value below 2^31 and 2^31 itself after scaling, -2^31 and the next float
    below it, ties to even around small integers, NaN, infinities, signed
    zeros and denormals."""
    s = np.float32(2.0 ** -k)
    ints = np.array([2147483520.0, 2147483648.0, 2147483904.0, -2147483648.0,
                     -2147483904.0, -2147483520.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5,
                     16777215.5, 8388607.5, 1.0, -1.0], np.float32)
    vals = np.concatenate([ints * s,
                           np.array([np.nan, -np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45,
                                     -1e-45, 1e-38, 3e38, -3e38], np.float32)])
    # neighbours one ulp either side of each scaled edge
    near = np.concatenate([np.nextafter(vals, np.float32(np.inf)),
                           np.nextafter(vals, np.float32(-np.inf))]).astype(np.float32)
    return np.concatenate([vals, near[np.isfinite(near)]]).astype(np.float32)


@pytest.mark.parametrize("k", [0, 24, 30])
def test_quantize_and_fixed_aggregate_at_format_edges(k):
    """The conversion's saturation, tie and NaN rules at the exact edges, in
    disdp_quantize (fp32 and bf16 input) and inside the fused fixed-point
    call, against the oracle."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    base = _quantize_edge_values(k)
    rng = np.random.default_rng(900 + k)
    n = 4 * base.size + 3                      # several groups and a ragged tail
    g = base[rng.integers(0, base.size, n)]
    g[:base.size] = base
    out = to_dev(np.zeros(n, np.int32))
    dd.quantize(to_dev(g), out, frac_bits=k)
    t_.cuda.synchronize()
    assert np.array_equal(to_host(out), oracle.quantize_array(g, k)), f"f32 k={k}"
    gb = t_.from_numpy(g).to(t_.bfloat16).view(t_.int16).numpy().view(np.uint16)
    dd.quantize(to_dev(gb), out, frac_bits=k)
    t_.cuda.synchronize()
    assert np.array_equal(to_host(out), oracle.quantize_array(gb, k)), f"bf16 k={k}"
    # W = 3 contributions built from the edge values: saturated sums too
    gs = [g, g[::-1].copy(), np.roll(g, 7)]
    p, m, v = synth.host_state(901, n, mv_sigma=1e-3)
    dg = [to_dev(x) for x in gs]
    dp, dm, dv = to_dev(p), to_dev(m), to_dev(v)
    d16 = to_dev(np.zeros(n, np.uint16))
    dai = to_dev(np.zeros(n, np.int32))
    daf = to_dev(np.zeros(n, np.float32))
    dd.aggregate_adam(dg, dp, dm, dv, d16, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                      eps=HP["eps"], weight_decay=HP["wd"], step=2, mode="fixed",
                      frac_bits=k, agg_out_f32=daf, agg_out_i32=dai)
    t_.cuda.synchronize()
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED, frac_bits=k, t=2,
                        want_agg_f32=True, want_agg_i32=True, **HP)
    assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv), "p16": to_host(d16),
                   "agg_f32": to_host(daf), "agg_i32": to_host(dai)}, want,
                  f"fixed edges k={k}")


@pytest.mark.parametrize("W", [1, 3, 8, 16, 20])
def test_int32_contributions_match_oracle_and_float_path(W):
    import paper_2409_00918_amd as dd
    t_ = torch()
    k = 24
    for i, n in enumerate((2, 1027, 100_003)):
        gs = synth.host_grads(410 + W, i, W, n, 1e-4, outlier_frac=0.01, outlier_scale=1e5)
        qs = [oracle.quantize_array(g, k) for g in gs]
        p, m, v = synth.host_state(410 + W, n, mv_sigma=1e-4)
        want = oracle.fused(qs, p, m, v, mode=oracle.AGG_FIXED, frac_bits=k, t=3,
                            want_agg_f32=True, want_agg_i32=True, **HP)
        outs = {}
        for label, srcs in (("int32", qs), ("float", gs)):
            dg = [to_dev(x) for x in srcs]
            st = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
            dai = to_dev(np.zeros(n, np.int32))
            daf = to_dev(np.zeros(n, np.float32))
            dd.aggregate_adam(dg, *st, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                              eps=HP["eps"], weight_decay=HP["wd"], step=3, mode="fixed",
                              frac_bits=k, agg_out_f32=daf, agg_out_i32=dai)
            t_.cuda.synchronize()
            outs[label] = {"p": to_host(st[0]), "m": to_host(st[1]), "v": to_host(st[2]),
                           "p16": to_host(st[3]), "agg_i32": to_host(dai),
                           "agg_f32": to_host(daf)}
        assert_parity(outs["int32"], want, f"int32 W={W} n={n}")
        for key in outs["int32"]:
            assert np.array_equal(outs["int32"][key], outs["float"][key]), key
        # the aggregation alone, unaligned int32 contributions
        dg = [to_dev(q, 1) for q in qs]
        dai = to_dev(np.zeros(n, np.int32))
        dd.aggregate(dg, mode="fixed", frac_bits=k, agg_out_i32=dai)
        t_.cuda.synchronize()
        assert np.array_equal(to_host(dai), want["agg_i32"])


def test_int32_contributions_rejected_in_fp32_mode():
    import paper_2409_00918_amd as dd
    t_ = torch()
    g = t_.zeros(8, dtype=t_.int32, device="cuda")
    with pytest.raises(dd.DisdpError) as ei:
        dd.aggregate([g, g], mode="fp32", agg_out_f32=t_.zeros(8, device="cuda"))
    assert ei.value.status == dd.ERR_UNSUPPORTED


# --------------------------------------------- host-resident (out-of-core) state --
def _pinned(a: np.ndarray):
    t_ = torch()
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    out = t_.empty(a.size, dtype=t_.from_numpy(a[:1].copy()).dtype, pin_memory=True)
    out.copy_(t_.from_numpy(a))
    return out


@pytest.mark.parametrize("where", ["state", "state+contributions"])
def test_fused_with_state_in_pinned_host_memory(where):
    """p, m, v and the bf16 copy in pinned host DRAM (streamed by the kernel
    over the host link), contributions in HBM or also in host memory."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    for mode in ("fp32", "fixed"):
        for n in (5, 4099, 250_001):
            gs = synth.host_grads(500, 1, 8, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
            p, m, v = synth.host_state(500, n, mv_sigma=1e-4)
            dg = [(_pinned(g) if where != "state" else to_dev(g)) for g in gs]
            hp_, hm, hv = _pinned(p), _pinned(m), _pinned(v)
            h16 = _pinned(np.zeros(n, np.uint16))
            dd.aggregate_adam(dg, hp_, hm, hv, h16, lr=HP["lr"], beta1=HP["beta1"],
                              beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                              step=2, mode=mode, frac_bits=24)
            t_.cuda.synchronize()
            want = oracle.fused(gs, p, m, v, t=2, mode=oracle.AGG_FIXED if mode == "fixed"
                                else oracle.AGG_FP32, frac_bits=24, **HP)
            got = {"p": hp_.numpy(), "m": hm.numpy(), "v": hv.numpy(),
                   "p16": h16.numpy().view(np.uint16)}
            assert_parity(got, want, f"{where} {mode} n={n}")


def test_pageable_host_memory_is_refused_before_any_launch():
    import ctypes
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 1024
    dev = [t_.zeros(n, device="cuda") for _ in range(2)]
    pageable = np.zeros(n, np.float32)          # malloc'd by numpy: not mapped
    # first confirm with the runtime itself that the buffer is unregistered,
    # so the library call below can only be refused, never launched
    hip = ctypes.CDLL("libamdhip64.so.7")

    class Attr(ctypes.Structure):
        _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int),
                    ("devicePointer", ctypes.c_void_p), ("hostPointer", ctypes.c_void_p),
                    ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]
    at = Attr()
    rc = hip.hipPointerGetAttributes(ctypes.byref(at), ctypes.c_void_p(pageable.ctypes.data))
    hip.hipGetLastError()
    if not (rc != 0 or at.type == 0):
        pytest.skip(f"runtime reports the pageable buffer as registered (rc={rc}, type={at.type})")
    st = dd.raw_aggregate([dev[0].data_ptr(), dev[1].data_ptr()], 2, dd.DT_F32, n,
                          dd.AGG_FP32, 0, pageable.ctypes.data, 0, 0)
    assert st == dd.ERR_INVALID_ARG
    st = dd.raw_quantize(pageable.ctypes.data, dd.DT_F32, n, 24, dev[0].data_ptr(), 0)
    assert st == dd.ERR_INVALID_ARG


@pytest.mark.parametrize("W,gdtype,mode", [(8, "f32", "fp32"), (16, "bf16", "fp32"),
                                           (4, "f32", "fixed")])
def test_fused_on_a_shard_placed_by_the_layout_planner(W, gdtype, mode):
    """All arrays as views of one allocation placed by disdp_shard_layout."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 100_003
    gs = synth.host_grads(600 + W, 1, W, n, 1e-4, gdtype=gdtype)
    p, m, v = synth.host_state(600 + W, n, mv_sigma=1e-4)
    sh = dd.allocate_shard(n, W, gdtype, agg_f32=True, agg_i32=(mode == "fixed"))
    for dst, src in zip(sh.grads, gs):
        dst.copy_(to_dev(src))
    for dst, src in ((sh.param, p), (sh.m, m), (sh.v, v)):
        dst.copy_(to_dev(src))
    dd.aggregate_adam(sh.grads, sh.param, sh.m, sh.v, sh.param_bf16, lr=HP["lr"],
                      beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                      step=4, mode=mode, frac_bits=24, agg_out_f32=sh.agg_f32,
                      agg_out_i32=sh.agg_i32)
    t_.cuda.synchronize()
    want = oracle.fused(gs, p, m, v, t=4, mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32,
                        frac_bits=24, want_agg_f32=True, want_agg_i32=(mode == "fixed"), **HP)
    got = {"p": to_host(sh.param), "m": to_host(sh.m), "v": to_host(sh.v),
           "p16": to_host(sh.param_bf16), "agg_f32": to_host(sh.agg_f32)}
    if mode == "fixed":
        got["agg_i32"] = to_host(sh.agg_i32)
    assert_parity(got, want, f"shard W={W} {gdtype} {mode}")


def test_contiguous_shard_slab_lifetime():
    """allocate_shard's physically contiguous slab: every view sits at the
    planner's offset inside it, the memory stays valid while any view is
    alive after the Shard object is gone, and when the last view goes the
    block returns to the process's pool (never to the device) and serves
    the next shard that fits."""
    import gc
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 50_000_000, 4
    gc.collect()
    t_.cuda.synchronize()
    free0, _ = t_.cuda.mem_get_info()
    held0, leased0, _ = dd.contiguous_pool()
    sh = dd.allocate_shard(n, W, "f32")
    assert sh.contiguous, "the runtime refused a physically contiguous slab"
    offs, total = dd.shard_layout(n, W, "f32")
    base = sh.slab.data_ptr()
    for i, x in enumerate(sh.grads + [sh.param, sh.m, sh.v, sh.param_bf16]):
        assert x.data_ptr() == base + offs[i], i
    held1, leased1, _ = dd.contiguous_pool()
    assert leased1 - leased0 >= total
    slack = 64 << 20                 # device-wide free-memory accounting is not exact
    if held1 > held0:                # a new block, not one from the pool
        free1, _ = t_.cuda.mem_get_info()
        assert free0 - free1 >= total - slack
    keep = sh.v
    keep.fill_(1.5)
    del sh, x
    gc.collect()
    t_.cuda.synchronize()
    assert dd.contiguous_pool()[1] == leased1                  # still held by the view
    assert bool((keep[-1000:] == 1.5).all()) and bool((keep[:1000] == 1.5).all())
    del keep
    gc.collect()
    t_.cuda.synchronize()
    held2, leased2, idle2 = dd.contiguous_pool()
    assert leased2 == leased0 and held2 == held1 and idle2 >= total   # back in the pool
    free2, _ = t_.cuda.mem_get_info()
    assert free0 - free2 >= (held1 - held0) - slack            # not back on the device
    # the next shard that fits takes the pooled block; a second one at the
    # same time gets a block of its own
    a = dd.allocate_shard(n - 1000, W, "f32")
    assert a.contiguous and dd.contiguous_pool()[0] == held2   # no new block
    b = dd.allocate_shard(n - 2000, W, "f32")
    assert b.contiguous and b.slab.data_ptr() != a.slab.data_ptr()
    assert dd.contiguous_pool()[1] >= leased0 + a.slab.numel() + b.slab.numel()
    del a, b
    gc.collect()
    assert dd.contiguous_pool()[1] == leased0
    # a small shard is not worth a block kept for the life of the process
    small = dd.allocate_shard(100_000, W, "f32")
    assert not small.contiguous and dd.contiguous_pool()[1] == leased0


def test_pooled_block_waits_for_work_queued_on_it():
    """A contiguous block released while fused calls on another stream still
    write into it is leased again only after that work is done: a fill made
    on the default stream right after the new lease survives."""
    import gc
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 50_000_000, 4
    a = dd.allocate_shard(n, W, "f32")
    assert a.contiguous, "the runtime refused a physically contiguous slab"
    base = a.slab.data_ptr()
    for x in a.grads + [a.param, a.m, a.v]:
        x.fill_(0.5)
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    for step in range(1, 41):          # about 15 ms of writes queued on `side`
        dd.aggregate_adam(a.grads, a.param, a.m, a.v, a.param_bf16, lr=1e-4,
                          beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1,
                          step=step, stream=side)
    del a, x
    gc.collect()
    b = dd.allocate_shard(n, W, "f32")
    assert b.contiguous and b.slab.data_ptr() == base, "the pooled block was not reused"
    b.slab.fill_(7)
    t_.cuda.synchronize()
    assert bool((b.slab == 7).all()), "queued work wrote into the block after its new lease"
    del b
    gc.collect()


def test_shard_falls_back_to_the_caching_allocator(monkeypatch):
    """Without a physically contiguous block (refused by the runtime, here
    forced) or with contiguous=False, the shard lives in torch's caching
    allocator at the same planned offsets and computes the same bits."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W = 70_001, 3
    gs = synth.host_grads(640, 1, W, n, 1e-4)
    p, m, v = synth.host_state(640, n, mv_sigma=1e-4)
    want = oracle.fused(gs, p, m, v, t=2, **HP)
    shards = [dd.allocate_shard(n, W, "f32", contiguous=False)]
    monkeypatch.setattr(dd, "contiguous_bytes", lambda nbytes, device="cuda": None)
    shards.append(dd.allocate_shard(n, W, "f32"))
    offs, _ = dd.shard_layout(n, W, "f32")
    for which, sh in enumerate(shards):
        assert not sh.contiguous
        assert sh.param.data_ptr() == sh.slab.data_ptr() + offs[W]
        for dst, src in zip(sh.grads, gs):
            dst.copy_(to_dev(src))
        for dst, src in ((sh.param, p), (sh.m, m), (sh.v, v)):
            dst.copy_(to_dev(src))
        dd.aggregate_adam(sh.grads, sh.param, sh.m, sh.v, sh.param_bf16, lr=HP["lr"],
                          beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
                          weight_decay=HP["wd"], step=2)
        t_.cuda.synchronize()
        got = {"p": to_host(sh.param), "m": to_host(sh.m), "v": to_host(sh.v),
               "p16": to_host(sh.param_bf16)}
        diag = []
        for k, inp in (("p", p), ("m", m), ("v", v)):
            d = np.flatnonzero(bits(got[k]) != bits(want[k]))
            if d.size:
                runs = int(np.count_nonzero(np.diff(d) != 1)) + 1
                unwritten = int(np.count_nonzero(bits(got[k][d]) == bits(inp[d])))
                diag.append(f"{k}: {d.size} differ in {runs} runs, [{d.min()}, {d.max()}], "
                            f"{unwritten} still the input, got {got[k][d[:3]]} "
                            f"want {want[k][d[:3]]}")
        assert_parity(got, want, f"caching-allocator shard {which} at "
                                 f"{sh.slab.data_ptr():#x}: {'; '.join(diag)}")


# ------------------------------------------------------------ many tensors --
def _multi_tensors(rng, T, W, gdtype, unrelated=False, sizes=None, seed=800):
    """T tensors, each in buffers of its own at random element offsets
    (one offset per tensor, or one per array), with host copies."""
    tensors, host = [], []
    choices = [0, 1, 2, 3, 4, 5, 63, 255, 256, 257, 1000, 4099, 20_001, 65_541]
    for j in range(T):
        n = sizes[j] if sizes is not None else int(rng.choice(choices))
        gt = "f32" if gdtype == "i32" else gdtype
        gs = synth.host_grads(seed + j, 1, W, n, 1e-4, gdtype=gt, outlier_frac=0.01,
                              outlier_scale=100.0)
        if gdtype == "i32":
            gs = [oracle.quantize_array(g, 24) for g in gs]
        p, m, v = synth.host_state(seed + j, n, mv_sigma=1e-4)
        off = [int(x) for x in rng.integers(0, 300, W + 4)] if unrelated else \
            [int(rng.integers(0, 300))] * (W + 4)
        dg = [to_dev(g, off[w]) for w, g in enumerate(gs)]
        dp, dm, dv = to_dev(p, off[W]), to_dev(m, off[W + 1]), to_dev(v, off[W + 2])
        d16 = to_dev(np.zeros(n, np.uint16), off[W + 3])
        tensors.append((dg, dp, dm, dv, d16))
        host.append((gs, p, m, v))
    return tensors, host


@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fp32"), ("f32", "fixed"),
                                         ("bf16", "fixed"), ("i32", "fixed")])
@pytest.mark.parametrize("W", [1, 3, 8, 13])
def test_multi_tensor_call_matches_oracle(gdtype, mode, W):
    """disdp_aggregate_adam_multi over 40 tensors of mixed sizes (empty ones
    included), each in buffers of its own at common or unrelated offsets
    (bf16 arrays of both parities take the single-tensor element path):
    every tensor against the oracle."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(1000 + W)
    for unrelated in (False, True):
        tensors, host = _multi_tensors(rng, 40, W, gdtype, unrelated=unrelated)
        dd.aggregate_adam_multi(tensors, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                                eps=HP["eps"], weight_decay=HP["wd"], step=3, mode=mode,
                                frac_bits=24)
        t_.cuda.synchronize()
        for j, ((dg, dp, dm, dv, d16), (gs, p, m, v)) in enumerate(zip(tensors, host)):
            want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed"
                                else oracle.AGG_FP32, frac_bits=24, t=3, **HP)
            assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv),
                           "p16": to_host(d16)}, want,
                          _label(j=j, n=p.size, unrelated=unrelated))


@pytest.mark.parametrize("W,T", [(8, 150), (64, 21), (2, 60)])
def test_multi_tensor_call_equals_one_call_per_tensor(W, T):
    """Across many batches (W = 8: 26 tensors per launch; W = 64: 4), with
    and without bf16 copies: the multi-tensor call gives the bits of one
    disdp_aggregate_adam per tensor."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(2000 + W)
    sizes = [int(x) for x in rng.integers(0, 30_000, T)]
    a, _ = _multi_tensors(rng, T, W, "f32", sizes=sizes, seed=900)
    b = [([g.clone() for g in dg], dp.clone(), dm.clone(), dv.clone(), d16.clone())
         for dg, dp, dm, dv, d16 in a]
    for copies in (True, False):
        kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
                  weight_decay=HP["wd"], step=5 if copies else 6)
        dd.aggregate_adam_multi([(g, p, m, v, c if copies else None) for g, p, m, v, c in a],
                                **kw)
        for g, p, m, v, c in b:
            dd.aggregate_adam(g, p, m, v, c if copies else None, **kw)
        t_.cuda.synchronize()
        for j, (x, y) in enumerate(zip(a, b)):
            for u, w in zip(x[1:], y[1:]):
                assert t_.equal(u, w), _label(j=j, n=sizes[j], copies=copies)


@pytest.mark.parametrize("gdtype,mode", [("f32", "fp32"), ("bf16", "fixed")])
def test_multi_tensor_step_object_over_steps(gdtype, mode):
    """MultiTensorStep (tensors checked and packed once) stepped four times
    with fresh contributions written into the same buffers: every tensor
    against the oracle's own trajectory each step, and bit-equal to one
    aggregate_adam_multi call per step on copies of the state."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(3100)
    W = 5
    a, host = _multi_tensors(rng, 30, W, gdtype, unrelated=True, seed=3200)
    b = [(dg, dp.clone(), dm.clone(), dv.clone(), d16.clone()) for dg, dp, dm, dv, d16 in a]
    step = dd.MultiTensorStep(a, mode=mode, frac_bits=24)
    assert step.T == 30 and step.W == W
    state = [(p.copy(), m.copy(), v.copy()) for _, p, m, v in host]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"])
    for t in range(1, 5):
        fresh = []
        for j, (dg, *_rest) in enumerate(a):
            n = dg[0].numel()
            gs = synth.host_grads(3300 + 10 * t + j, t, W, n, 1e-4, gdtype=gdtype)
            for d, g in zip(dg, gs):
                d.copy_(t_.from_numpy(np.ascontiguousarray(
                    g.view(np.int16) if g.dtype == np.uint16 else g)))
            fresh.append(gs)
        step(step=t, **kw)
        dd.aggregate_adam_multi(b, step=t, mode=mode, frac_bits=24, **kw)
        t_.cuda.synchronize()
        for j, ((dg, dp, dm, dv, d16), gs) in enumerate(zip(a, fresh)):
            p, m, v = state[j]
            want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if mode == "fixed"
                                else oracle.AGG_FP32, frac_bits=24, t=t, **HP)
            assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv),
                           "p16": to_host(d16)}, want, _label(t=t, j=j, n=p.size))
            state[j] = (want["p"], want["m"], want["v"])
            for u, w in zip((dp, dm, dv, d16), b[j][1:]):
                assert t_.equal(u, w), _label(t=t, j=j)
    with pytest.raises(TypeError):
        step(step=5)                       # neither hyperparameters nor scalars
    dd.MultiTensorStep([])(step=1, **kw)   # no tensors: nothing to do


def test_multi_tensor_call_with_pinned_host_state_and_on_a_cu_masked_stream():
    """The many-tensor call with every tensor's p, m, v and bf16 copy in
    pinned host memory (contributions in HBM): each tensor against the
    oracle; and on CU-masked streams (a raised occupancy cap), bit-equal to
    the default stream."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    W, sizes = 4, [5, 4099, 0, 250_001, 257, 64]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=2)
    for mode in ("fp32", "fixed"):
        tensors, want = [], []
        for j, n in enumerate(sizes):
            gs = synth.host_grads(4000 + j, 1, W, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
            p, m, v = synth.host_state(4000 + j, n, mv_sigma=1e-4)
            host = _pinned if n else to_dev    # an empty tensor has no pinned storage
            tensors.append(([to_dev(g) for g in gs], host(p), host(m), host(v),
                            host(np.zeros(n, np.uint16))))
            want.append(oracle.fused(gs, p, m, v, t=2, mode=oracle.AGG_FIXED if mode == "fixed"
                                     else oracle.AGG_FP32, frac_bits=24, **HP))
        dd.aggregate_adam_multi(tensors, mode=mode, frac_bits=24, **kw)
        t_.cuda.synchronize()
        for j, ((_, hp_, hm, hv, h16), w) in enumerate(zip(tensors, want)):
            got = {"p": to_host(hp_), "m": to_host(hm), "v": to_host(hv), "p16": to_host(h16)}
            assert_parity(got, w, _label(host_state=mode, j=j, n=sizes[j]))
    rng = np.random.default_rng(4100)
    a, _ = _multi_tensors(rng, 30, 8, "f32", unrelated=True, seed=4200)
    state0 = [[x.clone() for x in (dp, dm, dv, d16)] for _, dp, dm, dv, d16 in a]
    dd.aggregate_adam_multi(a, **kw)
    t_.cuda.synchronize()
    ref = [[x.clone() for x in (dp, dm, dv, d16)] for _, dp, dm, dv, d16 in a]
    for n_cus in (32, 200):
        for (_, dp, dm, dv, d16), st in zip(a, state0):
            for dst, src in zip((dp, dm, dv, d16), st):
                dst.copy_(src)
        t_.cuda.synchronize()
        s, h, hip = cu_masked_stream(n_cus)
        try:
            dd.aggregate_adam_multi(a, stream=s, **kw)
            s.synchronize()
            for j, ((_, dp, dm, dv, d16), r) in enumerate(zip(a, ref)):
                for u, w in zip((dp, dm, dv, d16), r):
                    assert t_.equal(u, w), _label(cus=n_cus, j=j)
        finally:
            t_.cuda.synchronize()
            hip.hipStreamDestroy(h)


def test_multi_tensor_call_captured_in_a_hip_graph():
    """The multi-tensor call enqueues kernel launches only: captured once,
    replayed three times with eager work between, it equals the same call
    made eagerly on copies of the state."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(77)
    a, _ = _multi_tensors(rng, 60, 8, "f32", seed=950)
    b = [(dg, dp.clone(), dm.clone(), dv.clone(), d16.clone()) for dg, dp, dm, dv, d16 in a]
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], step=2)
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    graph = t_.cuda.CUDAGraph()
    with t_.cuda.graph(graph, stream=side):
        dd.aggregate_adam_multi(a, **kw)
    t_.cuda.synchronize()
    other = t_.zeros(1 << 20, device="cuda")
    for r in range(3):
        graph.replay()
        dd.aggregate_adam_multi(b, **kw)
        t_.cuda.synchronize()
        other.add_(1.0)
        t_.cuda.synchronize()
        for j, (x, y) in enumerate(zip(a, b)):
            for u, w in zip(x[1:], y[1:]):
                assert t_.equal(u, w), _label(replay=r, j=j)
    del graph


def test_multi_tensor_graph_serves_every_step():
    """The multi-tensor call with the step's constants in device memory,
    captured once with the copy node that refreshes them, replayed for four
    steps with fresh contributions: every tensor against the oracle each
    step."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    rng = np.random.default_rng(88)
    W = 5
    tensors, host = _multi_tensors(rng, 30, W, "f32", seed=970)
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"])
    hst = t_.zeros(10, dtype=t_.float32, pin_memory=True)
    dev = t_.zeros(10, dtype=t_.float32, device="cuda")
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    graph = t_.cuda.CUDAGraph()
    with t_.cuda.graph(graph, stream=side):
        dev.copy_(hst, non_blocking=True)
        dd.aggregate_adam_multi(tensors, scalars=dev)
    t_.cuda.synchronize()
    state = [(p, m, v) for _, p, m, v in host]
    for t in range(1, 5):
        grads = []
        for j, (dg, *_rest) in enumerate(tensors):
            n = dg[0].numel()
            gs = synth.host_grads(5000 + 31 * t + j, t, W, n, 1e-4)
            for d, g in zip(dg, gs):
                d.copy_(t_.from_numpy(g))
            grads.append(gs)
        hst.copy_(t_.frombuffer(bytearray(dd.step_scalars(step=t, **kw)), dtype=t_.float32))
        t_.cuda.synchronize()
        graph.replay()
        t_.cuda.synchronize()
        for j, ((dg, dp, dm, dv, d16), gs) in enumerate(zip(tensors, grads)):
            p, m, v = state[j]
            want = oracle.fused(gs, p, m, v, t=t, **HP)
            assert_parity({"p": to_host(dp), "m": to_host(dm), "v": to_host(dv),
                           "p16": to_host(d16)}, want, _label(step=t, j=j))
            state[j] = (want["p"], want["m"], want["v"])
    del graph
