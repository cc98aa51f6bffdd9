"""The two launch shapes of the vector kernels, and the fused call running
next to a compute kernel on another stream of the same GPU.

DISDP_LAUNCH_SHAPE=shared selects four-wave blocks with one occupancy cap
per mode (for a GPU shared with compute kernels); the default is one-wave
blocks.  A launch shape changes only the grid, so every result must be bit
for bit the oracle's in both shapes, and a fused step run while a bf16 GEMM
loop occupies the chip must equal the same step run alone.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import (HP, assert_parity, cu_masked_stream, run_fused_case, to_dev, to_host,
                        torch)


pytestmark = pytest.mark.gpu

SHAPES = ["solo", "shared"]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import paper_2409_00918_amd as dd
    dd.lib()
    assert torch().cuda.is_available(), "GPU tests need a device"


@pytest.fixture
def shape(request, monkeypatch):
    if request.param == "shared":
        monkeypatch.setenv("DISDP_LAUNCH_SHAPE", "shared")
    else:
        monkeypatch.delenv("DISDP_LAUNCH_SHAPE", raising=False)
    return request.param


LENGTHS = [1, 5, 255, 257, 1023, 1025, 4099, 300_007]


@pytest.mark.parametrize("shape", SHAPES, indirect=True)
@pytest.mark.parametrize("W,gdtype,mode", [(1, "f32", "fp32"), (3, "bf16", "fixed"),
                                           (8, "f32", "fp32"), (8, "f32", "fixed"),
                                           (16, "bf16", "fp32"), (24, "f32", "fixed"),
                                           (64, "bf16", "fp32")])
def test_fused_in_each_shape_matches_oracle(shape, W, gdtype, mode):
    for i, n in enumerate(LENGTHS):
        got, want = run_fused_case(W, gdtype, mode, n, t=1 + i % 4, seed=300 + i)
        assert_parity(got, want, f"{shape} W={W} {gdtype} {mode} n={n}")


@pytest.mark.parametrize("shape", SHAPES, indirect=True)
@pytest.mark.parametrize("offsets", [(1, 0), (37, 200)])
def test_misaligned_arrays_in_each_shape(shape, offsets):
    """(1, 0) with bf16 contributions puts bf16 arrays at odd and even
    element offsets: the element-wise kernel.  (37, 200): a head before the
    vector kernel."""
    for gdtype, mode in (("bf16", "fp32"), ("f32", "fixed")):
        for n in (3, 1000, 70_001):
            got, want = run_fused_case(8, gdtype, mode, n, t=2, offsets=offsets, seed=31)
            assert_parity(got, want, f"{shape} offsets={offsets} {gdtype} {mode} n={n}")


@pytest.mark.parametrize("shape", SHAPES, indirect=True)
def test_aggregate_and_adam_step_in_each_shape(shape):
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = 100_003
    for W, gdtype, mode in ((8, "f32", "fixed"), (16, "bf16", "fp32"), (5, "f32", "fp32")):
        gs = synth.host_grads(700 + W, 1, W, n, 1e-4, gdtype=gdtype)
        daf = t_.empty(n, dtype=t_.float32, device="cuda")
        dai = t_.empty(n, dtype=t_.int32, device="cuda") if mode == "fixed" else None
        dd.aggregate([to_dev(g) for g in gs], mode=mode, frac_bits=24, agg_out_f32=daf,
                     agg_out_i32=dai)
        t_.cuda.synchronize()
        if mode == "fixed":
            ai, af = oracle.aggregate_fixed(gs, 24)
            assert np.array_equal(to_host(dai), ai), f"{shape} W={W} agg_i32"
        else:
            af = oracle.aggregate_f32(gs)
        assert np.array_equal(to_host(daf).view(np.uint32), af.view(np.uint32)), \
            f"{shape} W={W} agg_f32"
    agg = synth.host_grads(710, 1, 1, n, 3e-4)[0]
    p, m, v = synth.host_state(710, n, mv_sigma=1e-4)
    st = [to_dev(x) for x in (p, m, v)] + [to_dev(np.zeros(n, np.uint16))]
    dd.adam_step(to_dev(agg), *st, lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"],
                 eps=HP["eps"], weight_decay=HP["wd"], step=3)
    t_.cuda.synchronize()
    p1, m1, v1, p16 = oracle.adamw(agg, p, m, v, lr=HP["lr"], beta1=HP["beta1"],
                                   beta2=HP["beta2"], eps=HP["eps"], wd=HP["wd"], t=3)
    assert_parity({"p": to_host(st[0]), "m": to_host(st[1]), "v": to_host(st[2]),
                   "p16": to_host(st[3])}, {"p": p1, "m": m1, "v": v1, "p16": p16},
                  f"{shape} adam_step")


@pytest.mark.parametrize("shape", SHAPES, indirect=True)
@pytest.mark.parametrize("mode", ["fp32", "fixed"])
def test_fused_next_to_a_gemm_loop_equals_solo(shape, mode):
    """Five fused steps on one stream while another stream loops a bf16
    GEMM (4096^3, torch.matmul) equal, bit for bit, the same five steps run
    alone from the same start state; the concurrent result also matches the
    oracle's five steps on sampled elements."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n, W, K = (1 << 25) + 3, 8, 5
    dg = synth.device_grads(800, 1, W, n, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
    p0, m0, v0 = synth.device_state(800, n)
    gen = t_.Generator(device="cuda")
    gen.manual_seed(synth.seed_for(800, 0, 2000))
    A = t_.randn(4096, 4096, generator=gen, device="cuda").to(t_.bfloat16)
    B = t_.randn(4096, 4096, generator=gen, device="cuda").to(t_.bfloat16)
    C = t_.empty(4096, 4096, device="cuda", dtype=t_.bfloat16)
    kw = dict(lr=HP["lr"], beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
              weight_decay=HP["wd"], mode=mode, frac_bits=24)

    # streams with a full CU mask: each has a hardware queue of its own, so
    # the GEMMs and the fused steps really run at the same time
    total = t_.cuda.get_device_properties(0).multi_processor_count
    (side, hs, hip), (comp, hc, _) = cu_masked_stream(total), cu_masked_stream(total)

    def run(concurrent):
        st = [x.clone() for x in (p0, m0, v0)] + [t_.empty(n, dtype=t_.int16, device="cuda")]
        t_.cuda.synchronize()
        ev = []
        if concurrent:
            with t_.cuda.stream(comp):
                for _ in range(60):
                    a, b = t_.cuda.Event(enable_timing=True), t_.cuda.Event(enable_timing=True)
                    a.record(comp)
                    t_.matmul(A, B, out=C)
                    b.record(comp)
                    ev.append((a, b))
        f0, f1 = t_.cuda.Event(enable_timing=True), t_.cuda.Event(enable_timing=True)
        f0.record(side)
        for t in range(1, K + 1):
            dd.aggregate_adam(dg, *st, step=t, stream=side, **kw)
        f1.record(side)
        t_.cuda.synchronize()
        # GEMMs that started before the fused steps ended and ended after
        # they started: the two overlapped
        overlap = sum(1 for a, b in ev
                      if f0.elapsed_time(b) > 0 and a.elapsed_time(f1) > 0)
        return st, overlap

    try:
        solo, _ = run(False)
        conc, overlap = run(True)
    finally:
        t_.cuda.synchronize()
        hip.hipStreamDestroy(hs)
        hip.hipStreamDestroy(hc)
    print(f"[shapes] {shape} {mode}: {overlap} GEMMs overlapped the fused steps", flush=True)
    assert overlap > 0, "the GEMM loop and the fused steps did not overlap"
    for name, a, b in zip(("p", "m", "v", "p16"), solo, conc):
        assert t_.equal(a, b), f"{shape} {mode}: {name} differs next to the GEMM"
    idx = np.unique(np.concatenate([np.random.default_rng(8).integers(0, n, 1 << 15),
                                    np.arange(n - 300, n)]))
    ix = t_.from_numpy(idx).cuda()
    gs = [to_host(g[ix]) for g in dg]
    p, m, v = (to_host(x[ix]) for x in (p0, m0, v0))
    for t in range(1, K + 1):
        want = oracle.fused(gs, p, m, v, t=t, frac_bits=24,
                            mode=oracle.AGG_FIXED if mode == "fixed" else oracle.AGG_FP32, **HP)
        p, m, v = want["p"], want["m"], want["v"]
    assert_parity({"p": to_host(conc[0][ix]), "m": to_host(conc[1][ix]),
                   "v": to_host(conc[2][ix]), "p16": to_host(conc[3][ix])}, want,
                  f"{shape} {mode} concurrent vs oracle")


@pytest.mark.parametrize("value", ["SHARED", "bogus", ""])
def test_unrecognised_launch_shape_means_the_default(value, monkeypatch):
    """Only the exact value "shared" selects the shared shape; anything else
    launches the default shape, with the same (oracle-checked) bits."""
    monkeypatch.setenv("DISDP_LAUNCH_SHAPE", value)
    for W, gdtype, mode in ((8, "f32", "fp32"), (24, "f32", "fixed")):
        got, want = run_fused_case(W, gdtype, mode, 100_003, t=2, seed=400 + W)
        assert_parity(got, want, f"DISDP_LAUNCH_SHAPE={value!r} W={W} {mode}")
