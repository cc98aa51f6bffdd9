"""Parity at full shard sizes, in the same launch configuration the benchmark
times (the same library call on the same tensors): every element of the
first and last step against the oracle (run chunk by chunk on the host's
threads), sampled elements of the steps between, and long trajectories on
sampled elements.

Shards (seeded synthetic stand-ins for one data-parallel shard of the
paper's OPT-family models, Table V):
  * 7B / 8:    N = 875,000,000, W = 8 fp32 contributions ~ N(0, 1e-4) with a
               1% x100 outlier tail, AdamW lr 1e-4, t = 1..5;
  * 13B / 16:  N = 812,500,000, W = 16 bf16 contributions ~ N(0, 1e-4),
               AdamW lr 3e-4, t = 1..5;
  * 175B / 64: N = 2,734,375,000 (> 2^31), W = 8 fp32 contributions quantised
               at 2^24 and summed as integers, int32 aggregate written and
               compared bit for bit, t = 1..5.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import assert_parity, to_host, torch, whole_shard_mismatches

pytestmark = pytest.mark.gpu

SAMPLE = 1 << 18
TILE = 256             # elements per block tile in the vector kernels (64 lanes x 4)


def sample_indices(n, seed):
    rng = np.random.default_rng(seed)
    parts = [rng.integers(0, n, SAMPLE), np.arange(min(n, 4096)),
             np.arange(max(0, n - 4096), n)]
    # both sides of tile boundaries spread over the shard, and the int32
    # index boundary when the shard crosses it
    b = (rng.integers(1, max(2, n // TILE), 512) * TILE)
    parts += [b - 1, b, b + 1]
    for edge in (2**31 // 4, 2**31 // 2, 2**31):
        if edge + 8 < n:
            parts.append(np.arange(edge - 8, edge + 8))
    idx = np.unique(np.concatenate(parts))
    return idx[(idx >= 0) & (idx < n)].astype(np.int64)


def shard_bytes(wl):
    gb = 2 if wl.gdtype == "bf16" else 4
    return wl.n * (wl.W * gb + 12 + 2 + (4 if wl.mode == "fixed" else 0))


def bytes_needed(wl):
    return shard_bytes(wl) + wl.n * 4 * 3


def room_for(wl):
    """Device memory a shard test can use: what is free, plus an idle block
    of the contiguous pool large enough to hold the shard (a shard released
    by an earlier test stays in the pool and serves the next one)."""
    import paper_2409_00918_amd as dd
    free, _ = torch().cuda.mem_get_info()
    idle = dd.contiguous_pool()[2]
    return free + (idle if idle >= shard_bytes(wl) else 0)


def test_grids_beyond_2_to_the_32_lanes():
    """A shard of 2^34 + 12,345 elements needs more one-tile blocks (and
    more quantize lanes) than one dispatch counts (2^32 - 1 work-items):
    the library clamps its grids and the kernels walk the rest grid-stride.
    disdp_aggregate of one bf16 contribution in fp32 mode returns every
    element widened, checked over all of them (arbitrary bit patterns, NaNs
    included: no arithmetic touches them); disdp_quantize of the same array
    matches the oracle on sampled elements, including those the clamped grid
    reaches on its second pass and the last ones."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    n = (1 << 34) + 12_345
    free, _ = t_.cuda.mem_get_info()
    if n * 6 + (1 << 31) > 0.92 * free:
        pytest.skip(f"needs {n * 6 / 2**30:.0f} GiB, {free / 2**30:.0f} free")
    chunk = 1 << 28
    print(f"[fullsize] 2^34+ n={n} fill", flush=True)
    g = t_.empty(n, dtype=t_.int16, device="cuda")
    gen = t_.Generator(device="cuda")
    gen.manual_seed(34)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        g[s:e] = t_.randint(-32768, 32768, (e - s,), dtype=t_.int32, device="cuda",
                            generator=gen).to(t_.int16)
    agg = t_.empty(n, dtype=t_.float32, device="cuda")
    print("[fullsize] 2^34+ aggregate", flush=True)
    dd.aggregate([g], mode="fp32", agg_out_f32=agg)
    t_.cuda.synchronize()
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        same = t_.equal(agg[s:e].view(t_.int32), g[s:e].to(t_.int32) << 16)
        assert same, f"aggregate differs in [{s}, {e})"
    del agg
    out = t_.empty(n, dtype=t_.int32, device="cuda")
    print("[fullsize] 2^34+ quantize", flush=True)
    dd.quantize(g, out, frac_bits=24)
    t_.cuda.synchronize()
    # one 64-lane block per 256 elements, at most (2^32 - 1) // 64 blocks:
    # the first pass of the clamped grid ends here
    first_pass = ((2**32 - 1) // 64) * 64 * 4
    idx = np.unique(np.concatenate([sample_indices(n, 34),
                                    np.arange(first_pass - 300, first_pass + 300)]))
    ti = t_.from_numpy(idx).cuda()
    gh = g[ti].cpu().numpy().view(np.uint16)
    want = oracle.quantize_array(gh, 24)
    got = out[ti].cpu().numpy()
    assert np.array_equal(got, want)
    del out, g
    t_.cuda.empty_cache()


@pytest.mark.parametrize("name", ["opt7b_shard8_w8_f32", "opt13b_shard16_w16_bf16",
                                  "c175b_shard64_w8_fixed24"])
def test_full_size_shard_whole_parity(name):
    """Steps t = 1..5 of the shard in the launch configuration bench.py
    times.  At t = 1 and t = 5 every element of p, m, v, the bf16 copy and
    (175B/64) the int32 aggregate is compared bit for bit with the oracle,
    run chunk by chunk on the host's threads from a device snapshot of the
    state taken just before the step; at t = 2..4 sampled elements are.
    Zero mismatching elements are allowed."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS[name]
    free = room_for(wl)
    if bytes_needed(wl) > 0.92 * free:
        pytest.skip(f"{name} needs {bytes_needed(wl) / 2**30:.0f} GiB, {free / 2**30:.0f} free")
    n, W = wl.n, wl.W
    fixed = wl.mode == "fixed"
    print(f"[fullsize] {name} n={n} W={W} alloc", flush=True)
    # the same placement bench.py uses: one allocation, disdp_shard_layout
    sh = dd.allocate_shard(n, W, wl.gdtype, agg_i32=fixed)
    dg = synth.device_grads(wl.wid, 1, W, n, wl.sigma, gdtype=wl.gdtype,
                            outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale,
                            out=sh.grads)
    dp, dm, dv = synth.device_state(wl.wid, n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    d16 = sh.param_bf16
    dai = sh.agg_i32
    snap = [t_.empty_like(dp) for _ in range(3)]
    idx = sample_indices(n, wl.wid)
    ix = t_.from_numpy(idx).cuda()
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    whole_steps = (1, wl.steps)
    try:
        for t in range(1, wl.steps + 1):
            if t > 1:
                synth.device_grads(wl.wid, t, W, n, wl.sigma, gdtype=wl.gdtype,
                                   outlier_frac=wl.outlier_frac,
                                   outlier_scale=wl.outlier_scale, out=dg)
            if t in whole_steps:
                for dst, src in zip(snap, (dp, dm, dv)):
                    dst.copy_(src)
            else:
                gs = [to_host(g[ix]) for g in dg]
                p0, m0, v0 = (to_host(x[ix]) for x in (dp, dm, dv))
            dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                              beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                              step=t, mode=wl.mode, frac_bits=wl.frac_bits,
                              agg_out_i32=dai)
            t_.cuda.synchronize()
            if t in whole_steps:
                post = {"p": dp, "m": dm, "v": dv, "p16": d16}
                if fixed:
                    post["agg_i32"] = dai
                bad = whole_shard_mismatches(dg, snap, post, gdtype=wl.gdtype, mode=wl.mode,
                                             frac_bits=wl.frac_bits, t=t, hp=hp,
                                             label=f"{name} step {t}")
                assert bad["elements"] == n
                assert all(c == 0 for k, c in bad.items() if k != "elements"), \
                    f"{name} step {t}: mismatching elements {bad}"
                print(f"[fullsize] {name} step {t} ok (all {n} elements)", flush=True)
            else:
                got = {"p": to_host(dp[ix]), "m": to_host(dm[ix]), "v": to_host(dv[ix]),
                       "p16": to_host(d16[ix])}
                if fixed:
                    got["agg_i32"] = to_host(dai[ix])
                want = oracle.fused(gs, p0, m0, v0,
                                    mode=oracle.AGG_FIXED if fixed else oracle.AGG_FP32,
                                    frac_bits=wl.frac_bits, t=t, want_agg_i32=fixed, **hp)
                assert_parity(got, want, f"{name} step {t}")
                print(f"[fullsize] {name} step {t} ok ({idx.size} sampled elements)",
                      flush=True)
    finally:
        del dg, dp, dm, dv, d16, dai, sh, snap
        t_.cuda.empty_cache()


def test_full_size_trajectory_of_40_steps():
    """40 steps on the 7B/8 shard (fresh seeded gradients every step, the
    launch configuration bench.py times).  The oracle runs the same 40 steps
    on its own copy of a sampled subset of the state, from the initial state
    only, so any difference would compound; every 8 steps the sampled p, m,
    v and bf16 copy must match it bit for bit."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["opt7b_shard8_w8_f32"]
    free = room_for(wl)
    if bytes_needed(wl) > 0.92 * free:
        pytest.skip("not enough device memory")
    n, W = wl.n, wl.W
    sh = dd.allocate_shard(n, W, wl.gdtype)
    dp, dm, dv = synth.device_state(wl.wid, n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    idx = np.unique(np.random.default_rng(77).integers(0, n, 1 << 16)).astype(np.int64)
    ix = t_.from_numpy(idx).cuda()
    p, m, v = (to_host(x[ix]) for x in (dp, dm, dv))
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    try:
        for t in range(1, 41):
            synth.device_grads(wl.wid, 100 + t, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                               outlier_scale=wl.outlier_scale, out=sh.grads)
            gs = [to_host(g[ix]) for g in sh.grads]
            dd.aggregate_adam(sh.grads, dp, dm, dv, sh.param_bf16, lr=hp["lr"],
                              beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
                              weight_decay=hp["wd"], step=t)
            want = oracle.fused(gs, p, m, v, t=t, **hp)
            p, m, v = want["p"], want["m"], want["v"]
            if t % 8 == 0:
                t_.cuda.synchronize()
                got = {"p": to_host(dp[ix]), "m": to_host(dm[ix]), "v": to_host(dv[ix]),
                       "p16": to_host(sh.param_bf16[ix])}
                assert_parity(got, want, f"trajectory step {t}")
                print(f"[fullsize] trajectory step {t} ok", flush=True)
    finally:
        del dp, dm, dv, sh
        t_.cuda.empty_cache()


def test_full_size_graph_replayed_across_steps():
    """The 7B/8 shard driven by one captured HIP graph (copy node for the
    step's constants + disdp_aggregate_adam_dev), replayed for 5 steps with
    fresh seeded contributions written between replays: sampled elements
    against the oracle every step, and the bf16 copy checked everywhere."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["opt7b_shard8_w8_f32"]
    free = room_for(wl)
    if bytes_needed(wl) > 0.92 * free:
        pytest.skip("not enough device memory")
    n, W = wl.n, wl.W
    sh = dd.allocate_shard(n, W, wl.gdtype)
    dp, dm, dv = synth.device_state(wl.wid, n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    idx = sample_indices(n, 91)
    ix = t_.from_numpy(idx).cuda()
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    kw = dict(lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
              weight_decay=hp["wd"])
    host = t_.zeros(10, dtype=t_.float32, pin_memory=True)
    dev = t_.zeros(10, dtype=t_.float32, device="cuda")
    t_.cuda.synchronize()
    side = t_.cuda.Stream()
    graph = t_.cuda.CUDAGraph()
    with t_.cuda.graph(graph, stream=side):
        dev.copy_(host, non_blocking=True)
        dd.aggregate_adam_dev(sh.grads, dp, dm, dv, sh.param_bf16, scalars=dev)
    t_.cuda.synchronize()
    p, m, v = (to_host(x[ix]) for x in (dp, dm, dv))
    try:
        for t in range(1, 6):
            synth.device_grads(wl.wid, 200 + t, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                               outlier_scale=wl.outlier_scale, out=sh.grads)
            gs = [to_host(g[ix]) for g in sh.grads]
            host.copy_(t_.frombuffer(bytearray(dd.step_scalars(step=t, **kw)),
                                     dtype=t_.float32))
            t_.cuda.synchronize()
            graph.replay()
            t_.cuda.synchronize()
            want = oracle.fused(gs, p, m, v, t=t, **hp)
            got = {"p": to_host(dp[ix]), "m": to_host(dm[ix]), "v": to_host(dv[ix]),
                   "p16": to_host(sh.param_bf16[ix])}
            assert_parity(got, want, f"graph replay step {t}")
            assert t_.equal(dp.to(t_.bfloat16).view(t_.int16), sh.param_bf16), f"step {t}: p16"
            p, m, v = want["p"], want["m"], want["v"]
            print(f"[fullsize] graph replay step {t} ok", flush=True)
    finally:
        del graph, dp, dm, dv, sh
        t_.cuda.empty_cache()


def test_state_in_pinned_host_memory_at_scale():
    """The out-of-core launch bench.py --host-state times: W = 8 fp32
    contributions in HBM (the 7B/8 recipe), p, m, v and the bf16 copy in
    pinned host memory streamed by the kernel over the host link, on
    2^28 + 5 elements.  Step 1: every element against the oracle; steps 2
    and 3: sampled elements."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["opt7b_shard8_w8_f32"]
    n, W = (1 << 28) + 5, wl.W
    free, _ = t_.cuda.mem_get_info()
    if n * 4 * W > 0.9 * free:
        pytest.skip("not enough device memory")
    print(f"[fullsize] host state n={n} alloc", flush=True)
    dg = synth.device_grads(wl.wid, 1, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                            outlier_scale=wl.outlier_scale)
    dp, dm, dv = synth.device_state(wl.wid, n, wl.p_sigma)
    host = []
    for x in (dp, dm, dv):
        h = t_.empty(n, dtype=t_.float32, pin_memory=True)
        h.copy_(x)
        host.append(h)
    del dp, dm, dv
    h16 = t_.empty(n, dtype=t_.int16, pin_memory=True)
    snap = [x.clone() for x in host]
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    idx = sample_indices(n, 29)
    try:
        for t in range(1, 4):
            if t > 1:
                synth.device_grads(wl.wid, t, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                                   outlier_scale=wl.outlier_scale, out=dg)
                ix = t_.from_numpy(idx).cuda()
                gs = [to_host(g[ix]) for g in dg]
                p0, m0, v0 = (x.numpy()[idx] for x in host)
            dd.aggregate_adam(dg, *host, h16, lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"],
                              eps=hp["eps"], weight_decay=hp["wd"], step=t)
            t_.cuda.synchronize()
            if t == 1:
                bad = whole_shard_mismatches(dg, snap, {"p": host[0], "m": host[1],
                                                        "v": host[2], "p16": h16},
                                             gdtype="f32", mode="fp32", frac_bits=0, t=1,
                                             hp=hp, label="host state step 1")
                assert bad["elements"] == n
                assert all(c == 0 for k, c in bad.items() if k != "elements"), bad
            else:
                want = oracle.fused(gs, p0, m0, v0, t=t, **hp)
                got = {"p": host[0].numpy()[idx], "m": host[1].numpy()[idx],
                       "v": host[2].numpy()[idx], "p16": h16.numpy().view(np.uint16)[idx]}
                assert_parity(got, want, f"host state step {t}")
            print(f"[fullsize] host state step {t} ok", flush=True)
    finally:
        del dg, host, h16, snap
        t_.cuda.empty_cache()


def test_full_size_shard_in_the_shared_launch_shape(monkeypatch):
    """The 7B/8 shard in the four-wave launch shape (DISDP_LAUNCH_SHAPE=
    shared, the shape for a GPU shared with compute kernels): every element
    of t = 1 against the oracle."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["opt7b_shard8_w8_f32"]
    free = room_for(wl)
    if bytes_needed(wl) > 0.92 * free:
        pytest.skip("not enough device memory")
    monkeypatch.setenv("DISDP_LAUNCH_SHAPE", "shared")
    n, W = wl.n, wl.W
    sh = dd.allocate_shard(n, W, wl.gdtype)
    synth.device_grads(wl.wid, 1, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                       outlier_scale=wl.outlier_scale, out=sh.grads)
    synth.device_state(wl.wid, n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    snap = [x.clone() for x in (sh.param, sh.m, sh.v)]
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    try:
        dd.aggregate_adam(sh.grads, sh.param, sh.m, sh.v, sh.param_bf16, lr=hp["lr"],
                          beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
                          weight_decay=hp["wd"], step=1)
        t_.cuda.synchronize()
        bad = whole_shard_mismatches(sh.grads, snap, {"p": sh.param, "m": sh.m, "v": sh.v,
                                                      "p16": sh.param_bf16},
                                     gdtype="f32", mode="fp32", frac_bits=0, t=1, hp=hp,
                                     label="shared shape step 1")
        assert bad["elements"] == n
        assert all(c == 0 for k, c in bad.items() if k != "elements"), bad
    finally:
        del sh, snap
        t_.cuda.empty_cache()


def test_full_size_int32_contributions_equal_the_float_path():
    """NEXT-1 at full size: W = 8 contributions of the 7B/8 recipe converted
    by disdp_quantize to the switch's int32 format at 2^24 and summed as
    DISDP_DT_I32, against the same fp32 contributions converted inside the
    fused kernel (fixed mode; that path is checked element by element
    against the oracle on the 175B/64 shard).  t = 1 and t = 2 from the same
    state: every element of p, m, v, the bf16 copy and the int32 aggregate
    must be equal, compared on the device; sampled elements of the quantized
    contributions against the oracle's conversion."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    wl = synth.WORKLOADS["opt7b_shard8_w8_f32"]
    n, W, k = wl.n, wl.W, 24
    # the float side in a shard slab (a pooled block of an earlier test when
    # one is idle), the int32 side from the caching allocator
    free = room_for(wl)
    if n * (W * 4 + 12 + 2 + 4) * 2 > 0.9 * free:
        pytest.skip("not enough device memory")
    print(f"[fullsize] int32 contributions n={n}", flush=True)
    sh = dd.allocate_shard(n, W, "f32", agg_i32=True)
    gf = synth.device_grads(wl.wid, 1, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                            outlier_scale=wl.outlier_scale, out=sh.grads)
    gi = [t_.empty(n, dtype=t_.int32, device="cuda") for _ in range(W)]
    idx = sample_indices(n, 41)
    ix = t_.from_numpy(idx).cuda()
    hp = dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1), beta2=np.float32(wl.beta2),
              eps=np.float32(wl.eps), wd=np.float32(wl.wd))
    kw = dict(lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
              weight_decay=hp["wd"], mode="fixed", frac_bits=k)
    a = list(synth.device_state(wl.wid, n, wl.p_sigma, out=(sh.param, sh.m, sh.v)))
    b = [x.clone() for x in a]
    a16, ai = sh.param_bf16, sh.agg_i32
    b16 = t_.empty(n, dtype=t_.int16, device="cuda")
    bi = t_.empty(n, dtype=t_.int32, device="cuda")
    try:
        for t in (1, 2):
            if t > 1:
                synth.device_grads(wl.wid, t, W, n, wl.sigma, outlier_frac=wl.outlier_frac,
                                   outlier_scale=wl.outlier_scale, out=gf)
            for w in range(W):
                dd.quantize(gf[w], gi[w], frac_bits=k)
            t_.cuda.synchronize()
            for w in range(W):
                want = oracle.quantize_array(to_host(gf[w][ix]), k)
                assert np.array_equal(to_host(gi[w][ix]), want), f"quantize w={w} t={t}"
            dd.aggregate_adam(gf, *a, a16, step=t, agg_out_i32=ai, **kw)
            dd.aggregate_adam(gi, *b, b16, step=t, agg_out_i32=bi, **kw)
            t_.cuda.synchronize()
            for name, x, y in (("p", a[0], b[0]), ("m", a[1], b[1]), ("v", a[2], b[2]),
                               ("p16", a16, b16), ("agg_i32", ai, bi)):
                assert t_.equal(x.view(t_.int32) if x.dtype == t_.float32 else x,
                                y.view(t_.int32) if y.dtype == t_.float32 else y), \
                    f"t={t}: {name} differs between int32 and float contributions"
            print(f"[fullsize] int32 contributions step {t} ok (all {n} elements)", flush=True)
    finally:
        del gf, gi, a, b, a16, b16, ai, bi, sh
        t_.cuda.empty_cache()


@pytest.mark.parametrize("W,gdtype,mode,n", [(64, "bf16", "fp32", (1 << 28) + 3),
                                             (33, "f32", "fixed", (1 << 27) + 5)])
def test_run_time_worker_counts_at_scale(W, gdtype, mode, n):
    """The run-time worker-count kernels (W outside the compile-time set)
    at scale: every element of t = 1 against the oracle, the int32
    aggregate included in fixed mode."""
    import paper_2409_00918_amd as dd
    t_ = torch()
    gb = 2 if gdtype == "bf16" else 4
    fixed = mode == "fixed"
    need = n * (W * gb + 12 + 2 + (4 if fixed else 0) + 12)
    free, _ = t_.cuda.mem_get_info()
    if need > 0.9 * free:
        pytest.skip("not enough device memory")
    print(f"[fullsize] run-time W={W} {gdtype} {mode} n={n}", flush=True)
    dg = synth.device_grads(77, 1, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                            outlier_scale=100.0)
    dp, dm, dv = synth.device_state(77, n, 0.02)
    d16 = t_.empty(n, dtype=t_.int16, device="cuda")
    dai = t_.empty(n, dtype=t_.int32, device="cuda") if fixed else None
    snap = [x.clone() for x in (dp, dm, dv)]
    hp = dict(lr=np.float32(1e-4), beta1=np.float32(0.9), beta2=np.float32(0.95),
              eps=np.float32(1e-8), wd=np.float32(0.1))
    try:
        dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                          beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"], step=1,
                          mode=mode, frac_bits=24, agg_out_i32=dai)
        t_.cuda.synchronize()
        post = {"p": dp, "m": dm, "v": dv, "p16": d16}
        if fixed:
            post["agg_i32"] = dai
        bad = whole_shard_mismatches(dg, snap, post, gdtype=gdtype, mode=mode, frac_bits=24,
                                     t=1, hp=hp, label=f"run-time W={W} {gdtype} {mode}")
        assert bad["elements"] == n
        assert all(c == 0 for k, c in bad.items() if k != "elements"), bad
    finally:
        del dg, dp, dm, dv, d16, dai, snap
        t_.cuda.empty_cache()
