#!/usr/bin/env python3
"""Benchmark of the DisDP parameter-server hot path on one MI355X.

One step = one fused call (disdp_aggregate_adam) over the whole shard: the
W-way reduction of the workers' gradient contributions, the AdamW update of
the fp32 master weight and moments, and the bf16 parameter copy.  Inputs are
seeded synthetic tensors resident in HBM before the timed region.

Default workload: one 1/8 shard of a 7B-parameter model, N = 875,000,000,
W = 8 fp32 contributions ~ N(0, 1e-4) with a 1% x100 outlier tail, AdamW
lr 1e-4, betas (0.9, 0.95), eps 1e-8, weight decay 0.1.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
    python bench.py --interference      # fused call next to a bf16 GEMM loop
    python bench.py --copy-probe        # plain 4 GiB device copy (counter scale)
    python bench.py --entry aggregate   # another entry point on the same shard
    python bench.py --entry fused_graph # the fused call replayed as one HIP graph
    python bench.py --entry layers      # the shard updated tensor by tensor

Prints one JSON line.  ``roofline`` prices the kernel against HBM bandwidth
(8 TB/s) with algorithmic bytes (each byte the call must move, counted once);
``traffic`` is the HBM byte count read from committed rocprofv3 counters when
they were taken on the current kernel source, else null.  ``cpu_baseline``
times the CPU oracle (single thread) on a bounded sample of the same shard;
``cpu_baseline_threads`` the same sample split over the host's threads.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Section III-D, step 5 of the backward stage (and Table III): per element
# the parameter server's Adam reads a 2-byte gradient and 12 bytes of model
# state (fp32 master weight, m, v) and writes the 12 bytes back plus a
# 2-byte parameter copy, doing 17 floating-point operations.
ADAM_CORE_BYTES = {"grad_in": 2, "states_in": 12, "states_out": 12,
                   "param_copy_out": 2}
ADAM_FLOPS_PER_ELEMENT = 17

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published peak
DEFAULT_WORKLOAD = "opt7b_shard8_w8_f32"
KERNEL_SOURCES = ["paper_2409_00918_amd/csrc/disdp_kernels.hip",
                  "paper_2409_00918_amd/csrc/disdp_launch.h",
                  "paper_2409_00918_amd/csrc/disdp_api.cpp"]
CPU_SAMPLE = 1 << 26            # elements of the shard the oracle is timed on
CPU_STEPS = 12
COPY_PROBE_ELEMS = 1 << 30      # fp32 elements moved by the copy probe (4 GiB each way)


def kernel_source_hash() -> str:
    """Hash of what decides the fused kernel's machine code: its sources and
    the compile flags of libdisdp."""
    from paper_2409_00918_amd import build as _build
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    h.update(" ".join(a for a in _build.FLAGS if not a.startswith("/")).encode())
    return h.hexdigest()[:16]


def probe_lib():
    """libdisdp_probe.so (a plain copy kernel), loaded after torch so that it
    binds to torch's HIP runtime."""
    import ctypes
    import torch  # noqa: F401
    from paper_2409_00918_amd import build as _build
    L = ctypes.CDLL(_build.PROBE_LIB)
    L.disdp_probe_copy.restype = ctypes.c_int
    L.disdp_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.c_void_p]
    return L


def committed_traffic(workload: str, src_hash: str):
    """HBM bytes per launch from the committed counter summary of this
    workload, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"fused_{workload}.md")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            m = re.match(r"\s*traffic-json:\s*(\{.*\})\s*$", line)
            if m:
                rec = json.loads(m.group(1))
                if rec.get("kernel_source_hash") == src_hash:
                    return rec
    return None


def hparams(wl):
    import numpy as np
    return dict(lr=np.float32(wl.lr), beta1=np.float32(wl.beta1),
                beta2=np.float32(wl.beta2), eps=np.float32(wl.eps),
                wd=np.float32(wl.wd))


CONTIGUOUS = True   # --allocator: one physically contiguous block, or torch's allocator


def workload(args):
    """The workload named by --workload, with --n / --W overrides (for
    sweeps; the name then records them)."""
    import dataclasses
    import synth
    wl = synth.WORKLOADS[args.workload]
    n = getattr(args, "n", None)
    W = getattr(args, "W", None)
    if n or W:
        wl = dataclasses.replace(wl, n=n or wl.n, W=W or wl.W,
                                 name=f"{wl.name}@n={n or wl.n},W={W or wl.W}")
    return wl


def shard(n, W, gdtype, **kw):
    """dd.allocate_shard with the process's allocator choice."""
    import paper_2409_00918_amd as dd
    return dd.allocate_shard(n, W, gdtype, contiguous=CONTIGUOUS, **kw)


def allocate(wl):
    """The shard's arrays in one allocation placed by disdp_shard_layout
    (as a parameter server would lay out its shard), filled with the seeded
    step-1 inputs.  The returned Shard owns the allocation; its fields are
    views into it."""
    import synth
    sh = shard(wl.n, wl.W, wl.gdtype)
    synth.device_grads(wl.wid, 1, wl.W, wl.n, wl.sigma, gdtype=wl.gdtype,
                       outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale,
                       out=sh.grads)
    synth.device_state(wl.wid, wl.n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    return sh


def copy_ceiling_gbps(elems=1 << 30, reps=10):
    """Bytes moved per second by a plain copy kernel (16-byte non-temporal
    loads and stores, libdisdp_probe.so) of `elems` fp32 elements on this
    GPU, measured now: the practical HBM ceiling the fused kernel is
    compared with, next to the datasheet peak."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    L = probe_lib()
    # in the same kind of memory as the shard: one physically contiguous
    # block holding both buffers when the runtime has one
    nbytes = elems * 4
    gap = 64 << 20
    slab = dd.contiguous_bytes(2 * nbytes + gap, "cuda")
    if slab is not None:
        src = slab[:nbytes].view(torch.float32).fill_(1.0)
        dst = slab[nbytes + gap: 2 * nbytes + gap].view(torch.float32)
    else:
        src = torch.ones(elems, device="cuda")
        dst = torch.empty_like(src)
    s = torch.cuda.current_stream()
    assert L.disdp_probe_copy(src.data_ptr(), dst.data_ptr(), elems * 4, s.cuda_stream or None) == 0
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        a.record(s)
        L.disdp_probe_copy(src.data_ptr(), dst.data_ptr(), elems * 4, s.cuda_stream or None)
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del src, dst, slab
    torch.cuda.empty_cache()
    return round(2 * elems * 4 / (ms * 1e-3) / 1e9, 1)


def host_cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo when readable)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def host_threads() -> int:
    """Host threads this process may use, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_baseline(wl, dg, dp, dm, dv, threads=1):
    """The oracle on the first CPU_SAMPLE elements of the same shard for
    CPU_STEPS consecutive steps, each step updating p, m, v and the bf16
    copy in place (buffers read back and allocated before the clock
    starts).  threads > 1 splits the sample into that many contiguous
    chunks, one oracle call per chunk and step on a thread pool (the calls
    release the interpreter lock), as the paper's parameter server spreads
    its CPU Adam over threads.  The oracle's loop streams its arrays once per
    step with no reuse, so its per-element rate does not depend on the
    length once the arrays are far beyond the host's caches (the 2^26-element
    sample is 3.9 GB)."""
    import numpy as np
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    ns = min(CPU_SAMPLE, wl.n)
    gs = []
    for g in dg:
        a = g[:ns].cpu().numpy()
        gs.append(a.view(np.uint16) if wl.gdtype == "bf16" else a)
    p, m, v = (x[:ns].cpu().numpy().copy() for x in (dp, dm, dv))
    p16 = np.zeros(ns, np.uint16)
    hp = hparams(wl)
    mode = oracle.AGG_FIXED if wl.mode == "fixed" else oracle.AGG_FP32
    cuts = [ns * k // threads for k in range(threads + 1)]
    chunks = [(lo, hi) for lo, hi in zip(cuts[:-1], cuts[1:]) if hi > lo]
    pieces = [([g[lo:hi] for g in gs], p[lo:hi], m[lo:hi], v[lo:hi], p16[lo:hi])
              for lo, hi in chunks]

    def one(k, t):
        g, pk, mk, vk, ck = pieces[k]
        oracle.fused_inplace(g, pk, mk, vk, ck, mode=mode, frac_bits=wl.frac_bits, t=t, **hp)

    with ThreadPoolExecutor(max_workers=len(chunks)) as pool:
        t0 = time.perf_counter()
        for t in range(1, CPU_STEPS + 1):
            list(pool.map(lambda k: one(k, t), range(len(chunks))))
        dt = time.perf_counter() - t0
    how = "single-threaded" if len(chunks) == 1 else f"{len(chunks)} threads, one chunk each"
    return {"value": round(ns * CPU_STEPS / dt / 1e9, 5),
            "unit": "G params/s", "cores": len(chunks), "kind": "oracle",
            "sample_fraction": round(ns / wl.n, 4),
            "sample": f"first {ns:,} of the shard's {wl.n:,} elements "
                      f"({100 * ns / wl.n:.1f}%), {CPU_STEPS} consecutive steps, in place, "
                      f"C oracle (gcc -O2), {how}, "
                      f"{dt:.1f} s on {host_cpu_model()} "
                      f"({os.cpu_count()} host threads visible)"}


def run_bench(args):
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth

    wl = workload(args)
    torch.cuda.set_device(0)
    dd.lib()
    hp = hparams(wl)
    stream = torch.cuda.current_stream()
    contrib = "float"
    if args.contributions == "i32":
        # the workers' NICs converted their gradients before the push: the
        # fused call sums int32 contributions (fixed mode at the shard's scale)
        if wl.mode != "fixed":
            raise SystemExit("--contributions i32 needs a fixed-point workload")
        sh = shard(wl.n, wl.W, "i32")
        for w in range(wl.W):
            g = synth.device_grad(wl.wid, 1, w, wl.n, wl.sigma, wl.gdtype,
                                  wl.outlier_frac, wl.outlier_scale)
            dd.quantize(g, sh.grads[w], frac_bits=wl.frac_bits)
            del g
        synth.device_state(wl.wid, wl.n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
        torch.cuda.synchronize()
        dg, dp, dm, dv, d16 = sh.grads, sh.param, sh.m, sh.v, sh.param_bf16
        contrib = "int32"
    else:
        sh = allocate(wl)
        dg, dp, dm, dv, d16 = sh.grads, sh.param, sh.m, sh.v, sh.param_bf16

    def step(t):
        dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                          beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                          step=t, mode=wl.mode, frac_bits=wl.frac_bits,
                          stream=stream)

    # the oracle's sample is taken before any step, on the step-1 inputs
    base = base_mt = None
    if not args.no_cpu_baseline:
        base = cpu_baseline(wl, dg, dp, dm, dv)
        if host_threads() > 1:
            base_mt = cpu_baseline(wl, dg, dp, dm, dv, threads=host_threads())

    t = 0
    for _ in range(args.warmup):
        t += 1
        step(t)
    torch.cuda.synchronize()
    if torch.distributed.is_available() and torch.distributed.is_initialized():
        torch.distributed.barrier()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        t += 1
        ev[k][0].record(stream)
        step(t)
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    if torch.distributed.is_available() and torch.distributed.is_initialized():
        torch.distributed.barrier()
    wall = time.perf_counter() - t0
    kernel_ms = [s.elapsed_time(e) for s, e in ev]
    avg_kernel_ms = float(np.mean(kernel_ms))
    ms_per_step = wall * 1e3 / args.steps

    copy_gbps = None if args.no_copy_ceiling else copy_ceiling_gbps()

    gb = 2 if (wl.gdtype == "bf16" and contrib == "float") else 4
    bpe = dd.algorithmic_bytes_per_element(wl.W, gb)
    algo_bytes = wl.n * bpe
    achieved = algo_bytes / (avg_kernel_ms * 1e-3) / 1e9
    src_hash = kernel_source_hash()
    tr = committed_traffic(wl.name, src_hash)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": None if tr is None else tr["bytes_per_launch"],
                "traffic_GBps": None if tr is None else
                round(tr["bytes_per_launch"] / (avg_kernel_ms * 1e-3) / 1e9, 1),
                "kernel": "vector_kernel (fused aggregate + AdamW)",
                "algorithmic_bytes_per_element": bpe,
                "avg_kernel_ms": round(avg_kernel_ms, 4),
                "median_kernel_ms": round(float(np.median(kernel_ms)), 4),
                "min_kernel_ms": round(float(np.min(kernel_ms)), 4),
                "kernel_source_hash": src_hash,
                "copy_ceiling_GBps": copy_gbps,
                "frac_of_copy_ceiling": None if not copy_gbps else round(achieved / copy_gbps, 4)}
    value = wl.n / (ms_per_step * 1e-3) / 1e9
    line = {
        "metric": "G params/s aggregated+updated (fused W-way reduction + AdamW + bf16 copy)",
        "value": round(value, 3),
        "unit": "G params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if wl.mode == "fp32" else "i32+f32",
        "data": "synthetic",
        "achieved_hbm_tb_s": round(achieved / 1e3, 3),
        "hbm_frac_of_peak": round(achieved / HBM_PEAK_GBPS, 4),
        "config": {"workload": wl.name, "n": wl.n, "W": wl.W,
                   "grad_dtype": wl.gdtype if contrib == "float" else "i32",
                   "aggregation": wl.mode,
                   "frac_bits": wl.frac_bits, "optimizer": "AdamW",
                   "lr": wl.lr, "betas": [wl.beta1, wl.beta2], "eps": wl.eps,
                   "weight_decay": wl.wd, "bf16_copy": True,
                   "shard_memory": ("one physically contiguous allocation" if sh.contiguous
                                    else "one allocation (caching allocator)"),
                   "parallelism": "single GPU, one shard"},
        "roofline": roofline,
        "cpu_baseline": base,
        "cpu_baseline_threads": base_mt,
    }
    print(json.dumps(line), flush=True)


# PCIe 5.0 x16 (MI355X's host interface): 32 GT/s per lane, 16 lanes, per
# direction, before the 128b/130b encoding.
HOST_LINK_PEAK_GBPS = 64.0


def host_link_probe(nbytes=1 << 32, reps=5):
    """Host-link rates on this machine, GB/s per direction, median of `reps`:
    DMA copies between pinned host memory and HBM (torch's copy engine
    path), and the same bytes moved by the library's own kernel reading or
    writing pinned host memory in place (disdp_aggregate of one fp32
    contribution is a copy), the way the fused kernel reaches host state."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    n = nbytes // 4
    host = torch.ones(n, dtype=torch.float32, pin_memory=True)
    dev = torch.empty(n, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()

    def rate(fn):
        fn()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            fn()
            b.record(s)
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        return round(nbytes / (float(np.median(ms)) * 1e-3) / 1e9, 1)

    out = {"dma_h2d_GBps": rate(lambda: dev.copy_(host, non_blocking=True)),
           "dma_d2h_GBps": rate(lambda: host.copy_(dev, non_blocking=True)),
           "kernel_read_host_GBps": rate(lambda: dd.aggregate([host], agg_out_f32=dev)),
           "kernel_write_host_GBps": rate(lambda: dd.aggregate([dev], agg_out_f32=host)),
           "bytes_per_probe": nbytes}
    del host, dev
    torch.cuda.empty_cache()
    return out


def run_host_state(args):
    """Out-of-core shard: p, m, v and the bf16 copy in pinned host DRAM (as
    the paper's parameter server keeps its 12-byte states off the
    accelerator), W contributions in HBM.  The fused kernel streams the
    state over the host link: 12 bytes in and 14 bytes out per element.
    The line also carries the host link's measured rates (host_link_probe)
    and its published peak."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth
    wl = workload(args)
    torch.cuda.set_device(0)
    dd.lib()
    probe = host_link_probe()
    dg = synth.device_grads(wl.wid, 1, wl.W, wl.n, wl.sigma, gdtype=wl.gdtype,
                            outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale)
    dp, dm, dv = synth.device_state(wl.wid, wl.n, wl.p_sigma)
    host = []
    for x in (dp, dm, dv):
        h = torch.empty(wl.n, dtype=torch.float32, pin_memory=True)
        h.copy_(x)
        host.append(h)
    del dp, dm, dv
    h16 = torch.empty(wl.n, dtype=torch.int16, pin_memory=True)
    hp = hparams(wl)
    s = torch.cuda.current_stream()
    t = [0]

    def step():
        t[0] += 1
        dd.aggregate_adam(dg, *host, h16, lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"],
                          eps=hp["eps"], weight_decay=hp["wd"], step=t[0], mode=wl.mode,
                          frac_bits=wl.frac_bits, stream=s)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(s)
        step()
        b.record(s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    h2d = wl.n * 12 / (ms * 1e-3) / 1e9
    d2h = wl.n * 14 / (ms * 1e-3) / 1e9
    print(json.dumps({"metric": "G params/s aggregated+updated, state in pinned host memory",
                      "value": round(wl.n / (wall / args.steps) / 1e9, 3), "unit": "G params/s",
                      "ms_per_step": round(wall * 1e3 / args.steps, 3),
                      "avg_kernel_ms": round(ms, 3), "steps": args.steps,
                      "config": {"workload": wl.name, "n": wl.n, "W": wl.W,
                                 "state": "pinned host (hipHostMalloc), streamed by the kernel",
                                 "contributions": "HBM"},
                      "host_link": {"achieved_GBps_both_directions": round(h2d + d2h, 1),
                                    "h2d_GBps": round(h2d, 1), "d2h_GBps": round(d2h, 1),
                                    "bytes_per_element": {"h2d": 12, "d2h": 14},
                                    "published_peak_GBps_per_direction": HOST_LINK_PEAK_GBPS,
                                    "published_peak_note": "PCIe 5.0 x16, 32 GT/s x 16 lanes",
                                    "frac_of_published_both_directions":
                                        round((h2d + d2h) / (2 * HOST_LINK_PEAK_GBPS), 4),
                                    "probe": probe}}),
          flush=True)


def run_quantize(args):
    """The worker-side format conversion (disdp_quantize) over each of the
    shard's W contributions: s_g bytes read and 4 written per element."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth
    wl = workload(args)
    torch.cuda.set_device(0)
    dd.lib()
    dg = synth.device_grads(wl.wid, 1, wl.W, wl.n, wl.sigma, gdtype=wl.gdtype,
                            outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale)
    out = torch.empty(wl.n, dtype=torch.int32, device="cuda")
    k = wl.frac_bits or 24
    s = torch.cuda.current_stream()
    for w in range(min(args.warmup, wl.W)):
        dd.quantize(dg[w], out, frac_bits=k)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for i, (a, b) in enumerate(ev):
        a.record(s)
        dd.quantize(dg[i % wl.W], out, frac_bits=k)
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    gb = 2 if wl.gdtype == "bf16" else 4
    achieved = wl.n * (gb + 4) / (ms * 1e-3) / 1e9
    print(json.dumps({"metric": "format conversion (disdp_quantize), G elements/s",
                      "value": round(wl.n / (ms * 1e-3) / 1e9, 3), "unit": "G elements/s",
                      "avg_kernel_ms": round(ms, 4), "steps": args.steps,
                      "config": {"workload": wl.name, "n": wl.n, "grad_dtype": wl.gdtype,
                                 "frac_bits": k},
                      "roofline": {"bound": "hbm", "achieved": round(achieved, 1),
                                   "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                   "frac": round(achieved / HBM_PEAK_GBPS, 4),
                                   "algorithmic_bytes_per_element": gb + 4}}), flush=True)


def run_entry(args):
    """One entry point other than the fused call, on the same shard:
    aggregate  -- disdp_aggregate: W contributions read, the aggregate
                  written (fp32, or int32 in fixed mode);
    adam_step  -- disdp_adam_step on an fp32 aggregate: 4 + 12 bytes read,
                  12 + 2 written;
    two_call   -- disdp_aggregate into an fp32 aggregate, then
                  disdp_adam_step on it: the unfused path, 8 bytes per
                  element more than the fused call;
    fused_graph -- the fused call as one HIP graph captured once and
                  replayed every step: a copy node refreshes the step's
                  constants (disdp_step_scalars, written into pinned host
                  memory before each replay) in device memory, then
                  disdp_aggregate_adam_dev reads them.  Same bytes as the
                  fused call; the timed region is the replay."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth
    wl = workload(args)
    torch.cuda.set_device(0)
    dd.lib()
    hp = hparams(wl)
    fixed = wl.mode == "fixed"
    gb = 2 if wl.gdtype == "bf16" else 4
    kw = dict(lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
              weight_decay=hp["wd"])
    def prepare(t):
        pass

    if args.entry == "fused_graph":
        sh = allocate(wl)
        bpe = dd.algorithmic_bytes_per_element(wl.W, gb)
        host = torch.zeros(10, dtype=torch.float32, pin_memory=True)
        dev = torch.zeros(10, dtype=torch.float32, device="cuda")

        def set_step(t):
            sc = dd.step_scalars(step=t, **kw)
            host.copy_(torch.frombuffer(bytearray(sc), dtype=torch.float32))

        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            dev.copy_(host, non_blocking=True)
            dd.aggregate_adam_dev(sh.grads, sh.param, sh.m, sh.v, sh.param_bf16, scalars=dev,
                                  mode=wl.mode, frac_bits=wl.frac_bits)
        torch.cuda.synchronize()

        def prepare(t):
            torch.cuda.synchronize()          # the previous replay has read `host`
            set_step(t)

        def call(t):
            graph.replay()
    elif args.entry == "adam_step":
        sh = shard(wl.n, 1, "f32")
        # an aggregate-sized gradient: one draw at sqrt(W) times the spread
        synth.device_grads(wl.wid, 1, 1, wl.n, wl.sigma * wl.W ** 0.5, out=sh.grads)
        agg = sh.grads[0]
        bpe = dd.algorithmic_bytes_per_element(1, 4)

        def call(t):
            dd.adam_step(agg, sh.param, sh.m, sh.v, sh.param_bf16, step=t, **kw)
    else:
        two = args.entry == "two_call"
        sh = shard(wl.n, wl.W, wl.gdtype, bf16_copy=two,
                               agg_f32=two or not fixed, agg_i32=fixed and not two)
        synth.device_grads(wl.wid, 1, wl.W, wl.n, wl.sigma, gdtype=wl.gdtype,
                           outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale,
                           out=sh.grads)
        if two:
            bpe = dd.algorithmic_bytes_per_element(wl.W, gb, adam=False, agg_f32=True) + \
                dd.algorithmic_bytes_per_element(1, 4)

            def call(t):
                dd.aggregate(sh.grads, mode=wl.mode, frac_bits=wl.frac_bits,
                             agg_out_f32=sh.agg_f32)
                dd.adam_step(sh.agg_f32, sh.param, sh.m, sh.v, sh.param_bf16, step=t, **kw)
        else:
            bpe = dd.algorithmic_bytes_per_element(wl.W, gb, adam=False, agg_f32=not fixed,
                                                   agg_i32=fixed)

            def call(t):
                dd.aggregate(sh.grads, mode=wl.mode, frac_bits=wl.frac_bits,
                             agg_out_f32=None if fixed else sh.agg_f32,
                             agg_out_i32=sh.agg_i32 if fixed else None)
    if args.entry not in ("aggregate", "fused_graph"):
        synth.device_state(wl.wid, wl.n, wl.p_sigma, out=(sh.param, sh.m, sh.v))
    s = torch.cuda.current_stream()
    t = 0
    for _ in range(args.warmup):
        t += 1
        prepare(t)
        call(t)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        t += 1
        prepare(t)
        a.record(s)
        call(t)
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    achieved = wl.n * bpe / (ms * 1e-3) / 1e9
    names = {"aggregate": "disdp_aggregate", "adam_step": "disdp_adam_step",
             "two_call": "disdp_aggregate then disdp_adam_step",
             "fused_graph": "disdp_aggregate_adam_dev replayed as a HIP graph"}
    print(json.dumps({"metric": f"G elements/s ({names[args.entry]})",
                      "value": round(wl.n / (ms * 1e-3) / 1e9, 3), "unit": "G elements/s",
                      "avg_ms": round(ms, 4), "steps": args.steps,
                      "config": {"workload": wl.name, "n": wl.n, "W": wl.W,
                                 "grad_dtype": wl.gdtype, "aggregation": wl.mode},
                      "roofline": {"bound": "hbm", "achieved": round(achieved, 1),
                                   "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                   "frac": round(achieved / HBM_PEAK_GBPS, 4),
                                   "algorithmic_bytes_per_element": bpe}}), flush=True)


def run_layers(args):
    """The 7B/8 shard updated tensor by tensor, as a parameter server walks
    a model: one fused call per parameter tensor of OPT-6.7B (1/8 of each:
    322 sub-ranges of the shard's flat arrays at their natural offsets, 512
    to 25.7M elements, 832M in all), against one call over the same
    elements.  Per step, timed with events on the launch stream and
    interleaved over four rounds: (a) one call; (b) the 322 calls enqueued
    eagerly from Python; (c) the 322 calls (disdp_aggregate_adam_dev)
    captured once as a HIP graph, replayed per step after a copy node
    refreshes the step's constants; (d) one disdp_aggregate_adam_multi call
    (a batch of tensors per launch); (e) that call with the constants in
    device memory, captured once as a HIP graph with its copy node."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth
    wl = synth.WORKLOADS[DEFAULT_WORKLOAD]
    torch.cuda.set_device(0)
    dd.lib()
    sizes = synth.opt_tensor_shards()
    total = sum(sizes)
    if total > wl.n:
        raise SystemExit("the tensor list does not fit the shard")
    sh = allocate(wl)
    hp = hparams(wl)
    kw = dict(lr=hp["lr"], beta1=hp["beta1"], beta2=hp["beta2"], eps=hp["eps"],
              weight_decay=hp["wd"])
    offs = np.concatenate([[0], np.cumsum(sizes)[:-1]]).tolist()

    def cut(o, k):
        return ([g[o:o + k] for g in sh.grads], sh.param[o:o + k], sh.m[o:o + k],
                sh.v[o:o + k], sh.param_bf16[o:o + k])

    whole_args = cut(0, total)
    tensor_args = [cut(o, k) for o, k in zip(offs, sizes)]
    host = torch.zeros(10, dtype=torch.float32, pin_memory=True)
    dev = torch.zeros(10, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        dev.copy_(host, non_blocking=True)
        for g, p, m, v, p16 in tensor_args:
            dd.aggregate_adam_dev(g, p, m, v, p16, scalars=dev)
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()

    def one(t):
        g, p, m, v, p16 = whole_args
        dd.aggregate_adam(g, p, m, v, p16, step=t, **kw)

    def eager(t):
        for g, p, m, v, p16 in tensor_args:
            dd.aggregate_adam(g, p, m, v, p16, step=t, **kw)

    def replay(t):
        graph.replay()

    # the multi-tensor call with the tensors checked and packed once (the
    # library still checks every allocation on every call)
    mstep = dd.MultiTensorStep(tensor_args)

    mgraph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(mgraph, stream=side):
        dev.copy_(host, non_blocking=True)
        dd.aggregate_adam_multi(tensor_args, scalars=dev)
    torch.cuda.synchronize()

    def mreplay(t):
        mgraph.replay()

    def multi(t):
        mstep(step=t, **kw)

    def prepare(t, mode):
        torch.cuda.synchronize()            # a previous replay has read `host`
        if mode in ("graph_per_tensor", "multi_tensor_graph"):
            host.copy_(torch.frombuffer(bytearray(dd.step_scalars(step=t, **kw)),
                                        dtype=torch.float32))

    modes = {"one_call": one, "eager_per_tensor": eager, "graph_per_tensor": replay,
             "multi_tensor_call": multi, "multi_tensor_graph": mreplay}
    res = {k: [] for k in modes}
    host_ms = {k: [] for k in modes}
    t = 0
    for rnd in range(4 + 1):            # pass 0 warms up, passes 1-4 are timed
        for name, fn in modes.items():
            for _ in range(args.steps if rnd else 1):
                t += 1
                prepare(t, name)
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(s)
                h0 = time.perf_counter()
                fn(t)
                h1 = time.perf_counter()
                b.record(s)
                torch.cuda.synchronize()
                if rnd:                      # the first pass warms every mode up
                    res[name].append(a.elapsed_time(b))
                    host_ms[name].append((h1 - h0) * 1e3)
    out = {}
    for name, v in res.items():
        ms = float(np.median(v))
        out[name] = {"ms_per_step": round(ms, 4), "G_params_s": round(total / ms / 1e6, 2),
                     "TBps": round(total * 58 / ms / 1e9, 3),
                     "host_ms_per_step": round(float(np.median(host_ms[name])), 4)}
    print(json.dumps({"metric": "G params/s, a 7B/8 shard updated tensor by tensor",
                      "tensors": len(sizes), "elements": total,
                      "smallest_tensor": min(sizes), "largest_tensor": max(sizes),
                      "config": {"workload": wl.name, "W": wl.W, "grad_dtype": wl.gdtype,
                                 "tensors": "OPT-6.7B parameter tensors, 1/8 of each"},
                      "steps_per_mode": 4 * args.steps, **out}), flush=True)


def _cu_mask_stream(first_cu: int, count: int, total: int):
    """A default-priority stream restricted to CUs [first_cu, first_cu+count)
    (hipExtStreamCreateWithCUMask on torch's HIP runtime), wrapped for torch."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")      # torch's runtime, already loaded
    words = (total + 31) // 32
    mask = (ctypes.c_uint32 * words)()
    for cu in range(first_cu, first_cu + count):
        mask[cu // 32] |= 1 << (cu % 32)
    handle = ctypes.c_void_p()
    rc = hip.hipExtStreamCreateWithCUMask(ctypes.byref(handle), ctypes.c_uint32(words), mask)
    if rc != 0:
        raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
    return torch.cuda.ExternalStream(handle.value), handle, hip


def run_interference(args):
    """The fused call for the 7B / 8 shard on one stream next to a stream
    looping a bf16 GEMM M = N = K = 8192 (seeded N(0, 1) inputs).  Every
    kernel is bracketed by events measured from one common origin, so the
    overlap is observed, not assumed: `gemm_busy_frac` is the share of the
    fused calls' time window during which a GEMM was executing.  With
    --cu-split K the fused call runs on a stream masked to K CUs and the GEMM
    on a stream masked to the other CUs (K = 0: both streams on every CU;
    they are still created with a full CU mask, which gives each its own
    hardware queue).
    --shape lists the library's launch shapes to measure (DISDP_LAUNCH_SHAPE:
    solo, shared).  After each concurrent run the fused steps are run again
    alone from the same start state and must give the same bits on every
    element.  torch.matmul is the
    vendor GEMM, the antagonist only.  Per setting the kernels run in this
    order (the `phases` field), so a kernel trace can be cut into them:
    2 warm-up fused calls and GEMMs interleaved, the fused calls alone, the
    GEMMs alone, the concurrent GEMMs and fused calls, the fused calls again
    alone for the check."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth

    wl = synth.WORKLOADS[DEFAULT_WORKLOAD]
    torch.cuda.set_device(0)
    dd.lib()
    sh = allocate(wl)
    dg, dp, dm, dv, d16 = sh.grads, sh.param, sh.m, sh.v, sh.param_bf16
    hp = hparams(wl)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.seed_for(4, 0, 2000))
    A = torch.randn(8192, 8192, generator=gen, device="cuda").to(torch.bfloat16)
    B = torch.randn(8192, 8192, generator=gen, device="cuda").to(torch.bfloat16)
    C = torch.empty(8192, 8192, device="cuda", dtype=torch.bfloat16)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    t_state = [0]
    med = lambda x: float(np.median(x)) if len(x) else None
    snap = [torch.empty_like(dp) for _ in range(3)]
    conc_out = [torch.empty_like(x) for x in (dp, dm, dv, d16)]

    def fused(stream, t=None):
        if t is None:
            t_state[0] += 1
            t = t_state[0]
        dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                          beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                          step=t, stream=stream)

    def gemm(stream):
        with torch.cuda.stream(stream):
            torch.matmul(A, B, out=C)

    def enqueue(stream, fn, reps):
        ev = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn(stream)
            b.record(stream)
            ev.append((a, b))
        return ev

    def spans(origin, ev):
        return [(origin.elapsed_time(a), origin.elapsed_time(b)) for a, b in ev]

    def check(side, t_first, reps):
        """The concurrent result against the same steps run alone from the
        snapshot, every element (the oracle's check of such a concurrent
        run is the GPU test of the fused call next to a GEMM loop)."""
        for dst, src in zip(conc_out, (dp, dm, dv, d16)):
            dst.copy_(src)
        for dst, src in zip((dp, dm, dv), snap):
            dst.copy_(src)
        torch.cuda.synchronize()
        for k in range(reps):
            fused(side, t_first + k)
        torch.cuda.synchronize()
        same = all(torch.equal(a, b) for a, b in zip(conc_out, (dp, dm, dv, d16)))
        return {"concurrent_equals_solo_all_elements": bool(same)}

    saved_shape = os.environ.get("DISDP_LAUNCH_SHAPE")
    all_ok = True
    try:
        for shape in args.shape.split(","):
            os.environ["DISDP_LAUNCH_SHAPE"] = shape
            for k in [int(x) for x in args.cu_split.split(",")]:
                if k == 0:
                    # both streams on every CU: a CU-masked stream has a hardware
                    # queue of its own, whereas two ordinary streams can share
                    # one and then run one after the other
                    side, h1, hip = _cu_mask_stream(0, n_cu, n_cu)
                    comp, h2, _ = _cu_mask_stream(0, n_cu, n_cu)
                else:
                    side, h1, hip = _cu_mask_stream(0, k, n_cu)
                    comp, h2, _ = _cu_mask_stream(k, n_cu - k, n_cu)
                handles = [(hip, h1), (hip, h2)]
                for _ in range(2):
                    fused(side)
                    gemm(comp)
                torch.cuda.synchronize()
                origin = torch.cuda.Event(enable_timing=True)
                origin.record(torch.cuda.current_stream())
                torch.cuda.synchronize()
                ev = enqueue(side, fused, args.steps)
                torch.cuda.synchronize()
                f_solo = spans(origin, ev)
                n_gemm_solo = 30
                ev = enqueue(comp, gemm, n_gemm_solo)
                torch.cuda.synchronize()
                g_solo = spans(origin, ev)
                fs_ms = med([e - b for b, e in f_solo])
                gs_ms = med([e - b for b, e in g_solo])
                n_gemm = int(3 * args.steps * fs_ms / gs_ms) + 10
                for dst, src in zip(snap, (dp, dm, dv)):
                    dst.copy_(src)
                torch.cuda.synchronize()
                t_first = t_state[0] + 1
                evg = enqueue(comp, gemm, n_gemm)
                evf = enqueue(side, fused, args.steps)
                torch.cuda.synchronize()
                g_conc, f_conc = spans(origin, evg), spans(origin, evf)
                w0, w1 = min(b for b, _ in f_conc), max(e for _, e in f_conc)
                inside = [e - b for b, e in g_conc if b >= w0 and e <= w1]
                busy = sum(max(0.0, min(e, w1) - max(b, w0)) for b, e in g_conc) / (w1 - w0)
                fc_ms = med([e - b for b, e in f_conc])
                gc_ms = med(inside)
                parity = check(side, t_first, args.steps)
                all_ok = all_ok and parity["concurrent_equals_solo_all_elements"]
                line = {
                    "metric": "interference: fused aggregate+AdamW vs a concurrent bf16 GEMM loop",
                    "workload": wl.name, "gemm": "bf16 8192x8192x8192 (torch.matmul)",
                    "launch_shape": shape,
                    "cu_split": None if k == 0 else {"fused_cus": k, "gemm_cus": n_cu - k},
                    "fused_solo_ms": round(fs_ms, 4), "fused_concurrent_ms": round(fc_ms, 4),
                    "fused_slowdown": round(fc_ms / fs_ms, 3),
                    "fused_solo_TBps": round(wl.n * 58 / (fs_ms * 1e-3) / 1e12, 3),
                    "gemm_solo_ms": round(gs_ms, 4),
                    "gemm_concurrent_ms": None if gc_ms is None else round(gc_ms, 4),
                    "gemm_slowdown": None if gc_ms is None else round(gc_ms / gs_ms, 3),
                    "gemm_solo_tflops": round(2 * 8192**3 / (gs_ms * 1e-3) / 1e12, 1),
                    "gemms_inside_fused_window": len(inside),
                    "gemm_busy_frac": round(busy, 3),
                    "fused_reps": args.steps,
                    "phases": {"warmup_fused_and_gemm": 2, "fused_solo": args.steps,
                               "gemm_solo": n_gemm_solo, "gemm_concurrent": n_gemm,
                               "fused_concurrent": args.steps, "fused_check": args.steps},
                    "parity": parity,
                    "streams": "default priority, CU-masked" + (" (full mask: every CU)" if k == 0 else ""),
                }
                print(json.dumps(line), flush=True)
                torch.cuda.synchronize()
                for hip, h in handles:
                    hip.hipStreamDestroy(h)
    finally:
        if saved_shape is None:
            os.environ.pop("DISDP_LAUNCH_SHAPE", None)
        else:
            os.environ["DISDP_LAUNCH_SHAPE"] = saved_shape
    if not all_ok:
        raise SystemExit("interference: a concurrent result differs from the solo run")


def run_copy_probe(args):
    """The plain copy kernel of libdisdp_probe.so over COPY_PROBE_ELEMS fp32
    elements: known bytes read and written per launch, against which the HBM
    byte counters of the fused kernel are scaled."""
    import numpy as np
    import torch
    torch.cuda.set_device(0)
    L = probe_lib()
    src = torch.ones(COPY_PROBE_ELEMS, device="cuda")
    dst = torch.empty_like(src)
    nbytes = COPY_PROBE_ELEMS * 4
    s = torch.cuda.current_stream()
    for _ in range(args.warmup):
        assert L.disdp_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, s.cuda_stream or None) == 0
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record(s)
        assert L.disdp_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, s.cuda_stream or None) == 0
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    assert torch.equal(src[:4096], dst[:4096]) and torch.equal(src[-4096:], dst[-4096:])
    print(json.dumps({"metric": "copy probe", "kernel": "copy16 (libdisdp_probe.so)",
                      "bytes_read_per_launch": nbytes,
                      "bytes_written_per_launch": nbytes, "avg_ms": round(ms, 4),
                      "GBps": round(2 * nbytes / (ms * 1e-3) / 1e9, 1),
                      "launches": args.steps}), flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--n", type=int, default=None,
                    help="sweeps: override the workload's element count")
    ap.add_argument("--W", type=int, default=None,
                    help="sweeps: override the workload's contribution count")
    ap.add_argument("--allocator", choices=["contiguous", "caching"], default="contiguous",
                    help="shard slab: one physically contiguous block, or torch's "
                         "caching allocator")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", action="store_true")
    ap.add_argument("--interference", action="store_true")
    ap.add_argument("--cu-split", default="0,32,64,128",
                    help="interference: CUs given to the fused call (0 = shared)")
    ap.add_argument("--shape", default="solo,shared",
                    help="interference: the library's launch shapes to measure")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--quantize", action="store_true",
                    help="time the format conversion over the shard's contributions")
    ap.add_argument("--host-state", action="store_true",
                    help="p, m, v and the bf16 copy in pinned host memory")
    ap.add_argument("--contributions", choices=["float", "i32"], default="float",
                    help="i32: feed the fused call pre-quantised contributions")
    ap.add_argument("--entry", choices=["fused", "aggregate", "adam_step", "two_call",
                                        "fused_graph", "layers"],
                    default="fused",
                    help="time another entry point on the same shard (not the headline)")
    args = ap.parse_args(argv)
    global CONTIGUOUS
    CONTIGUOUS = args.allocator == "contiguous"
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py measures one GPU: the shard's reduction and optimizer step "
              "run on a single MI355X, and no multi-GPU path is built.",
              file=sys.stderr)
        return 2
    if args.interference:
        run_interference(args)
    elif args.copy_probe:
        run_copy_probe(args)
    elif args.quantize:
        run_quantize(args)
    elif args.host_state:
        run_host_state(args)
    elif args.entry == "layers":
        run_layers(args)
    elif args.entry != "fused":
        run_entry(args)
    else:
        run_bench(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
