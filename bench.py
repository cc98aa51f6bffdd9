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

Prints one JSON line.  ``roofline`` prices the kernel against HBM bandwidth
(8 TB/s) with algorithmic bytes (each byte the call must move, counted once);
``traffic`` is the HBM byte count read from committed rocprofv3 counters when
they were taken on the current kernel source, else null.  ``cpu_baseline``
times the CPU oracle (single thread) on a bounded sample of the same shard.
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
                  "paper_2409_00918_amd/csrc/disdp_api.cpp",
                  "paper_2409_00918_amd/build.py"]
CPU_SAMPLE = 1 << 26            # elements of the shard the oracle is timed on
CPU_STEPS = 12
COPY_PROBE_ELEMS = 1 << 30      # fp32 elements moved by the copy probe (4 GiB each way)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def committed_traffic(workload: str, src_hash: str):
    """HBM bytes per launch from the committed counter summary of this
    workload, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"counters_fused_{workload}.md")
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


def allocate(wl):
    import torch
    import synth
    dg = synth.device_grads(wl.wid, 1, wl.W, wl.n, wl.sigma, gdtype=wl.gdtype,
                            outlier_frac=wl.outlier_frac,
                            outlier_scale=wl.outlier_scale)
    dp, dm, dv = synth.device_state(wl.wid, wl.n, wl.p_sigma)
    d16 = torch.empty(wl.n, dtype=torch.int16, device="cuda")
    return dg, dp, dm, dv, d16


def copy_ceiling_gbps(elems=1 << 30, reps=10):
    """Bytes moved per second by a plain device copy (torch's copy kernel)
    of `elems` fp32 elements on this GPU, measured now: the practical HBM
    ceiling the fused kernel is compared with, next to the datasheet peak."""
    import numpy as np
    import torch
    src = torch.ones(elems, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        a.record(s)
        dst.copy_(src)
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del src, dst
    torch.cuda.empty_cache()
    return round(2 * elems * 4 / (ms * 1e-3) / 1e9, 1)


def cpu_baseline(wl, dg, dp, dm, dv):
    """The oracle, single-threaded, on the first CPU_SAMPLE elements of the
    same shard for CPU_STEPS consecutive steps."""
    import numpy as np
    import oracle
    ns = min(CPU_SAMPLE, wl.n)
    gs = []
    for g in dg:
        a = g[:ns].cpu().numpy()
        gs.append(a.view(np.uint16) if wl.gdtype == "bf16" else a)
    p, m, v = (x[:ns].cpu().numpy() for x in (dp, dm, dv))
    hp = hparams(wl)
    mode = oracle.AGG_FIXED if wl.mode == "fixed" else oracle.AGG_FP32
    t0 = time.perf_counter()
    for t in range(1, CPU_STEPS + 1):
        out = oracle.fused(gs, p, m, v, mode=mode, frac_bits=wl.frac_bits, t=t, **hp)
        p, m, v = out["p"], out["m"], out["v"]
    dt = time.perf_counter() - t0
    return {"value": round(ns * CPU_STEPS / dt / 1e9, 5),
            "unit": "G params/s", "cores": 1, "kind": "oracle",
            "sample": f"first {ns} elements of the shard, {CPU_STEPS} consecutive "
                      f"steps, single-threaded C oracle (gcc -O2), "
                      f"{dt:.1f} s on {platform.processor() or platform.machine()} "
                      f"({os.cpu_count()} host threads visible)"}


def run_bench(args):
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth

    wl = synth.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    dd.lib()
    dg, dp, dm, dv, d16 = allocate(wl)
    hp = hparams(wl)
    stream = torch.cuda.current_stream()

    def step(t):
        dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                          beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                          step=t, mode=wl.mode, frac_bits=wl.frac_bits,
                          stream=stream)

    # the oracle's sample is taken before any step, on the step-1 inputs
    base = None if args.no_cpu_baseline else cpu_baseline(wl, dg, dp, dm, dv)

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

    gb = 2 if wl.gdtype == "bf16" else 4
    bpe = dd.algorithmic_bytes_per_element(wl.W, gb)
    algo_bytes = wl.n * bpe
    achieved = algo_bytes / (avg_kernel_ms * 1e-3) / 1e9
    src_hash = kernel_source_hash()
    tr = committed_traffic(wl.name, src_hash)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": None if tr is None else tr["bytes_per_launch"],
                "kernel": "vector_kernel (fused aggregate + AdamW)",
                "algorithmic_bytes_per_element": bpe,
                "avg_kernel_ms": round(avg_kernel_ms, 4),
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
                   "grad_dtype": wl.gdtype, "aggregation": wl.mode,
                   "frac_bits": wl.frac_bits, "optimizer": "AdamW",
                   "lr": wl.lr, "betas": [wl.beta1, wl.beta2], "eps": wl.eps,
                   "weight_decay": wl.wd, "bf16_copy": True,
                   "parallelism": "single GPU, one shard"},
        "roofline": roofline,
        "cpu_baseline": base,
    }
    print(json.dumps(line), flush=True)


def run_interference(args):
    """The fused call for the 7B / 8 shard on a side stream next to a compute
    stream looping a bf16 GEMM M = N = K = 8192 (seeded N(0, 1) inputs); the
    slowdown of each against its solo time.  torch.matmul is the vendor GEMM,
    used only as the antagonist."""
    import numpy as np
    import torch
    import paper_2409_00918_amd as dd
    import synth

    wl = synth.WORKLOADS[DEFAULT_WORKLOAD]
    torch.cuda.set_device(0)
    dd.lib()
    dg, dp, dm, dv, d16 = allocate(wl)
    hp = hparams(wl)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.seed_for(4, 0, 2000))
    A = torch.randn(8192, 8192, generator=gen, device="cuda").to(torch.bfloat16)
    B = torch.randn(8192, 8192, generator=gen, device="cuda").to(torch.bfloat16)
    C = torch.empty(8192, 8192, device="cuda", dtype=torch.bfloat16)
    side = torch.cuda.Stream()
    comp = torch.cuda.Stream()
    t_state = [0]

    def fused_on(stream):
        t_state[0] += 1
        dd.aggregate_adam(dg, dp, dm, dv, d16, lr=hp["lr"], beta1=hp["beta1"],
                          beta2=hp["beta2"], eps=hp["eps"], weight_decay=hp["wd"],
                          step=t_state[0], stream=stream)

    def timed(stream, fn, reps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        with torch.cuda.stream(stream):
            for s, e in ev:
                s.record(stream)
                fn(stream)
                e.record(stream)
        return ev

    def gemm(stream):
        torch.matmul(A, B, out=C)

    reps_f = args.steps
    # warm both up
    for _ in range(2):
        fused_on(side)
        with torch.cuda.stream(comp):
            gemm(comp)
    torch.cuda.synchronize()
    ev = timed(side, fused_on, reps_f)
    torch.cuda.synchronize()
    fused_solo = [s.elapsed_time(e) for s, e in ev]
    ev = timed(comp, gemm, 20)
    torch.cuda.synchronize()
    gemm_solo = [s.elapsed_time(e) for s, e in ev]
    # concurrent: enough GEMMs to cover three times the fused calls
    n_gemm = int(3 * reps_f * np.median(fused_solo) / np.median(gemm_solo)) + 10
    evg = timed(comp, gemm, n_gemm)
    evf = timed(side, fused_on, reps_f)
    torch.cuda.synchronize()
    gemm_conc = [s.elapsed_time(e) for s, e in evg]
    fused_conc = [s.elapsed_time(e) for s, e in evf]
    # GEMMs that ran while the fused calls were in flight: the middle third
    lo, hi = n_gemm // 3, 2 * n_gemm // 3
    med = lambda x: float(np.median(x))
    line = {
        "metric": "interference: slowdown of the fused call and of a bf16 GEMM when run concurrently",
        "workload": wl.name, "gemm": "bf16 8192x8192x8192 (torch.matmul)",
        "fused_solo_ms": round(med(fused_solo), 4),
        "fused_concurrent_ms": round(med(fused_conc), 4),
        "fused_slowdown": round(med(fused_conc) / med(fused_solo), 3),
        "gemm_solo_ms": round(med(gemm_solo), 4),
        "gemm_concurrent_ms": round(med(gemm_conc[lo:hi]), 4),
        "gemm_slowdown": round(med(gemm_conc[lo:hi]) / med(gemm_solo), 3),
        "gemm_solo_tflops": round(2 * 8192**3 / (med(gemm_solo) * 1e-3) / 1e12, 1),
        "fused_reps": reps_f, "gemm_reps": n_gemm,
        "streams": "default priority, separate streams",
    }
    print(json.dumps(line), flush=True)


def run_copy_probe(args):
    """A plain device-to-device copy of COPY_PROBE_ELEMS fp32 elements
    (torch's elementwise copy kernel): known bytes read and written per
    launch, against which the HBM byte counters of the fused kernel are
    scaled."""
    import numpy as np
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(COPY_PROBE_ELEMS, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record(s)
        dst.copy_(src)
        b.record(s)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    nbytes = COPY_PROBE_ELEMS * 4
    print(json.dumps({"metric": "copy probe", "bytes_read_per_launch": nbytes,
                      "bytes_written_per_launch": nbytes, "avg_ms": round(ms, 4),
                      "GBps": round(2 * nbytes / (ms * 1e-3) / 1e9, 1),
                      "launches": args.steps}), flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", action="store_true")
    ap.add_argument("--interference", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    args = ap.parse_args(argv)
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
    else:
        run_bench(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
