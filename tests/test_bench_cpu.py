"""bench.py's host-side logic, on the CPU: the one-GPU guard, the committed
counter records it reads, and the CPU-baseline leg on a tiny sample."""
import json
import os
import re

import numpy as np
import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env, monkeypatch, capsys):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    assert bench.main(argv) == 2
    assert "one GPU" in capsys.readouterr().err


def test_kernel_source_hash_is_stable():
    h = bench.kernel_source_hash()
    assert re.fullmatch(r"[0-9a-f]{16}", h)
    assert h == bench.kernel_source_hash()


def _records():
    out = []
    for name in sorted(os.listdir(os.path.join(ROOT, "profiles"))):
        if not name.startswith("fused_"):
            continue
        with open(os.path.join(ROOT, "profiles", name)) as f:
            for line in f:
                m = re.match(r"\s*traffic-json:\s*(\{.*\})\s*$", line)
                if m:
                    out.append((name, json.loads(m.group(1))))
    return out


def test_committed_counter_records_are_consistent():
    """Each committed record: read + write = total, the per-element figure is
    total / N of its workload, and the measured HBM bytes are within 2% of the
    algorithmic bytes (a kernel that re-read data would show more)."""
    import paper_2409_00918_amd as dd
    recs = _records()
    assert recs, "no counter summaries under profiles/"
    for name, r in recs:
        wl = synth.WORKLOADS[r["workload"]]
        assert name == f"fused_{wl.name}.md"
        # each of the three is rounded to whole bytes on its own
        assert abs(r["read_bytes_per_launch"] + r["write_bytes_per_launch"]
                   - r["bytes_per_launch"]) <= 2
        assert r["bytes_per_element"] == pytest.approx(r["bytes_per_launch"] / wl.n, abs=1e-3)
        algo = dd.algorithmic_bytes_per_element(wl.W, 2 if wl.gdtype == "bf16" else 4)
        assert abs(r["bytes_per_element"] / algo - 1) < 0.02, name
        # per-dispatch KiB x scale reproduces the byte counts (scales are stored
        # rounded to 5 decimals)
        assert r["fetch_kib_per_dispatch"] * 1024 * r["fetch_scale"] == \
            pytest.approx(r["read_bytes_per_launch"], rel=1e-4)
        assert r["write_kib_per_dispatch"] * 1024 * r["write_scale"] == \
            pytest.approx(r["write_bytes_per_launch"], rel=1e-4)


def test_committed_bench_lines_reproduce_their_roofline():
    """The bench line committed in each fused-kernel summary: achieved =
    N x algorithmic bytes per element / the average kernel time, frac =
    achieved / 8 TB/s, and the G params/s value = N / wall time per step."""
    import paper_2409_00918_amd as dd
    found = 0
    for name in sorted(os.listdir(os.path.join(ROOT, "profiles"))):
        if not name.startswith("fused_"):
            continue
        with open(os.path.join(ROOT, "profiles", name)) as f:
            lines = [json.loads(x) for x in f if x.startswith('{"metric"')]
        for d in lines:
            found += 1
            # a sweep line names its workload with its overrides: name@n=..,W=..
            name, _, over = d["config"]["workload"].partition("@")
            wl = synth.WORKLOADS[name]
            n, W = d["config"]["n"], d["config"]["W"]
            if not over:
                assert (n, W) == (wl.n, wl.W)
            else:
                assert over == f"n={n},W={W}"
            r = d["roofline"]
            bpe = dd.algorithmic_bytes_per_element(W, 2 if wl.gdtype == "bf16" else 4)
            assert r["algorithmic_bytes_per_element"] == bpe
            assert r["achieved"] == pytest.approx(n * bpe / (r["avg_kernel_ms"] * 1e-3) / 1e9,
                                                  rel=2e-4)
            assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-4)
            assert d["value"] == pytest.approx(n / (d["ms_per_step"] * 1e-3) / 1e9, rel=2e-4)
    assert found >= 3


def test_committed_traffic_is_tied_to_the_kernel_source():
    recs = _records()
    wl, h = recs[0][1]["workload"], recs[0][1]["kernel_source_hash"]
    assert bench.committed_traffic(wl, h) is not None
    assert bench.committed_traffic(wl, "0" * 16) is None
    assert bench.committed_traffic("no_such_workload", h) is None


def test_cpu_baseline_leg_on_a_tiny_sample(monkeypatch):
    import torch
    wl = synth.WORKLOADS["tiny_n1M_w4_f32"]
    n = 4099
    monkeypatch.setattr(bench, "CPU_SAMPLE", 2048)
    monkeypatch.setattr(bench, "CPU_STEPS", 2)
    gs = [torch.from_numpy(g) for g in synth.host_grads(wl.wid, 1, wl.W, n, wl.sigma)]
    p, m, v = (torch.from_numpy(x) for x in synth.host_state(wl.wid, n))
    r = bench.cpu_baseline(wl, gs, p, m, v)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["unit"] == "G params/s"
    assert r["value"] > 0 and "first 2,048 of" in r["sample"]
    assert r["sample_fraction"] == round(2048 / wl.n, 4)
    # the sample is read, not modified
    assert np.array_equal(p.numpy(), synth.host_state(wl.wid, n)[0])


def test_cpu_baseline_threads_cover_the_sample_like_one_call(monkeypatch):
    """The threaded leg splits the sample into chunks; since every element is
    independent its final state equals the single call's."""
    import torch
    import oracle
    wl = synth.WORKLOADS["tiny_n1M_w4_f32"]
    n = 5003
    monkeypatch.setattr(bench, "CPU_SAMPLE", 4099)
    monkeypatch.setattr(bench, "CPU_STEPS", 2)
    calls = []
    real = oracle.fused
    real_inplace = oracle.fused_inplace

    def spy(gs, p, m, v, p16, **kw):
        real_inplace(gs, p, m, v, p16, **kw)
        calls.append((kw["t"], p.size, p.copy()))

    monkeypatch.setattr(oracle, "fused_inplace", spy)
    gs = [torch.from_numpy(g) for g in synth.host_grads(wl.wid, 1, wl.W, n, wl.sigma)]
    p, m, v = (torch.from_numpy(x) for x in synth.host_state(wl.wid, n))
    r = bench.cpu_baseline(wl, gs, p, m, v, threads=3)
    assert r["cores"] == 3 and "3 threads" in r["sample"]
    sizes = sorted(s for t, s, _ in calls if t == 1)
    assert sum(sizes) == 4099 and len(sizes) == 3
    # the chunks' step-2 results laid end to end equal one call over the sample
    ref = real([g[:4099].numpy() for g in gs], p[:4099].numpy(), m[:4099].numpy(),
               v[:4099].numpy(), mode=oracle.AGG_FP32, frac_bits=0, t=1,
               **bench.hparams(wl))
    ref = real([g[:4099].numpy() for g in gs], ref["p"], ref["m"], ref["v"],
               mode=oracle.AGG_FP32, frac_bits=0, t=2, **bench.hparams(wl))
    got = [out for t, s, out in calls if t == 2]
    assert len(got) == 3
    # calls are recorded in completion order: look each expected chunk up
    cuts = [4099 * k // 3 for k in range(4)]
    want = [ref["p"][lo:hi] for lo, hi in zip(cuts[:-1], cuts[1:])]
    for w in want:
        assert any(g.size == w.size and np.array_equal(g, w) for g in got)


def test_workload_overrides_for_sweeps():
    """--n / --W give a renamed variant of the workload (so no committed
    counter record of the real workload is attached to it); without them
    the workload is the named one itself."""
    import argparse
    base = bench.workload(argparse.Namespace(workload="opt7b_shard8_w8_f32", n=None, W=None))
    assert base is synth.WORKLOADS["opt7b_shard8_w8_f32"]
    v = bench.workload(argparse.Namespace(workload="opt13b_shard16_w16_bf16", n=200_000_000,
                                          W=24))
    assert (v.n, v.W, v.gdtype, v.mode) == (200_000_000, 24, "bf16", "fp32")
    assert v.name != base.name and v.name not in synth.WORKLOADS
    assert bench.committed_traffic(v.name, bench.kernel_source_hash()) is None
