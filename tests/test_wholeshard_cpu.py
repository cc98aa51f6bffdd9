"""The whole-shard checker of the full-size GPU tests, exercised on the CPU:
with the oracle's own results as the "device" outputs it reports zero
mismatches over every chunk and thread split, and a single planted bit flip
in any output (first, last or a chunk-boundary element) is counted exactly
once."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import HP, whole_shard_mismatches


def _case(mode, gdtype, n=10_007, W=5, t=3):
    import torch
    gs = synth.host_grads(900, t, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                          outlier_scale=100.0)
    p, m, v = synth.host_state(900, n, mv_sigma=1e-4)
    fixed = mode == "fixed"
    want = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED if fixed else oracle.AGG_FP32,
                        frac_bits=24, t=t, want_agg_i32=fixed, **HP)

    def tt(a):
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a.copy())
    grads = [tt(g) for g in gs]
    pre = [tt(x) for x in (p, m, v)]
    post = {k: tt(want[k]) for k in ("p", "m", "v", "p16")}
    if fixed:
        post["agg_i32"] = tt(want["agg_i32"])
    return grads, pre, post, n


@pytest.mark.parametrize("mode,gdtype", [("fp32", "f32"), ("fp32", "bf16"), ("fixed", "f32")])
def test_checker_finds_no_mismatch_in_the_oracle_itself(mode, gdtype):
    grads, pre, post, n = _case(mode, gdtype)
    for chunk, threads in ((1 << 26, 1), (1000, 3), (4096, 7)):
        bad = whole_shard_mismatches(grads, pre, post, gdtype=gdtype, mode=mode, frac_bits=24,
                                     t=3, hp=HP, chunk=chunk, threads=threads)
        assert bad.pop("elements") == n
        assert set(bad.values()) == {0}, bad


@pytest.mark.parametrize("key", ["p", "m", "v", "p16", "agg_i32"])
@pytest.mark.parametrize("where", [0, 999, 1000, 10_006])
def test_checker_counts_one_planted_bit_flip(key, where):
    grads, pre, post, n = _case("fixed", "f32")
    a = post[key].numpy()
    u = a.view(np.uint16 if a.dtype == np.int16 else np.uint32)
    u[where] ^= 1
    bad = whole_shard_mismatches(grads, pre, post, gdtype="f32", mode="fixed", frac_bits=24,
                                 t=3, hp=HP, chunk=1000, threads=3)
    bad.pop("elements")
    assert bad == {k: (1 if k == key else 0) for k in bad}, bad
