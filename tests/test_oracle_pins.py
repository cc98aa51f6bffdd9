"""Pins of the CPU oracle against what the paper and mathematics fix.

No GPU.  Nothing here re-types the oracle's C code: each test checks it
against something independent of it --
  * exact rational / 320-bit arithmetic (Python ``fractions``, ``mpmath``)
    with error bounds derived from binary32 rounding (running error analysis),
  * closed forms (t = 1 Adam step, zero-gradient shrinkage, identical
    contributions, ordering counterexamples),
  * library routines (``torch``'s bf16 conversion, ``torch.optim.AdamW``),
  * invariants (worker permutation, chunking, composition),
  * the byte and flop accounting the paper prints in Table III.

Paper: arXiv 2409.00918.  Aggregation = the switch's W-way sum (Section III-A,
III-C); integer format = the SmartNIC format-conversion unit (Section III-B);
optimizer = step 5 of the parameter server's backward stage (Section III-D).
"""
import fractions
import os

import mpmath
import numpy as np
import pytest
import torch

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))

I32_MAX, I32_MIN = 2**31 - 1, -(2**31)
mp = mpmath.mp
mp.prec = 320
U = mpmath.mpf(2) ** -24          # unit roundoff, binary32, round to nearest
ETA = mpmath.mpf(2) ** -150        # absolute rounding bound in the subnormal range


def f32(x):
    return np.float32(x)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


# ----------------------------------------------------------------------------
# environment
# ----------------------------------------------------------------------------
def test_host_fpu_keeps_denormals():
    assert oracle.fp_env_ok()


# ----------------------------------------------------------------------------
# bf16 conversions (the 2-byte parameter copy)
# ----------------------------------------------------------------------------
def test_bf16_widening_exhaustive_against_torch():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_to_f32(h)
    ref = torch.from_numpy(h.view(np.int16).copy()).view(torch.bfloat16) \
        .float().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(bits(ours[~nan]), bits(ref[~nan]))


def test_bf16_round_trip_exhaustive():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    keep = (h & 0x7FFF) <= 0x7F80          # finite and +-inf
    f = oracle.bf16_to_f32(h[keep])
    assert np.array_equal(oracle.bf16_rne(f), h[keep])


def test_bf16_rne_matches_torch_including_ties():
    rng = np.random.default_rng(11)
    b = rng.integers(0, 2**32, 120_000, dtype=np.uint64).astype(np.uint32)
    b[0::4] = (b[0::4] & 0xFFFF0000) | 0x8000     # exact ties
    b[1::8] = (b[1::8] & 0xFFFF0000) | 0x7FFF     # just below a tie
    b[3::8] = (b[3::8] & 0xFFFF0000) | 0x8001     # just above a tie
    x = b.view(np.float32)
    x = x[~np.isnan(x)]
    specials = np.array([0.0, -0.0, np.inf, -np.inf, 3.4028235e38,
                         -3.4028235e38, 1e-45, -1e-45, 1.1754942e-38,
                         3.3961776e38, 3.3961778e38], dtype=np.float32)
    x = np.concatenate([x, specials])
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_rne(x), ref)


def test_bf16_rne_tie_cases_by_hand():
    # 1 + 2^-8 lies halfway between bf16 1.0 and 1 + 2^-7: ties go to even (1.0)
    assert oracle.bf16_rne(f32(1 + 2**-8))[0] == 0x3F80
    # 1 + 3*2^-8 is halfway between 1+2^-7 (odd) and 1+2^-6 (even): rounds up
    assert oracle.bf16_rne(f32(1 + 3 * 2**-8))[0] == 0x3F82
    # the largest finite fp32 rounds to +inf in bf16
    assert oracle.bf16_rne(f32(3.4028235e38))[0] == 0x7F80


def test_bf16_nan_keeps_sign_and_is_quiet():
    pos = np.array([0x7FC00000, 0x7F800001, 0x7FFFFFFF], np.uint32).view(np.float32)
    neg = np.array([0xFFC00000, 0xFF800001], np.uint32).view(np.float32)
    assert set(oracle.bf16_rne(pos).tolist()) == {0x7FC0}
    assert set(oracle.bf16_rne(neg).tolist()) == {0xFFC0}


# ----------------------------------------------------------------------------
# format conversion: quantise to int32 at 2^k
# ----------------------------------------------------------------------------
def exact_quantize(x, k):
    """Round x*2^k to the nearest integer (ties to even) in exact rational
    arithmetic, then saturate to int32; NaN -> 0."""
    x = float(x)
    if np.isnan(x):
        return 0
    if np.isinf(x):
        return I32_MAX if x > 0 else I32_MIN
    q = round(fractions.Fraction(x) * 2**k)    # Fraction.__round__: half-even
    return max(I32_MIN, min(I32_MAX, q))


@pytest.mark.parametrize("k", [0, 1, 8, 16, 24, 30])
def test_quantize_matches_exact_rational(k):
    rng = np.random.default_rng(100 + k)
    xs = [rng.standard_normal(3000).astype(np.float32) * f32(s)
          for s in (1e-9, 1e-4, 1e-1, 10.0, 3e3)]
    # ties at small integers, both parities, both signs
    n = np.arange(-40, 40, dtype=np.float64)
    ties = ((n + 0.5) * 2.0**-k).astype(np.float32)
    # around the int32 range ends
    edge = np.array([2.0**31, -2.0**31, 2.0**31 - 128, -2.0**31 + 128,
                     2.0**31 + 256, -2.0**31 - 256, 2.0**40, -2.0**40],
                    np.float64) * 2.0**-k
    special = np.array([0.0, -0.0, 1e-45, -1e-45, 1.1754942e-38, np.inf,
                        -np.inf, 3.4028235e38, -3.4028235e38], np.float32)
    x = np.concatenate(xs + [ties, edge.astype(np.float32), special])
    got = oracle.quantize(x, k)
    want = np.array([exact_quantize(v, k) for v in x], dtype=np.int64)
    assert np.array_equal(got.astype(np.int64), want)


def test_quantize_nan_is_zero():
    nan = np.array([0x7FC00000, 0xFFC00000, 0x7F800001], np.uint32).view(np.float32)
    assert oracle.quantize(nan, 24).tolist() == [0, 0, 0]


# ----------------------------------------------------------------------------
# W-way aggregation, fixed-point mode (bit-exact)
# ----------------------------------------------------------------------------
def exact_aggregate_fixed(gs, k):
    ai, af = [], []
    for i in range(gs[0].size):
        s = sum(exact_quantize(g[i], k) for g in gs)     # Python int: exact
        a = max(I32_MIN, min(I32_MAX, s))
        ai.append(a)
        # int32 -> binary32 is one rounding (float(a) is exact in binary64);
        # scaling by 2^-k is then exact
        af.append(np.ldexp(np.float32(float(a)), -k))
    return np.array(ai, np.int32), np.array(af, np.float32)


@pytest.mark.parametrize("W,k", [(1, 24), (3, 24), (8, 24), (16, 20), (8, 30), (5, 0)])
def test_aggregate_fixed_matches_exact(W, k):
    n = 1500
    gs = synth.host_grads(7, W, W, n, 1e-4, outlier_frac=0.05,
                          outlier_scale=1e5)
    # plant saturating contributions of both signs in a few elements
    gs[0][:7] = np.float32(1e30)
    gs[-1][3:10] = np.float32(-1e30)
    got_i, got_f = oracle.aggregate_fixed(gs, k)
    want_i, want_f = exact_aggregate_fixed(gs, k)
    assert np.array_equal(got_i, want_i)
    assert np.array_equal(bits(got_f), bits(want_f))


def test_aggregate_fixed_bf16_contributions():
    gs = synth.host_grads(8, 0, 6, 700, 1e-3, gdtype="bf16")
    got_i, _ = oracle.aggregate_fixed(gs, 24)
    widened = [oracle.bf16_to_f32(g) for g in gs]
    want_i, _ = exact_aggregate_fixed(widened, 24)
    assert np.array_equal(got_i, want_i)


def test_aggregate_fixed_saturation_is_per_contribution_then_sum():
    # +inf and -inf saturate to INT32_MAX and INT32_MIN and cancel to -1 in
    # the 64-bit sum; a plain int32 sum of the saturated values would wrap.
    gs = [np.array([np.inf], np.float32), np.array([-np.inf], np.float32),
          np.array([5 * 2.0**-24], np.float32)]
    ai, af = oracle.aggregate_fixed(gs, 24)
    assert ai[0] == -1 + 5
    # four maximal contributions overflow int32 and clamp once
    gs = [np.array([1e9], np.float32)] * 4
    ai, _ = oracle.aggregate_fixed(gs, 24)
    assert ai[0] == I32_MAX


def test_aggregate_fixed_is_worker_order_independent():
    W = 9
    gs = synth.host_grads(9, 0, W, 2000, 1e-4, outlier_frac=0.02,
                          outlier_scale=1e6)
    ref_i, ref_f = oracle.aggregate_fixed(gs, 24)
    rng = np.random.default_rng(3)
    for _ in range(4):
        perm = rng.permutation(W)
        ai, af = oracle.aggregate_fixed([gs[j] for j in perm], 24)
        assert np.array_equal(ai, ref_i)
        assert np.array_equal(bits(af), bits(ref_f))


def test_aggregate_fixed_identical_contributions():
    g = synth.host_grads(10, 0, 1, 3000, 1e-3)[0]
    q = oracle.quantize(g, 24).astype(np.int64)
    for W in (1, 2, 7, 16, 64):
        ai, _ = oracle.aggregate_fixed([g] * W, 24)
        assert np.array_equal(ai.astype(np.int64),
                              np.clip(W * q, I32_MIN, I32_MAX))


# ----------------------------------------------------------------------------
# W-way aggregation, fp32 mode
# ----------------------------------------------------------------------------
def short_significand(n, bits_kept, seed):
    """fp32 values whose significand has at most `bits_kept` bits."""
    rng = np.random.default_rng(seed)
    mant = rng.integers(2**(bits_kept - 1), 2**bits_kept, n).astype(np.float64)
    e = rng.integers(-30, 0, n)
    sign = rng.choice([-1.0, 1.0], n)
    return (sign * np.ldexp(mant, e - bits_kept)).astype(np.float32)


@pytest.mark.parametrize("W", [1, 2, 3, 4, 8, 16, 64])
def test_aggregate_identical_contributions_sum_to_W_g(W):
    # With at most 24 - ceil(log2 W) significant bits every partial sum j*g
    # (j <= W) is representable, so the fp32 sum is exactly W*g.
    kept = 24 - int(np.ceil(np.log2(W))) if W > 1 else 24
    g = short_significand(4000, kept, seed=W)
    agg = oracle.aggregate_f32([g] * W)
    want = (g.astype(np.float64) * W).astype(np.float32)   # exact product
    assert np.array_equal(bits(agg), bits(want))


def test_aggregate_order_is_worker_0_first():
    a, b = f32(1.0), f32(2.0**-24)
    # 1 + 2^-24 is a tie and rounds back to 1, twice
    fwd = oracle.aggregate_f32([np.array([a]), np.array([b]), np.array([b])])
    # 2^-24 + 2^-24 = 2^-23 is exact, and 2^-23 + 1 is representable
    rev = oracle.aggregate_f32([np.array([b]), np.array([b]), np.array([a])])
    assert fwd[0] == f32(1.0)
    assert rev[0] == f32(1.0 + 2.0**-23)


@pytest.mark.parametrize("W,gdtype", [(2, "f32"), (5, "f32"), (8, "f32"),
                                      (16, "bf16"), (33, "f32")])
def test_aggregate_within_recursive_summation_bound(W, gdtype):
    # |fl(sum) - sum| <= gamma_{W-1} * sum |g_w|  (recursive summation)
    n = 3000
    gs = synth.host_grads(11, W, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                          outlier_scale=100.0)
    agg = oracle.aggregate_f32(gs)
    vals = [oracle.bf16_to_f32(g) if gdtype == "bf16" else g for g in gs]
    exact = [sum(fractions.Fraction(float(v[i])) for v in vals) for i in range(n)]
    absum = [sum(abs(fractions.Fraction(float(v[i]))) for v in vals) for i in range(n)]
    u = fractions.Fraction(1, 2**24)
    gamma = (W - 1) * u / (1 - (W - 1) * u)
    tiny = fractions.Fraction(W, 2**150)
    for i in range(n):
        err = abs(fractions.Fraction(float(agg[i])) - exact[i])
        assert err <= gamma * absum[i] + tiny, i


def test_aggregate_bf16_widening_is_exact():
    gs = synth.host_grads(12, 0, 4, 2000, 1e-2, gdtype="bf16")
    a = oracle.aggregate_f32(gs)
    b = oracle.aggregate_f32([oracle.bf16_to_f32(g) for g in gs])
    assert np.array_equal(bits(a), bits(b))


# ----------------------------------------------------------------------------
# step scalars
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("b1,b2", [(0.9, 0.95), (0.9, 0.999), (0.5, 0.5), (0.0, 0.0)])
def test_scalars_bias_corrections(b1, b2):
    lr, wd = f32(1e-4), f32(0.1)
    b1, b2 = f32(b1), f32(b2)
    s1 = oracle.scalars(lr, b1, b2, wd, 1)
    assert s1[0] == b1 and s1[2] == b2
    assert s1[1] == f32(1.0) - b1 and s1[3] == f32(1.0) - b2
    # at t = 1 the bias correction equals 1 - beta exactly
    assert s1[4] == s1[1] and s1[5] == s1[3]
    for t in (1, 2, 3, 5, 10, 100, 1000, 10**6):
        s = oracle.scalars(lr, b1, b2, wd, t)
        for got, beta in ((s[4], b1), (s[5], b2)):
            exact = 1 - mpmath.mpf(float(beta)) ** t
            assert abs(mpmath.mpf(float(got)) - exact) <= U * abs(exact) + mpmath.mpf(2)**-50
        exact_decay = 1 - mpmath.mpf(float(lr)) * mpmath.mpf(float(wd))
        assert abs(mpmath.mpf(float(s[6])) - exact_decay) <= U * exact_decay
    assert oracle.scalars(lr, f32(0.9), f32(0.95), wd, 10**6)[4] == f32(1.0)


# ----------------------------------------------------------------------------
# Adam with decoupled weight decay
# ----------------------------------------------------------------------------
HP = dict(lr=f32(1e-4), beta1=f32(0.9), beta2=f32(0.95), eps=f32(1e-8),
          wd=f32(0.1))


def test_adamw_first_step_closed_form():
    # t = 1, m = v = 0, wd = 0: m^ = g and v^ = g^2 in exact arithmetic, so
    # the update is -lr * g / (|g| + eps).
    n = 5000
    rng = np.random.default_rng(21)
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-12, 2, n))).astype(np.float32)
    g[:4] = [1e-9, -1e-9, 1e-7, -3.0]
    p = rng.standard_normal(n).astype(np.float32) * f32(0.02)
    z = np.zeros(n, np.float32)
    lr, eps = HP["lr"], HP["eps"]
    p1, _, _, _ = oracle.adamw(g, p, z, z, lr=lr, beta1=HP["beta1"],
                               beta2=HP["beta2"], eps=eps, wd=f32(0.0), t=1)
    g64 = g.astype(np.float64)
    want = p.astype(np.float64) - float(lr) * g64 / (np.abs(g64) + float(eps))
    u = 2.0**-24
    bound = u * np.abs(want) + 8 * u * float(lr) + 2.0**-149
    assert np.all(np.abs(p1.astype(np.float64) - want) <= bound)
    # |g| >> eps: the step is -lr * sign(g), up to eps/|g| relative, a few
    # ulp of lr, and the rounding of p itself
    big = np.abs(g) > 1e-3
    step = (p1.astype(np.float64) - p.astype(np.float64))[big]
    tol = u * np.abs(p1[big]) + 8 * u * float(lr) + float(lr) * 1e-5
    assert np.all(np.abs(step + float(lr) * np.sign(g64[big])) <= tol)


def test_adamw_zero_gradient_is_pure_decoupled_decay():
    n = 4000
    p = synth.host_state(31, n)[0]
    z = np.zeros(n, np.float32)
    decay = oracle.scalars(HP["lr"], HP["beta1"], HP["beta2"], HP["wd"], 1)[6]
    pt, m, v = p.copy(), z.copy(), z.copy()
    for t in range(1, 11):
        prev = pt.copy()
        pt, m, v, p16 = oracle.adamw(z, pt, m, v, t=t, **HP)
        # m and v stay exactly zero, the update is exactly zero, and the
        # parameter is multiplied by the rounded decay factor
        assert not m.any() and not v.any()
        assert np.array_equal(bits(pt), bits(prev * decay))
        # against the real closed form p0 (1 - lr wd)^t
        closed = p.astype(np.float64) * (1 - float(HP["lr"]) * float(HP["wd"])) ** t
        assert np.all(np.abs(pt - closed) <= 2.0 * (t + 1) * 2.0**-24 * np.abs(closed))


class E:
    """Running error analysis: an exact real value and a bound on how far a
    binary32 evaluation of the same expression can lie from it."""
    __slots__ = ("x", "e")

    def __init__(self, x, e=0):
        self.x = mpmath.mpf(x)
        self.e = mpmath.mpf(e)

    @staticmethod
    def rounded(x, e):
        # the result carries the propagated error e plus one rounding
        return E(x, e + U * (abs(x) + e) + ETA)

    def __add__(a, b):
        return E.rounded(a.x + b.x, a.e + b.e)

    def __sub__(a, b):
        return E.rounded(a.x - b.x, a.e + b.e)

    def __mul__(a, b):
        return E.rounded(a.x * b.x, abs(a.x) * b.e + abs(b.x) * a.e + a.e * b.e)

    def __truediv__(a, b):
        assert b.e < abs(b.x)
        q = a.x / b.x
        return E.rounded(q, (a.e + abs(q) * b.e) / (abs(b.x) - b.e))

    def sqrt(a):
        r = mpmath.sqrt(a.x)
        prop = mpmath.sqrt(a.e)
        if a.x > 0:
            prop = min(prop, a.e / r)
        return E.rounded(r, prop)


def adamw_exact_with_bound(agg, p, m, v, lr, beta1, beta2, eps, wd, t, scale):
    """The real-valued AdamW step on binary32 inputs, plus the running error
    bound of a binary32 evaluation.  Hyperparameters are the exact values of
    the binary32 numbers the caller passes."""
    X = lambda f: E(float(f))
    b1, b2 = X(beta1), X(beta2)
    one = E(1)
    omb1, omb2 = one - b1, one - b2
    bc1x = 1 - mpmath.mpf(float(beta1)) ** t
    bc2x = 1 - mpmath.mpf(float(beta2)) ** t
    small = mpmath.mpf(2) ** -50           # binary64 evaluation before rounding
    bc1 = E(bc1x, U * abs(bc1x) + small)
    bc2 = E(bc2x, U * abs(bc2x) + small)
    dx = 1 - mpmath.mpf(float(lr)) * mpmath.mpf(float(wd))
    decay = E(dx, U * abs(dx) + small)
    g = X(agg) * X(scale)
    m1 = b1 * X(m) + omb1 * g
    v1 = b2 * X(v) + omb2 * (g * g)
    mh = m1 / bc1
    vh = v1 / bc2
    d = vh.sqrt() + X(eps)
    p1 = X(p) * decay - X(lr) * (mh / d)
    return p1, m1, v1


@pytest.mark.parametrize("t", [1, 2, 3, 5, 10, 1000])
@pytest.mark.parametrize("hp", [dict(HP), dict(HP, lr=f32(3e-4)),
                                dict(HP, beta2=f32(0.999), wd=f32(0.0)),
                                dict(HP, eps=f32(1e-6), wd=f32(0.5))])
def test_adamw_within_running_error_bound_of_exact(t, hp):
    n = 160
    rng = np.random.default_rng(1000 * t + int(hp["lr"] * 1e6))
    agg = (rng.standard_normal(n) * np.exp(rng.uniform(-16, 3, n))).astype(np.float32)
    agg[:6] = [0.0, -0.0, 1e-30, -2e-38, 50.0, -7e-3]
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = (rng.standard_normal(n) * 1e-3).astype(np.float32) ** 2
    m[:2] = 0.0
    v[:2] = 0.0
    scale = f32(1.0) if t != 3 else f32(0.125)
    p1, m1, v1, p16 = oracle.adamw(agg, p, m, v, t=t, grad_scale=scale, **hp)
    for i in range(n):
        ep, em, ev = adamw_exact_with_bound(agg[i], p[i], m[i], v[i], hp["lr"],
                                            hp["beta1"], hp["beta2"],
                                            hp["eps"], hp["wd"], t, scale)
        for got, ref in ((p1[i], ep), (m1[i], em), (v1[i], ev)):
            assert abs(mpmath.mpf(float(got)) - ref.x) <= ref.e, (i, got, ref.x, ref.e)
    assert np.array_equal(p16, oracle.bf16_rne(p1))


def _torch_reference(opt_cls, steps, n, wd, seed):
    """Each step, torch's optimizer starts from the oracle's previous state
    (p, m, v, step count), so every step compares the two on equal inputs."""
    rng = np.random.default_rng(seed)
    p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    grads = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(steps)]
    po, mo, vo = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
    hp = dict(HP, wd=f32(wd))
    for t, g in enumerate(grads, start=1):
        tp = torch.nn.Parameter(torch.from_numpy(po.copy()))
        opt = opt_cls([tp], lr=float(HP["lr"]),
                      betas=(float(HP["beta1"]), float(HP["beta2"])),
                      eps=float(HP["eps"]), weight_decay=float(wd),
                      foreach=False)
        if t > 1:
            opt.state[tp] = {"step": torch.tensor(float(t - 1)),
                             "exp_avg": torch.from_numpy(mo.copy()),
                             "exp_avg_sq": torch.from_numpy(vo.copy())}
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        m_prev, v_prev = mo.copy(), vo.copy()
        po, mo, vo, _ = oracle.adamw(g, po, mo, vo, t=t, **hp)
        st = opt.state[tp]
        yield (t, g, m_prev, v_prev, po, mo, vo, tp.detach().numpy().copy(),
               st["exp_avg"].numpy().copy(), st["exp_avg_sq"].numpy().copy())


def test_adamw_matches_torch_adamw():
    # Same real formula, different binary32 operation order inside torch, so
    # this is a tolerance check (1e-6 relative), not bit parity.
    b1, b2 = float(HP["beta1"]), float(HP["beta2"])
    for (t, g, mp_, vp_, po, mo, vo, tp, tm, tv) in _torch_reference(
            torch.optim.AdamW, 5, 4096, 0.1, seed=41):
        scale_p = np.abs(tp) + float(HP["lr"])
        assert np.max(np.abs(po - tp) / scale_p) <= 1e-6, t
        scale_m = b1 * np.abs(mp_) + (1 - b1) * np.abs(g)
        assert np.all(np.abs(mo - tm) <= 1e-6 * scale_m), t
        scale_v = b2 * np.abs(vp_) + (1 - b2) * g.astype(np.float64) ** 2
        assert np.all(np.abs(vo - tv) <= 1e-6 * scale_v), t


def test_adamw_decay_is_decoupled_not_l2():
    # torch.optim.Adam with weight_decay folds wd * p into the gradient
    # (coupled L2); the paper's optimizer reading is AdamW, and the two must
    # be far apart at these scales.
    worst = 0.0
    for (t, *_rest, po, mo, vo, tp, tm, tv) in _torch_reference(
            torch.optim.Adam, 3, 2048, 0.1, seed=42):
        worst = max(worst, float(np.max(np.abs(mo - tm))))
    assert worst > 1e-5


def test_adamw_grad_scale_is_applied_to_the_aggregate():
    n = 1000
    g = synth.host_grads(51, 0, 1, n, 1e-3)[0]
    p, m, v = synth.host_state(51, n, mv_sigma=1e-3)
    a = oracle.adamw(g, p, m, v, t=4, grad_scale=f32(1.0), **HP)
    b = oracle.adamw(g * f32(4.0), p, m, v, t=4, grad_scale=f32(0.25), **HP)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(bits(x), bits(y))


def test_adamw_eps_zero_with_zero_gradient_is_nan():
    z = np.zeros(3, np.float32)
    p = np.ones(3, np.float32)
    p1, m1, v1, _ = oracle.adamw(z, p, z, z, t=1, **dict(HP, eps=f32(0.0)))
    assert np.all(np.isnan(p1)) and not m1.any() and not v1.any()


# ----------------------------------------------------------------------------
# the composed path
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("W,gdtype,mode", [(4, "f32", oracle.AGG_FP32),
                                           (8, "f32", oracle.AGG_FIXED),
                                           (16, "bf16", oracle.AGG_FP32),
                                           (3, "bf16", oracle.AGG_FIXED)])
def test_fused_is_aggregate_then_adamw(W, gdtype, mode):
    n = 3001
    gs = synth.host_grads(61, 2, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                          outlier_scale=100.0)
    p, m, v = synth.host_state(61, n, mv_sigma=1e-4)
    out = oracle.fused(gs, p, m, v, mode=mode, frac_bits=24, t=2,
                       want_agg_f32=True, want_agg_i32=(mode == oracle.AGG_FIXED),
                       **HP)
    if mode == oracle.AGG_FIXED:
        ai, af = oracle.aggregate_fixed(gs, 24)
        assert np.array_equal(out["agg_i32"], ai)
    else:
        af = oracle.aggregate_f32(gs)
    assert np.array_equal(bits(out["agg_f32"]), bits(af))
    p1, m1, v1, p16 = oracle.adamw(af, p, m, v, t=2, **HP)
    for x, y in ((out["p"], p1), (out["m"], m1), (out["v"], v1)):
        assert np.array_equal(bits(x), bits(y))
    assert np.array_equal(out["p16"], p16)


def test_fused_is_independent_of_chunking():
    n, W = 5000, 5
    gs = synth.host_grads(62, 1, W, n, 1e-4)
    p, m, v = synth.host_state(62, n, mv_sigma=1e-4)
    whole = oracle.fused(gs, p, m, v, t=3, **HP)
    cut = 1777
    a = oracle.fused([g[:cut] for g in gs], p[:cut], m[:cut], v[:cut], t=3, **HP)
    b = oracle.fused([g[cut:] for g in gs], p[cut:], m[cut:], v[cut:], t=3, **HP)
    for key in ("p", "m", "v", "p16"):
        assert np.array_equal(whole[key], np.concatenate([a[key], b[key]]))


# ----------------------------------------------------------------------------
# Table III: per-element bytes and flops of the parameter server's step
# ----------------------------------------------------------------------------
def _read_table3():
    rows = []
    with open(os.path.join(HERE, "golden", "table3_requirements.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                gbps, stage, flops, mem, ssd = line.split()
                rows.append((int(gbps), stage, float(flops), float(mem), float(ssd)))
    return rows


def test_table3_byte_and_flop_accounting():
    from bench import ADAM_CORE_BYTES, ADAM_FLOPS_PER_ELEMENT
    # step 5 reads a 2-byte gradient and 12 bytes of state and writes 12
    # bytes of state and a 2-byte parameter copy
    core = sum(ADAM_CORE_BYTES.values())
    assert core == 28
    for gbps, stage, flops, mem, ssd in _read_table3():
        elems = gbps * 1e9 / 8 / 2            # 2-byte items per second
        gib = 2.0**30                         # the table's "GB" is 2^30 bytes
        fwd_mem = 2 + 2                       # steps 1 and 2
        fwd_ssd = 2
        if stage == "fwd":
            want = (0.0, fwd_mem, fwd_ssd)
        else:
            bwd_mem = fwd_mem + 2 + 12 + core + 14   # + steps 3, 4, 5, 6
            bwd_ssd = fwd_ssd + 12                   # reads: steps 1 and 4
            want = (ADAM_FLOPS_PER_ELEMENT, bwd_mem, bwd_ssd)
        got = (want[0] * elems / gib, want[1] * elems / gib, want[2] * elems / gib)
        for g_, p_ in zip(got, (flops, mem, ssd)):
            unit = 1.0 if p_ >= 100 else 0.1      # last printed digit
            assert abs(g_ - p_) <= unit, (gbps, stage, got)


# ----------------------------------------------------------------------------
# the format conversion as a producer, and int32 contributions
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("gdtype,k", [("f32", 24), ("f32", 0), ("bf16", 24), ("bf16", 30)])
def test_quantize_array_matches_exact_rational(gdtype, k):
    g = synth.host_grads(70, 0, 1, 4000, 1e-3, gdtype=gdtype, outlier_frac=0.02,
                         outlier_scale=1e6)[0]
    vals = oracle.bf16_to_f32(g) if gdtype == "bf16" else g
    want = np.array([exact_quantize(v, k) for v in vals], dtype=np.int64)
    assert np.array_equal(oracle.quantize_array(g, k).astype(np.int64), want)


def test_aggregate_fixed_of_int32_contributions_is_the_exact_sum():
    rng = np.random.default_rng(71)
    n, W = 3000, 7
    gs = [rng.integers(I32_MIN, I32_MAX, n, dtype=np.int64, endpoint=True).astype(np.int32)
          for _ in range(W)]
    gs[0][:5] = I32_MAX
    gs[1][:5] = I32_MAX                       # overflow: clamps to INT32_MAX
    gs[2][5:9] = I32_MIN
    gs[3][5:9] = I32_MIN
    small = [rng.integers(-1000, 1000, n).astype(np.int32) for _ in range(3)]
    for case in (gs, small):
        ai, af = oracle.aggregate_fixed(case, 24)
        s = [sum(int(c[i]) for c in case) for i in range(n)]
        want = np.array([max(I32_MIN, min(I32_MAX, x)) for x in s], dtype=np.int64)
        assert np.array_equal(ai.astype(np.int64), want)
        want_f = np.array([np.ldexp(np.float32(float(a)), -24) for a in want], np.float32)
        assert np.array_equal(bits(af), bits(want_f))


@pytest.mark.parametrize("gdtype", ["f32", "bf16"])
def test_quantise_then_aggregate_equals_aggregate_of_floats(gdtype):
    # the switch sums what the NICs produced: converting first and summing
    # int32 contributions gives the same bits as converting inside the sum
    n, W, k = 2500, 6, 24
    gs = synth.host_grads(72, 0, W, n, 1e-4, gdtype=gdtype, outlier_frac=0.01,
                          outlier_scale=1e5)
    qs = [oracle.quantize_array(g, k) for g in gs]
    a_i, a_f = oracle.aggregate_fixed(gs, k)
    b_i, b_f = oracle.aggregate_fixed(qs, k)
    assert np.array_equal(a_i, b_i) and np.array_equal(bits(a_f), bits(b_f))
    p, m, v = synth.host_state(72, n, mv_sigma=1e-4)
    x = oracle.fused(gs, p, m, v, mode=oracle.AGG_FIXED, frac_bits=k, t=2, **HP)
    y = oracle.fused(qs, p, m, v, mode=oracle.AGG_FIXED, frac_bits=k, t=2, **HP)
    for key in ("p", "m", "v", "p16"):
        assert np.array_equal(x[key], y[key])


def test_fused_inplace_equals_fused():
    """The in-place wrapper (used to time the oracle) runs the same C step."""
    gs = synth.host_grads(77, 2, 4, 5003, 1e-4, outlier_frac=0.01, outlier_scale=100.0)
    p, m, v = synth.host_state(77, 5003, mv_sigma=1e-4)
    hp = dict(lr=np.float32(1e-4), beta1=np.float32(0.9), beta2=np.float32(0.95),
              eps=np.float32(1e-8), wd=np.float32(0.1))
    for mode in (oracle.AGG_FP32, oracle.AGG_FIXED):
        want = oracle.fused(gs, p, m, v, mode=mode, frac_bits=24, t=2, **hp)
        q, mm, vv = p.copy(), m.copy(), v.copy()
        q16 = np.zeros(p.size, np.uint16)
        oracle.fused_inplace(gs, q, mm, vv, q16, mode=mode, frac_bits=24, t=2, **hp)
        for k, a in (("p", q), ("m", mm), ("v", vv), ("p16", q16)):
            assert np.array_equal(a.view(a.dtype), want[k]), k
