"""Pins of the CPU oracle against facts that do not come from the oracle.

Each ``pin_*`` function takes a loaded oracle library, runs it on small inputs
and raises AssertionError when the oracle disagrees with a closed form, an
invariant, a textbook special case or torch's independent implementation of
AdamW and gradient clipping.  ``tests/test_oracle_pins.py`` runs them on the
real oracle; ``tests/test_oracle_mutants.py`` runs them on copies with a
planted mistake and checks that some pin fails for every mistake.
"""
import numpy as np
import torch

import oracle
import synth

F32_ULP_RTOL = 2.0 ** -23


def bf16_bits(x):
    return synth.to_bf16_bits(np.asarray(x, dtype=np.float32))


def bf16_value(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def rand_grads(n, R, sigma=1e-3, seed=1, outlier_p=0.0):
    return [bf16_bits(synth.normal_f32(synth.seed(seed, 7, r), n, sigma,
                                       outlier_p=outlier_p, outlier_scale=100.0))
            for r in range(R)]


def rand_master(n, seed=1):
    return synth.normal_f32(synth.seed(seed, 9), n, 0.02)


def run(lib, masters, grads, hp, ms=None, vs=None):
    st = oracle.State(masters, ms, vs)
    rc, norm = oracle.step(st, grads, hp, lib=lib)
    return st, rc, norm


def ulps_apart(a, b):
    """Distance in FP32 ulps between two float32 arrays of finite values."""
    ia = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    ib = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7fffffff), ia)
    ib = np.where(ib < 0, -(ib & 0x7fffffff), ib)
    return np.abs(ia - ib)


# ---------------------------------------------------------------------------
# BF16 rounding (targeted; the exhaustive sweep is in test_oracle_bf16.py)

def pin_bf16_special_values(lib):
    cases = {
        0x00000000: 0x0000, 0x80000000: 0x8000,          # signed zeros
        0x3f800000: 0x3f80,                              # 1.0 exact
        0x3f808000: 0x3f80,                              # tie, even below
        0x3f818000: 0x3f82,                              # tie, odd below -> up
        0x3f808001: 0x3f81,                              # just above the tie
        0x3f807fff: 0x3f80,                              # just below the tie
        0x7f7fffff: 0x7f80,                              # max float -> inf
        0x7f7f7fff: 0x7f7f,                              # stays finite
        0x7f7f8000: 0x7f80,                              # tie at the top, odd -> inf
        0x7f800000: 0x7f80, 0xff800000: 0xff80,          # infinities
        0x00000001: 0x0000,                              # smallest subnormal
        0x00008000: 0x0000,                              # subnormal tie, even
        0x00018000: 0x0002,                              # subnormal tie, odd
        0x007fffff: 0x0080,                              # subnormal rounds to normal
    }
    u = np.array(list(cases.keys()), dtype=np.uint32)
    want = np.array(list(cases.values()), dtype=np.uint16)
    out = oracle.bf16(u.view(np.float32), lib=lib)
    assert np.array_equal(out, want), [(hex(a), hex(b), hex(c)) for a, b, c in zip(u, out, want) if b != c]
    # NaNs stay NaN, quiet, with sign kept
    nans = np.array([0x7f800001, 0x7fc00000, 0xffbfffff, 0x7f80ffff], dtype=np.uint32)
    o = oracle.bf16(nans.view(np.float32), lib=lib).astype(np.uint32)
    assert np.all((o & 0x7f80) == 0x7f80) and np.all(o & 0x0040)
    assert np.array_equal(o >> 15, nans >> 31)


def pin_bf16_random_vs_torch(lib):
    u = synth.raw_u32(synth.seed(3, 3), 0, 1 << 16)
    f = u.view(np.float32)
    keep = ~np.isnan(f)
    o = oracle.bf16(f, lib=lib)
    t = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(o[keep], t[keep])


# ---------------------------------------------------------------------------
# Step 1: aggregate

def pin_mean_closed_forms(lib):
    n = 300
    for R in (1, 2, 3, 4, 5, 8):
        gs = [bf16_bits(np.full(n, r + 1, np.float32)) for r in range(R)]
        got = oracle.mean_grads(gs, lib=lib)
        want = np.float32((R + 1) / 2.0)   # mean of 1..R
        assert np.all(got == want), (R, got[:3])
    x = rand_grads(1000, 1)[0]
    neg = x ^ np.uint16(0x8000)
    assert np.all(oracle.mean_grads([x, neg], lib=lib) == 0.0)
    # mean of the three values 1, 1, 2 is 4/3 rounded once to FP32
    gs = [bf16_bits(np.full(8, v, np.float32)) for v in (1.0, 1.0, 2.0)]
    assert np.all(oracle.mean_grads(gs, lib=lib) == np.float32(4.0 / 3.0))


def pin_mean_vs_fraction(lib):
    """Random BF16 gradients: the oracle's mean is the exact rational mean
    rounded once to FP32 (fractions.Fraction)."""
    import mean_cases
    n = 1500
    for R in (1, 2, 3, 4, 7, 8):
        gs = rand_grads(n, R, seed=R, outlier_p=0.01)
        want = mean_cases.exact_means(np.stack(gs))
        got = oracle.mean_grads(gs, lib=lib)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), R


def pin_mean_exact_quotient(lib):
    """Rank sets built to make the single rounding of S / R hard -- quotients
    on, or a tiny value away from, FP32 midpoints, sums whose FP64 evaluation
    in rank order is inexact (magnitudes spanning far more than 2^45),
    every exponent, and subnormal quotients whose rounding only the division's
    remainder decides -- against fractions.Fraction, bit for bit.  The same
    sets must also show that an FP64 sum divided in FP64 and rounded again
    is not the same thing (else they would not test the rounding)."""
    import mean_cases
    double_rounding_misses = 0
    remainder_decides = 0
    for R in (1, 2, 3, 4, 5, 7, 8, 11, 13, 15, 16):
        sets = [mean_cases.wide_span(R, 100, seed=R)]
        if R >= 3:
            sets.append(mean_cases.near_midpoint(R, 200, seed=100 + R))
        sub = mean_cases.subnormal_remainder(R)
        if R in (11, 13, 15):
            assert sub.shape[1] > 0
        remainder_decides += mean_cases.remainder_decides(sub)
        sets.append(sub)
        ranks = np.concatenate(sets, axis=1)
        want = mean_cases.exact_means(ranks)
        got = oracle.mean_grads([ranks[r].copy() for r in range(R)], lib=lib)
        bad = np.flatnonzero(got.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, (R, [(ranks[:, i].tolist(), float(got[i]), float(want[i])) for i in bad[:3]])
        if R in (3, 5, 7, 13):
            naive = mean_cases.rank_order_f64_mean(ranks)
            double_rounding_misses += int(np.count_nonzero(naive.view(np.uint32) != want.view(np.uint32)))
    assert double_rounding_misses > 0
    assert remainder_decides > 0


# ---------------------------------------------------------------------------
# Steps 2-3: norm and clip

def pin_norm_constant(lib):
    g0 = np.float32(bf16_value(bf16_bits([3.0e-3]))[0])
    n = 1024 * 1024
    gs = [bf16_bits(np.full(n, g0, np.float32))] * 2
    norm = oracle.grad_norm([gs], lib=lib)
    assert norm == 1024.0 * abs(float(g0)), (norm, 1024.0 * abs(float(g0)))
    # two segments: norms combine as sqrt(a^2 + b^2), here 3-4-5
    a = [bf16_bits(np.full(4096, 3.0 / 64, np.float32))]
    b = [bf16_bits(np.full(4096, 4.0 / 64, np.float32))]
    assert oracle.grad_norm([a, b], lib=lib) == 5.0


def pin_exact_sum_vs_fsum(lib):
    """The norm's sum is the exactly rounded sum: compare with math.fsum
    (a correctly rounded library summation) on values of widely spread
    magnitude, where any rounding inside the sum would show."""
    import math
    rng = np.random.default_rng(8)
    for trial in range(6):
        n = int(rng.integers(1, 20000))
        x = (rng.normal(0, 1, n) * np.exp2(rng.integers(-140, 126, n).astype(np.float64))).astype(np.float32)
        x = x[np.isfinite(x)]
        want = math.fsum(float(v) * float(v) for v in x)
        assert oracle.sum_squares(x, lib=lib) == want, trial


def pin_exact_sum_ties_and_carries(lib):
    import math
    cases = [
        [1.0, 2.0 ** -27, 2.0 ** -27],                 # 1 + 2^-53: a tie, stays 1
        [1.0, 2.0 ** -27, 2.0 ** -27, 2.0 ** -100],    # just above the tie: rounds up
        [1.0 + 2.0 ** -23, 2.0 ** -27, 2.0 ** -27],    # tie next to an odd significand
        [2.0 ** 63] * 4096 + [2.0 ** -60] * 3,         # long carry chains, tiny tail
        [2.0 ** -149] * 1000 + [3.0],                  # subnormal squares
        [1e-20, 1e20, -1e20, 3e-15],
    ]
    for k, c in enumerate(cases):
        x = np.array(c, np.float32)
        want = math.fsum(float(v) * float(v) for v in x)
        assert oracle.sum_squares(x, lib=lib) == want, (k, oracle.sum_squares(x, lib=lib), want)
    # the norm itself: sqrt of that exact sum, over two segments and ranks
    gs = [rand_grads(3000, 3, seed=31, outlier_p=0.05), rand_grads(77, 3, seed=32)]
    means = np.concatenate([oracle.mean_grads(g, lib=lib) for g in gs])
    want = math.sqrt(math.fsum(float(v) * float(v) for v in means))
    assert oracle.grad_norm(gs, lib=lib) == want


def pin_norm_vs_torch(lib):
    segs = [rand_grads(n, 3, seed=n, outlier_p=0.01) for n in (1, 1000, 4097, 70000)]
    got = oracle.grad_norm(segs, lib=lib)
    means = [torch.from_numpy(oracle.mean_grads(g, lib=lib).astype(np.float64)) for g in segs]
    ps = [torch.zeros(m.numel(), dtype=torch.float64, requires_grad=True) for m in means]
    for p, m in zip(ps, means):
        p.grad = m.clone()
    want = float(torch.nn.utils.clip_grad_norm_(ps, max_norm=1e30, foreach=False))
    assert abs(got - want) <= 1e-13 * want, (got, want)


def pin_clip_coef(lib):
    for norm, mx in ((0.5, 1.0), (2.0, 1.0), (70.0, 1.0), (1e-9, 1e-3), (3.0, 0.0), (3.0, -1.0)):
        ps = [torch.zeros(1, dtype=torch.float64, requires_grad=True)]
        ps[0].grad = torch.tensor([norm], dtype=torch.float64)
        got = oracle.clip_coef(norm, mx, lib=lib)
        if mx > 0:
            torch.nn.utils.clip_grad_norm_(ps, max_norm=mx, foreach=False)
            want = float(ps[0].grad[0]) / norm
            assert abs(got - want) <= 1e-15 * want, (norm, mx, got, want)
        else:
            assert got == 1.0


# ---------------------------------------------------------------------------
# Step 4: AdamW

def _torch_adamw_one(p, m, v, g, hp):
    """One torch.optim.AdamW step on float64 tensors starting from (m, v) at t-1."""
    pt = torch.tensor(p, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([pt], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False, fused=False)
    pt.grad = torch.tensor(g, dtype=torch.float64)
    if hp.step > 1:
        opt.state[pt] = {"step": torch.tensor(float(hp.step - 1)),
                         "exp_avg": torch.tensor(m, dtype=torch.float64),
                         "exp_avg_sq": torch.tensor(v, dtype=torch.float64)}
    else:
        assert np.all(m == 0) and np.all(v == 0)
    opt.step()
    st = opt.state[pt]
    return pt.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def pin_adamw_f64_vs_torch(lib):
    rng = np.random.default_rng(5)
    n = 2048
    settings = [
        dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01),
        dict(lr=3e-2, beta1=0.8, beta2=0.95, eps=1e-3, weight_decay=0.2),
        dict(lr=1e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1),
        dict(lr=5e-2, beta1=0.0, beta2=0.5, eps=1e-6, weight_decay=0.0),
    ]
    for s in settings:
        p = rng.normal(0, 0.02, n)
        m = np.zeros(n)
        v = np.zeros(n)
        for t in (1, 2, 3, 7, 1000):
            g = rng.normal(0, 1e-3, n) * np.where(rng.random(n) < 0.05, 100.0, 1.0)
            hp = oracle.hparams(step=t, max_grad_norm=0.0, **s)
            po, mo, vo = oracle.adamw_f64(p, m, v, g, hp, lib=lib)
            tp, tm, tv = _torch_adamw_one(p, m, v, g, hp)
            scale_m = np.abs(s["beta1"] * m) + np.abs((1 - s["beta1"]) * g)
            scale_v = s["beta2"] * v + (1 - s["beta2"]) * g * g
            step_mag = np.abs(tp - p * (1 - s["lr"] * s["weight_decay"]))
            scale_p = np.abs(p) + step_mag
            assert np.all(np.abs(mo - tm) <= 1e-12 * scale_m + 1e-300), (s, t)
            assert np.all(np.abs(vo - tv) <= 1e-12 * scale_v + 1e-300), (s, t)
            assert np.all(np.abs(po - tp) <= 1e-12 * scale_p), (s, t, np.max(np.abs(po - tp) / scale_p))
            p, m, v = po, mo, vo


def pin_first_step_sign(lib):
    """t = 1, m = v = 0, eps = 0, no clip: p' = p (1 - lr wd) - lr sign(g)."""
    n = 4096
    R = 2
    gs = rand_grads(n, R, seed=11)
    master = rand_master(n, seed=11)
    hp = oracle.hparams(lr=1e-3, eps=0.0, weight_decay=0.05, max_grad_norm=0.0, step=1)
    st, rc, _ = run(lib, [master], [gs], hp)
    assert rc == oracle.ORC_OK
    g = oracle.mean_grads(gs, lib=lib).astype(np.float64)
    nz = g != 0
    want = (master.astype(np.float64) * (1 - 1e-3 * 0.05) - 1e-3 * np.sign(g)).astype(np.float32)
    assert ulps_apart(st.master[0][nz], want[nz]).max() <= 1
    # the moments are the scaled gradient and scaled squared gradient
    assert ulps_apart(st.exp_avg[0], (0.1 * g).astype(np.float32)).max() <= 1
    assert ulps_apart(st.exp_avg_sq[0], (0.001 * g * g).astype(np.float32)).max() <= 1


def pin_zero_gradient(lib):
    """A zero mean gradient leaves only the decoupled decay."""
    n = 3000
    x = rand_grads(n, 1, seed=12)[0]
    gs = [x, x ^ np.uint16(0x8000)]
    master = rand_master(n, seed=12)
    hp = oracle.hparams(lr=1e-2, eps=1e-8, weight_decay=0.1, step=1)
    st, rc, norm = run(lib, [master], [gs], hp)
    assert rc == oracle.ORC_OK and norm == 0.0
    want = (master.astype(np.float64) * (1 - 1e-2 * 0.1)).astype(np.float32)
    assert ulps_apart(st.master[0], want).max() <= 1
    assert np.all(st.exp_avg[0] == 0) and np.all(st.exp_avg_sq[0] == 0)


def pin_sign_descent(lib):
    """beta1 = beta2 = 0: every step is p(1 - lr wd) - lr g / (|g| + eps)."""
    n = 2048
    R = 3
    master = rand_master(n, seed=13)
    st = oracle.State([master])
    lr, wd, eps = 2e-3, 0.03, 1e-4
    for t in (1, 2, 3, 4):
        gs = rand_grads(n, R, seed=100 + t)
        hp = oracle.hparams(lr=lr, beta1=0.0, beta2=0.0, eps=eps, weight_decay=wd,
                            max_grad_norm=0.0, step=t)
        p0 = st.master[0].astype(np.float64)
        rc, _ = oracle.step(st, [gs], hp, lib=lib)
        assert rc == oracle.ORC_OK
        g = oracle.mean_grads(gs, lib=lib).astype(np.float64)
        want = (p0 * (1 - lr * wd) - lr * g / (np.abs(g) + eps)).astype(np.float32)
        assert ulps_apart(st.master[0], want).max() <= 1, t


def pin_lr_zero(lib):
    n = 1000
    master = rand_master(n, seed=14)
    gs = rand_grads(n, 2, seed=14)
    hp = oracle.hparams(lr=0.0, step=1)
    st, rc, _ = run(lib, [master], [gs], hp)
    assert rc == oracle.ORC_OK
    assert np.array_equal(st.master[0], master)
    assert np.array_equal(st.param_bf16[0], bf16_bits(master))
    assert np.any(st.exp_avg[0] != 0) and np.any(st.exp_avg_sq[0] != 0)


# ---------------------------------------------------------------------------
# Invariants (bit-exact)

def pin_identical_ranks(lib):
    n = 5000
    master = rand_master(n, seed=15)
    g = rand_grads(n, 1, seed=15, outlier_p=0.01)[0]
    hp = oracle.hparams(step=1, max_grad_norm=0.05)
    ref, _, nref = run(lib, [master], [[g]], hp)
    for R in (2, 4, 8):
        st, _, nr = run(lib, [master], [[g] * R], hp)
        assert nr == nref
        for a, b in ((st.master, ref.master), (st.exp_avg, ref.exp_avg),
                     (st.exp_avg_sq, ref.exp_avg_sq), (st.param_bf16, ref.param_bf16)):
            assert np.array_equal(a[0], b[0]), R


def pin_clip_noop(lib):
    n = 5000
    master = rand_master(n, seed=16)
    gs = rand_grads(n, 2, seed=16)
    norm = oracle.grad_norm([gs], lib=lib)
    assert 0 < norm < 1.0
    a, _, _ = run(lib, [master], [gs], oracle.hparams(step=1, max_grad_norm=1.0))
    b, _, _ = run(lib, [master], [gs], oracle.hparams(step=1, max_grad_norm=0.0))
    for x, y in ((a.master, b.master), (a.exp_avg, b.exp_avg), (a.exp_avg_sq, b.exp_avg_sq)):
        assert np.array_equal(x[0], y[0])


def pin_nonfinite(lib):
    n = 100
    master = rand_master(n, seed=17)
    for bad in (np.inf, -np.inf, np.nan):
        gs = rand_grads(n, 2, seed=17)
        gs[1] = gs[1].copy()
        gs[1][37] = bf16_bits([bad])[0]
        st, rc, norm = run(lib, [master], [gs], oracle.hparams(step=1))
        assert rc == oracle.ORC_NONFINITE and not np.isfinite(norm)
        assert np.array_equal(st.master[0], master)
        assert np.all(st.exp_avg[0] == 0) and np.all(st.exp_avg_sq[0] == 0)


def pin_param_is_bf16_of_master(lib):
    n = 4097
    st, _, _ = run(lib, [rand_master(n, 18)], [rand_grads(n, 2, 18)], oracle.hparams(step=1))
    assert np.array_equal(st.param_bf16[0], bf16_bits(st.master[0]))


# ---------------------------------------------------------------------------
# Variant: the update fed the mean gradient rounded to BF16

def _bf16_route_case(n, seed):
    """Rank gradients whose FP32 mean lies exactly on, below or above a BF16
    midpoint, and the BF16 value that round-to-nearest-even must give.  A is a
    random finite BF16 value away from its binade's top, so A+1 and A+2 (the
    next BF16 values away from zero) share its exponent."""
    rng = np.random.default_rng(seed)
    sign = rng.integers(0, 2, n).astype(np.uint16) << 15
    expo = rng.integers(0x70, 0x7c, n).astype(np.uint16) << 7   # |a| in [2^-15, 2^-3)
    mant = rng.integers(0, 0x7d, n).astype(np.uint16)
    A = sign | expo | mant
    kind = np.arange(n) % 3
    g = [A.copy(), A.copy(), A.copy(), A.copy()]
    # kind 0: mean a + u/2 (two ranks at A, two at A+1): tie, even bits win
    # kind 1: mean a + u/4 (one rank at A+1): rounds down to A
    # kind 2: mean a + 3u/4 (three ranks at A+1): rounds up to A+1
    for r in range(4):
        up = (kind == 0) & (r >= 2) | (kind == 1) & (r == 3) | (kind == 2) & (r >= 1)
        g[r][up] += 1
    want = np.where(kind == 0, np.where(A % 2 == 0, A, A + 1),
                    np.where(kind == 1, A, A + 1)).astype(np.uint16)
    return g, want


def pin_bf16_gradient_route(lib):
    # R = 1: the mean is a BF16 value already, so rounding it changes nothing
    n = 3000
    master = rand_master(n, seed=31)
    g1 = rand_grads(n, 1, seed=31, outlier_p=0.01)
    hp = oracle.hparams(step=2, max_grad_norm=0.05)
    a = oracle.State([master])
    b = oracle.State([master])
    ra, na = oracle.step(a, [g1], hp, lib=lib)
    rb, nb = oracle.step(b, [g1], hp, lib=lib, gbar_bf16=True)
    assert ra == rb == 0 and na == nb
    for x, y in ((a.master, b.master), (a.exp_avg, b.exp_avg), (a.exp_avg_sq, b.exp_avg_sq),
                 (a.param_bf16, b.param_bf16)):
        assert np.array_equal(x[0], y[0])
    # R = 4 with the mean on, below and above BF16 midpoints: without
    # clipping the step equals the step on the single rounded gradient
    g4, want = _bf16_route_case(n, seed=32)
    hp0 = oracle.hparams(step=1, max_grad_norm=0.0)
    c = oracle.State([master])
    d = oracle.State([master])
    _, nc = oracle.step(c, [g4], hp0, lib=lib, gbar_bf16=True)
    _, nd = oracle.step(d, [[want]], hp0, lib=lib)
    for x, y in ((c.master, d.master), (c.exp_avg, d.exp_avg), (c.exp_avg_sq, d.exp_avg_sq),
                 (c.param_bf16, d.param_bf16)):
        assert np.array_equal(x[0], y[0])
    # the norm (and so the clip decision) comes from the unrounded FP32 mean
    exact = np.float64(np.sum(np.square(oracle.mean_grads(g4, lib=lib).astype(np.float64))))
    assert abs(nc - np.sqrt(exact)) <= 1e-12 * nc and nc != nd
    # the sampled-point entry takes the same rounding
    po, mo, vo, pb = oracle.update_points(master, np.zeros(n, np.float32), np.zeros(n, np.float32),
                                          np.stack(g4, axis=1), 1.0, hp0, lib=lib, gbar_bf16=True)
    assert np.array_equal(po, d.master[0]) and np.array_equal(vo, d.exp_avg_sq[0])
    assert np.array_equal(pb, d.param_bf16[0])


def pin_update_given_clip_equals_step(lib):
    """The array update with a known clip coefficient (used to check states
    too large for one oracle call) is the step with that coefficient."""
    n, R = 70001, 3
    grads = [rand_grads(n, R, seed=31, outlier_p=0.01)]
    master = rand_master(n, seed=31)
    for t, mgn in ((1, 0.05), (2, 0.0)):
        hp = oracle.hparams(lr=1e-3, weight_decay=0.02, max_grad_norm=mgn, step=t)
        st = oracle.State([master])
        _, norm = oracle.step(st, grads, hp, lib=lib)
        c = oracle.clip_coef(norm, mgn, lib=lib)
        p, m, v, pb = master.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32), np.zeros(n, np.uint16)
        oracle.update_given_clip(p, m, v, pb, grads[0], c, hp, lib=lib)
        for x, y in ((p, st.master[0]), (m, st.exp_avg[0]), (v, st.exp_avg_sq[0]), (pb, st.param_bf16[0])):
            assert np.array_equal(x, y), t


# ---------------------------------------------------------------------------
# The whole step against torch (library special case, brute force sizes)

def torch_step(masters, ms, vs, grads, hp):
    """Reference of one step built from torch library calls in float64."""
    means = []
    for gs in grads:
        vals = torch.stack([torch.from_numpy(bf16_value(g).astype(np.float64)) for g in gs])
        means.append((vals.sum(0) / len(gs)).to(torch.float32).to(torch.float64))
    ps = [torch.tensor(m.astype(np.float64), requires_grad=True) for m in masters]
    for p, g in zip(ps, means):
        p.grad = g.clone()
    if hp.max_grad_norm > 0:
        norm = float(torch.nn.utils.clip_grad_norm_(ps, hp.max_grad_norm, foreach=False))
    else:
        norm = float(torch.linalg.vector_norm(torch.cat(means)))
    opt = torch.optim.AdamW(ps, lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False, fused=False)
    if hp.step > 1:
        for p, m, v in zip(ps, ms, vs):
            opt.state[p] = {"step": torch.tensor(float(hp.step - 1)),
                            "exp_avg": torch.from_numpy(m.astype(np.float64)),
                            "exp_avg_sq": torch.from_numpy(v.astype(np.float64))}
    opt.step()
    out = []
    for p in ps:
        st = opt.state[p]
        out.append((p.detach().numpy().astype(np.float32),
                    st["exp_avg"].numpy().astype(np.float32),
                    st["exp_avg_sq"].numpy().astype(np.float32)))
    return out, norm


def check_against_torch(lib, sizes, R, steps, seed, hp_kw, max_ulps=1):
    masters = [rand_master(n, seed + k) for k, n in enumerate(sizes)]
    st = oracle.State(masters)
    for t in range(1, steps + 1):
        grads = [rand_grads(n, R, seed=1000 * seed + 10 * t + k, outlier_p=0.01)
                 for k, n in enumerate(sizes)]
        hp = oracle.hparams(step=t, **hp_kw)
        ref, tnorm = torch_step(st.master, st.exp_avg, st.exp_avg_sq, grads, hp)
        rc, norm = oracle.step(st, grads, hp, lib=lib)
        assert rc == oracle.ORC_OK
        assert abs(norm - tnorm) <= 1e-12 * tnorm, (norm, tnorm)
        for s in range(len(sizes)):
            for got, want in zip((st.master[s], st.exp_avg[s], st.exp_avg_sq[s]), ref[s]):
                d = ulps_apart(got, want)
                assert d.max() <= max_ulps, (sizes, R, t, s, int(d.max()))
            assert np.array_equal(st.param_bf16[s], bf16_bits(st.master[s]))


def pin_step_vs_torch(lib):
    check_against_torch(lib, [1000, 4097, 1], R=4, steps=3, seed=21,
                        hp_kw=dict(lr=1e-3, weight_decay=0.01, max_grad_norm=0.5))
    check_against_torch(lib, [70000], R=3, steps=2, seed=22,
                        hp_kw=dict(lr=1e-2, beta1=0.85, beta2=0.99, eps=1e-6,
                                   weight_decay=0.1, max_grad_norm=0.0))


def pin_brute_force(lib):
    for n in (1, 7, 8, 9, 63, 64, 65, 4095, 4097, 65537):
        for R in (1, 2, 3, 4, 8):
            if n == 65537 and R not in (1, 8):
                continue
            check_against_torch(lib, [n], R=R, steps=2, seed=n * 10 + R,
                                hp_kw=dict(lr=1e-3, weight_decay=0.01, max_grad_norm=0.05))


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
