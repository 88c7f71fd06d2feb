"""Property tests of the CPU oracle (no GPU), drawn with hypothesis.

Each property holds for every configuration and follows from the update and
averaging equations (Algorithms 1-3) together with IEEE arithmetic, not from
another implementation of them:

- with eps = 0, Adam and ADOPT are invariant to a power-of-two scale of the
  gradients: v scales by 4^k, Adam's u by 2^k (ADOPT's u averages the
  normalised gradient, so it does not move), the update direction is
  unchanged and x follows the same trajectory bit for bit (scaling by a
  power of two commutes with every rounding, and sqrt(4^k y) = 2^k sqrt(y)
  exactly); SGDM's momenta scale by 2^k exactly;
- the workers are interchangeable: permuting their gradients permutes every
  state, bit for bit;
- identical gradients keep every worker identical, and every sync is then
  an exact no-op;
- the replica mean of rows whose fp64 sum is exact is the exact mean,
  rounded once, written to every row (checked against exact rational
  arithmetic).
"""

from fractions import Fraction

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as hst

import oracle

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@hst.composite
def configs(draw, forms=("adam", "adopt", "sgdm"), eps=None):
    form = draw(hst.sampled_from(forms))
    n = draw(hst.integers(1, 4))
    betas = tuple(float(np.float32(b)) for b in
                  draw(hst.lists(hst.sampled_from([0.0, 0.5, 0.9, 0.99, 0.999]), min_size=n, max_size=n)))
    raw = draw(hst.lists(hst.floats(0.05, 1.0), min_size=n, max_size=n))
    total = draw(hst.sampled_from([1.0, 0.9, 0.6]))
    omega = tuple(float(np.float32(total * r / sum(raw))) for r in raw)
    periods = hst.sampled_from([0, 1, 2, 3])
    return oracle.OracleConfig(
        form=form, beta1=betas, omega=omega, beta2=float(np.float32(draw(hst.sampled_from([0.99, 0.999])))),
        eps=float(np.float32(1e-8)) if eps is None else eps, clip_rho=0.0,
        bias_correction=draw(hst.booleans()), adopt_order=draw(hst.sampled_from(["prev", "cur"])),
        period_x=draw(periods), period_u=tuple(draw(periods) for _ in range(n)), period_v=draw(periods))


def _grads(seed, steps, K, P):
    rng = np.random.Generator(np.random.PCG64(seed))
    return [(1e-2 * rng.standard_normal((K, P))).astype(np.float32) for _ in range(steps)]


def _x0(seed, P):
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    return (0.02 * rng.standard_normal(P)).astype(np.float32)


def _run(cfg, x0, gs, K, lr=1e-3):
    st = oracle.new_state(cfg, x0, K)
    oracle.run(cfg, st, lambda s: gs[s - 1], list(range(1, len(gs) + 1)), lambda s: lr)
    return st


@SETTINGS
@given(cfg=configs(forms=("adam", "adopt"), eps=0.0), k=hst.integers(-8, 8), K=hst.integers(1, 4),
       P=hst.integers(1, 48), steps=hst.integers(1, 6), seed=hst.integers(0, 2**31))
def test_adaptive_forms_are_invariant_to_a_power_of_two_gradient_scale(cfg, k, K, P, steps, seed):
    gs = _grads(seed, steps, K, P)
    x0 = _x0(seed, P)
    a = _run(cfg, x0, gs, K)
    b = _run(cfg, x0, [g * np.float32(2.0 ** k) for g in gs], K)
    assert np.array_equal(a.x, b.x)
    u_scale = np.float32(2.0 ** k) if cfg.form == "adam" else np.float32(1.0)
    for ua, ub in zip(a.u, b.u):
        assert np.array_equal(ua * u_scale, ub)
    assert np.array_equal(a.v * np.float32(4.0 ** k), b.v)


@SETTINGS
@given(cfg=configs(forms=("sgdm",)), k=hst.integers(-8, 8), K=hst.integers(1, 4), P=hst.integers(1, 48),
       steps=hst.integers(1, 6), seed=hst.integers(0, 2**31))
def test_sgdm_momenta_scale_with_a_power_of_two_gradient_scale(cfg, k, K, P, steps, seed):
    gs = _grads(seed, steps, K, P)
    x0 = _x0(seed, P)
    a = _run(cfg, x0, gs, K)
    b = _run(cfg, x0, [g * np.float32(2.0 ** k) for g in gs], K)
    for ua, ub in zip(a.u, b.u):
        assert np.array_equal(ua * np.float32(2.0 ** k), ub)


@SETTINGS
@given(cfg=configs(), K=hst.integers(2, 5), P=hst.integers(1, 48), steps=hst.integers(1, 6),
       seed=hst.integers(0, 2**31), perm_seed=hst.integers(0, 2**31))
def test_workers_are_interchangeable(cfg, K, P, steps, seed, perm_seed):
    # local steps only, so no sum over workers enters and the property is exact
    cfg = oracle.OracleConfig(**{**cfg.__dict__, "period_x": 0, "period_u": (0,) * cfg.n, "period_v": 0})
    perm = np.random.Generator(np.random.PCG64(perm_seed)).permutation(K)
    gs = _grads(seed, steps, K, P)
    x0 = _x0(seed, P)
    a = _run(cfg, x0, gs, K)
    b = _run(cfg, x0, [np.ascontiguousarray(g[perm]) for g in gs], K)
    for sa, sb in zip(a.arrays(), b.arrays()):
        assert np.array_equal(sa[perm], sb)


@SETTINGS
@given(cfg=configs(), K=hst.integers(1, 5), P=hst.integers(1, 48), steps=hst.integers(1, 6),
       seed=hst.integers(0, 2**31))
def test_identical_gradients_keep_workers_identical_and_syncs_exact(cfg, K, P, steps, seed):
    g1 = _grads(seed, steps, 1, P)
    gs = [np.repeat(g, K, axis=0) for g in g1]
    st = oracle.new_state(cfg, _x0(seed, P), K)
    for s in range(1, steps + 1):
        oracle.local_step(cfg, st, gs[s - 1], s, 1e-3, 0.0, oracle.clip_scales(cfg, gs[s - 1]))
        before = [a.copy() for a in st.arrays()]
        oracle.sync(cfg, st, (1 << (1 + cfg.n + (1 if cfg.has_v else 0))) - 1)
        for b, a in zip(before, st.arrays()):
            assert np.array_equal(a, b)
            assert np.array_equal(a, np.repeat(a[:1], K, axis=0))


@SETTINGS
@given(K=hst.integers(1, 8), P=hst.integers(1, 32), seed=hst.integers(0, 2**31))
def test_replica_mean_is_the_exact_mean_rounded_once(K, P, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    a = (1e-2 * (1.0 + rng.random((K, P)))).astype(np.float32)  # one binade: the fp64 sum is exact
    src = a.copy()
    oracle.replica_mean(a, "f32")
    for i in range(P):
        exact = sum(Fraction(float(src[m, i])) for m in range(K)) / K
        lo = np.float32(float(exact))  # the float32 value nearest the double nearest the exact mean
        cands = [np.nextafter(lo, np.float32(-1)), lo, np.nextafter(lo, np.float32(1))]
        want = min(cands, key=lambda c: (abs(Fraction(float(c)) - exact), int(np.float32(c).view(np.uint32)) & 1))
        assert np.all(a[:, i] == want), (i, a[:, i], want)
