"""Pins of the CPU oracle: checks against what the paper and the
mathematics fix, independent of the oracle's own code.

Each ``pin_*`` function raises AssertionError when the oracle disagrees.  The
functions are collected by ``test_oracle_pins.py`` and re-run against
deliberately broken builds of the oracle by ``test_oracle_mutants.py``
(every planted mistake must fail at least one pin).

Textbook and library anchors:
  * torch.optim.Adam / torch.optim.SGD (fp64, CPU) -- library routines;
  * ADOPT as published (Taniguchi et al., 2024, Algorithm 1) and QHM /
    QHAdam (Ma & Yarats, 2019), written from those papers;
  * closed forms from Section 2.1 (unrolled EMA, local-momentum variance,
    half-life, 0.9^32 ~ 0.03) and Section 2.3 (communication reduction);
  * the virtual-average identity of the convergence analysis (Appendix,
    auxiliary notation: the worker mean of u^j is the EMA of the mean
    gradient);
  * hand-worked 3-element examples (tests/golden/hand_worked_examples.json).
"""

from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def f32(a: float) -> float:
    """The fp32 value the oracle receives for a hyper-parameter."""
    return float(np.float32(a))


def _cfg(form, beta1, omega, **kw):
    kw.setdefault("x_dtype", "f64")
    kw.setdefault("g_dtype", "f64")
    kw.setdefault("m_dtype", "f64")
    return oracle.OracleConfig(form=form, beta1=tuple(beta1), omega=tuple(omega), **kw)


def _close(a, b, rtol, atol=0.0, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    err = np.abs(a - b)
    lim = atol + rtol * np.abs(b)
    if not np.all(err <= lim):
        i = int(np.argmax(err - lim))
        raise AssertionError(f"{what}: max violation at {i}: got {a.flat[i]!r} want {b.flat[i]!r}")


# ----------------------------------------------------------------- P1, P2


def pin_adam_reduces_to_torch_adam():
    """N=1, omega=1, no clip: Algorithm 1 with Kingma-Ba bias correction is
    textbook Adam; compared with torch.optim.Adam in fp64."""
    rng = np.random.default_rng(11)
    P, T = 64, 25
    b1, b2, eps, lr = f32(0.9), f32(0.995), f32(1e-6), f32(3e-3)
    cfg = _cfg("adam", (b1,), (1.0,), beta2=b2, eps=eps, period_x=0, period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    p = torch.tensor(x0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps)
    for s in range(1, T + 1):
        g = rng.normal(0, 0.1, P) * (1 + s % 3)
        oracle.local_step(cfg, st, g[None, :], s, lr)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    state = opt.state[p]
    _close(st.x[0], p.detach().numpy(), 1e-12, 1e-15, "x")
    _close(st.u[0][0], state["exp_avg"].numpy(), 1e-12, 1e-18, "u")
    _close(st.v[0], state["exp_avg_sq"].numpy(), 1e-12, 1e-20, "v")


def pin_adam_weight_selects_one_moment():
    """N=2 with omega=(0,1): only the second EMA drives x, so x follows
    textbook Adam with that EMA's beta while u^1 keeps its own beta."""
    rng = np.random.default_rng(12)
    P, T = 32, 12
    b1a, b1b, b2, eps, lr = f32(0.5), f32(0.97), f32(0.99), f32(1e-8), f32(1e-2)
    cfg = _cfg("adam", (b1a, b1b), (0.0, 1.0), beta2=b2, eps=eps, period_x=0, period_u=(0, 0),
               period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    p = torch.tensor(x0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=lr, betas=(b1b, b2), eps=eps)
    ua = np.zeros(P)
    for s in range(1, T + 1):
        g = rng.normal(0, 1, P)
        oracle.local_step(cfg, st, g[None, :], s, lr)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        ua = b1a * ua + (1 - b1a) * g
    _close(st.x[0], p.detach().numpy(), 1e-12, 1e-15, "x")
    _close(st.u[0][0], ua, 1e-12, 1e-18, "u1")


def pin_sgdm_reduces_to_torch_sgd():
    """SGDM N=1, omega=1: the dampened EMA momentum from a zero buffer,
    i.e. torch.optim.SGD(momentum=beta, dampening=beta) whose buffer starts
    at zero (torch's own first step would copy g instead)."""
    rng = np.random.default_rng(13)
    P, T = 48, 20
    b, lr = f32(0.95), f32(0.05)
    cfg = _cfg("sgdm", (b,), (1.0,), period_x=0, period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    p = torch.tensor(x0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=lr, momentum=b, dampening=b)
    opt.state[p]["momentum_buffer"] = torch.zeros(P, dtype=torch.float64)
    for s in range(1, T + 1):
        g = rng.normal(0, 1, P)
        oracle.local_step(cfg, st, g[None, :], s, lr)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    _close(st.x[0], p.detach().numpy(), 1e-12, 1e-15, "x")
    _close(st.u[0][0], opt.state[p]["momentum_buffer"].numpy(), 1e-12, 1e-18, "u")


def pin_adopt_reduces_to_published_adopt():
    """N=1, omega=1, previous-v order: ADOPT as published (v_0 = g_0^2;
    m_t = b1 m + (1-b1) clip(g_t / max(sqrt(v_{t-1}), eps), c_t);
    x_t = x_{t-1} - lr m_t; v_t = b2 v + (1-b2) g_t^2; c_t = t^(1/4)).
    With eps far below sqrt(v) the paper's sqrt(v)+eps equals max(sqrt(v), eps)."""
    rng = np.random.default_rng(14)
    P, T = 40, 16
    b1, b2, lr, eps = f32(0.9), f32(0.999), f32(1e-2), f32(1e-30)
    cfg = _cfg("adopt", (b1,), (1.0,), beta2=b2, eps=eps, adopt_order="prev", period_x=0,
               period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    x, m, v = x0.copy(), np.zeros(P), None
    for s in range(1, T + 1):
        g = rng.standard_t(2.5, P)
        t = s - 1
        c = f32(t ** 0.25) if t > 0 else 0.0
        oracle.local_step(cfg, st, g[None, :], s, lr, c)
        if v is None:
            v = g * g
            continue
        n = np.clip(g / np.maximum(np.sqrt(v), eps), -c, c)
        m = b1 * m + (1 - b1) * n
        x = x - lr * m
        v = b2 * v + (1 - b2) * g * g
    _close(st.x[0], x, 1e-12, 1e-15, "x")
    _close(st.u[0][0], m, 1e-12, 1e-18, "u")
    _close(st.v[0], v, 1e-12, 1e-20, "v")


def pin_adopt_current_order_is_algorithm_as_printed():
    """The literal order of Algorithm 2 (v updated first, then used to
    normalise the same gradient), N=1, omega=nu: QH-ADOPT per the listing."""
    rng = np.random.default_rng(15)
    P, T = 24, 10
    b1, b2, lr, eps, nu = f32(0.8), f32(0.99), f32(1e-2), f32(1e-8), f32(0.75)
    cfg = _cfg("adopt", (b1,), (nu,), beta2=b2, eps=eps, adopt_order="cur", period_x=0,
               period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    x, m, v = x0.copy(), np.zeros(P), np.zeros(P)
    for s in range(1, T + 1):
        g = rng.normal(0, 1, P)
        c = f32(s ** 0.25)
        oracle.local_step(cfg, st, g[None, :], s, lr, c)
        v = b2 * v + (1 - b2) * g * g
        n = np.clip(g / (np.sqrt(v) + eps), -c, c)
        m = b1 * m + (1 - b1) * n
        x = x - lr * ((1 - nu) * n + nu * m)
    _close(st.x[0], x, 1e-12, 1e-15, "x")
    _close(st.v[0], v, 1e-12, 1e-20, "v")


def pin_sgdm_is_qhm():
    """SGDM N=1, omega=nu is QHM (Ma & Yarats): buf = b buf + (1-b) g;
    x -= lr ((1-nu) g + nu buf)."""
    rng = np.random.default_rng(16)
    P, T = 30, 15
    b, nu, lr = f32(0.999), f32(0.7), f32(0.1)
    cfg = _cfg("sgdm", (b,), (nu,), period_x=0, period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    x, buf = x0.copy(), np.zeros(P)
    for s in range(1, T + 1):
        g = rng.normal(0, 1, P)
        oracle.local_step(cfg, st, g[None, :], s, lr)
        buf = b * buf + (1 - b) * g
        x = x - lr * ((1 - nu) * g + nu * buf)
    _close(st.x[0], x, 1e-12, 1e-15, "x")


def pin_adam_is_qhadam():
    """Adam N=1, omega=nu1 is QHAdam with nu2 = 1:
    x -= lr ((1-nu1) g + nu1 m_hat) / (sqrt(v_hat) + eps)."""
    rng = np.random.default_rng(17)
    P, T = 30, 15
    b1, b2, nu, lr, eps = f32(0.95), f32(0.98), f32(0.6), f32(1e-2), f32(1e-8)
    cfg = _cfg("adam", (b1,), (nu,), beta2=b2, eps=eps, period_x=0, period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, 1)
    x, m, v = x0.copy(), np.zeros(P), np.zeros(P)
    for s in range(1, T + 1):
        g = rng.normal(0, 1, P)
        oracle.local_step(cfg, st, g[None, :], s, lr)
        m = b1 * m + (1 - b1) * g
        v = b2 * v + (1 - b2) * g * g
        mh, vh = m / (1 - b1 ** s), v / (1 - b2 ** s)
        x = x - lr * ((1 - nu) * g + nu * mh) / (np.sqrt(vh) + eps)
    _close(st.x[0], x, 1e-12, 1e-15, "x")


# ----------------------------------------------------------------- P3, P4, P5


def pin_adam_first_step_closed_form():
    """At s=1 every bias-corrected EMA equals g and v_hat = g^2, so for any
    betas and weights x_1 = x_0 - lr g / (|g| + eps); g = 0 leaves x_0."""
    rng = np.random.default_rng(18)
    P = 50
    lr, eps = f32(1e-3), f32(1e-8)
    for betas, omegas in [((0.9, 0.99), (0.5, 0.3)), ((0.3, 0.6, 0.999), (0.1, 0.2, 0.3)),
                          ((0.0,), (0.4,))]:
        cfg = _cfg("adam", [f32(b) for b in betas], [f32(w) for w in omegas], beta2=f32(0.95),
                   eps=eps, period_x=0, period_u=(0,) * len(betas), period_v=0)
        x0 = rng.normal(0, 1, P)
        g = rng.normal(0, 1e-2, P)
        g[::7] = 0.0
        st = oracle.new_state(cfg, x0, 1)
        oracle.local_step(cfg, st, g[None, :], 1, lr)
        _close(st.x[0], x0 - lr * g / (np.abs(g) + eps), 1e-12, 1e-16, f"x {betas}")
        assert np.array_equal(st.x[0][::7], x0[::7])


def pin_constant_gradient_closed_forms():
    """A constant gradient g on every worker: syncs are no-ops, Adam moves
    x by exactly lr g/(|g|+eps) per step; SGDM by
    lr g (1 - sum_j omega_j beta_j^k) at step k (u^j_k = (1-beta_j^k) g)."""
    P, T, K = 6, 20, 3
    g = np.array([0.3, -0.01, 2.0, -1.5, 1e-3, 0.0])
    x0 = np.linspace(-1, 1, P)
    lr, eps = f32(1e-2), f32(1e-8)
    cfg = _cfg("adam", (f32(0.9), f32(0.99)), (f32(0.5), f32(0.25)), beta2=f32(0.999), eps=eps,
               period_x=3, period_u=(4, 5), period_v=7)
    st = oracle.new_state(cfg, x0, K)
    G = np.broadcast_to(g, (K, P)).copy()
    oracle.run(cfg, st, lambda s: G, range(1, T + 1), lambda s: lr)
    for m in range(K):
        _close(st.x[m], x0 - T * lr * g / (np.abs(g) + eps), 1e-11, 1e-15, "adam x")
    betas, omegas = (f32(0.9), f32(0.5)), (f32(0.3), f32(0.6))
    cfg = _cfg("sgdm", betas, omegas, period_x=2, period_u=(3, 5), period_v=0)
    st = oracle.new_state(cfg, x0, K)
    oracle.run(cfg, st, lambda s: G, range(1, T + 1), lambda s: lr)
    dist = sum(1 - sum(w * b ** k for b, w in zip(betas, omegas)) for k in range(1, T + 1))
    for m in range(K):
        _close(st.x[m], x0 - lr * g * dist, 1e-11, 1e-15, "sgdm x")
        for j in range(2):
            _close(st.u[j][m], (1 - betas[j] ** T) * g, 1e-11, 1e-16, "sgdm u")


def pin_unrolled_ema():
    """Section 2.1: from a synchronised u_t, K local steps give
    u_{t+K} = beta^K u_t + (1-beta) sum_{k=0}^{K-1} beta^k g_{t+K-k}."""
    rng = np.random.default_rng(19)
    P, Kw, H = 16, 3, 9
    b = f32(0.8)
    cfg = _cfg("sgdm", (b,), (f32(0.5),), period_x=0, period_u=(H,), period_v=0)
    st = oracle.new_state(cfg, np.zeros(P), Kw)
    G = {s: rng.normal(0, 1, (Kw, P)) for s in range(1, 2 * H + 1)}
    oracle.run(cfg, st, lambda s: G[s], range(1, H + 1), lambda s: 0.01)
    ut = st.u[0].copy()
    assert np.all(ut == ut[0]), "u not identical after its sync"
    cfg_nosync = _cfg("sgdm", (b,), (f32(0.5),), period_x=0, period_u=(0,), period_v=0)
    oracle.run(cfg_nosync, st, lambda s: G[s], range(H + 1, 2 * H + 1), lambda s: 0.01)
    for m in range(Kw):
        want = b ** H * ut[m] + (1 - b) * sum(b ** k * G[2 * H - k][m] for k in range(H))
        _close(st.u[0][m], want, 1e-12, 1e-16, "unrolled")


# ----------------------------------------------------------------- P6


def pin_local_momentum_variance():
    """Section 2.1 / Appendix derivation: from a synchronised u and iid
    N(0, sigma^2) gradients over K local steps the element variance of u is
    (1-b)/(1+b) (1 - b^{2K}) sigma^2."""
    rng = np.random.default_rng(20)
    P, K, sigma = 1 << 19, 32, 0.5
    betas = (f32(0.9), f32(0.95), f32(0.999))
    cfg = _cfg("sgdm", betas, (0.2, 0.2, 0.2), x_dtype="f32", g_dtype="f32", m_dtype="f64",
               period_x=0, period_u=(0, 0, 0), period_v=0)
    st = oracle.new_state(cfg, np.zeros(P, dtype=np.float32), 1)
    for s in range(1, K + 1):
        g = (sigma * rng.standard_normal((1, P))).astype(np.float32)
        oracle.local_step(cfg, st, g, s, 0.0)
    for j, b in enumerate(betas):
        want = (1 - b) / (1 + b) * (1 - b ** (2 * K)) * sigma ** 2
        got = float(np.var(st.u[j][0]))
        # relative std of a sample variance is sqrt(2/P) ~ 0.2 %
        assert abs(got / want - 1) < 0.012, (b, got, want)


# ----------------------------------------------------------------- P7, P8, R16


def pin_identical_gradients_make_sync_a_noop():
    """Identical per-worker gradients keep the workers identical, so every
    averaging event leaves the states bit for bit unchanged, for every form
    and storage type."""
    rng = np.random.default_rng(21)
    P, K, T = 37, 3, 12
    # (fp32 and bf16 storage: a sum of K equal fp32 values is exact in double)
    for form, xd in [("adam", "f32"), ("adopt", "bf16"), ("sgdm", "f32"), ("sgdm", "bf16")]:
        kw = dict(beta2=f32(0.99), eps=f32(1e-8), x_dtype=xd, g_dtype="f32", m_dtype="f32",
                  adopt_order="prev", clip_rho=f32(0.5) if form != "adopt" else 0.0)
        cfg_s = _cfg(form, (f32(0.9), f32(0.99)), (f32(0.3), f32(0.5)), period_x=2,
                     period_u=(3, 1), period_v=4, **kw)
        cfg_n = _cfg(form, (f32(0.9), f32(0.99)), (f32(0.3), f32(0.5)), period_x=0,
                     period_u=(0, 0), period_v=0, **kw)
        x0 = rng.normal(0, 0.1, P).astype(np.float32)
        if xd == "bf16":
            x0 = (x0.view(np.uint32) & 0xFFFF0000).view(np.float32)
        G = {s: np.broadcast_to(rng.normal(0, 0.3, P).astype(np.float32), (K, P)).copy()
             for s in range(1, T + 1)}
        xrow = x0 if xd != "bf16" else (x0.view(np.uint32) >> 16).astype(np.uint16)
        a = oracle.new_state(cfg_s, xrow, K)
        b = oracle.new_state(cfg_n, xrow, K)
        clip = (lambda s: f32(max(s - 1, 1) ** 0.25)) if form == "adopt" else (lambda s: 0.0)
        ma = oracle.run(cfg_s, a, lambda s: G[s], range(1, T + 1), lambda s: 0.01, clip)
        oracle.run(cfg_n, b, lambda s: G[s], range(1, T + 1), lambda s: 0.01, clip)
        assert any(ma), "schedule never fired"
        for p, q in zip(a.arrays(), b.arrays()):
            assert np.array_equal(p, q), form


def pin_rows_identical_after_sync_and_mean_preserved():
    """Right after its averaging event a state is identical on every worker,
    and the event keeps its worker mean (to storage rounding)."""
    rng = np.random.default_rng(22)
    P, K = 41, 5
    for dt, npdt, tol in [("f32", np.float32, 1e-7), ("f64", np.float64, 1e-15)]:
        a = rng.normal(0, 1, (K, P)).astype(npdt)
        mean_before = a.astype(np.float64).mean(axis=0)
        oracle.replica_mean(a, dt)
        assert np.all(a == a[0])
        _close(a[0], mean_before, tol, 1e-30, f"mean {dt}")
    # K = 1 is the identity
    a = rng.normal(0, 1, (1, P)).astype(np.float32)
    b = a.copy()
    oracle.replica_mean(a, "f32")
    assert np.array_equal(a, b)


def pin_virtual_average_sgdm_equals_ddp():
    """Appendix, auxiliary notation of the SGDM analysis: with linear local
    updates the worker means obey u^j = beta_j u^j + (1-beta_j) mean(g) and
    x = x - lr ((1-sum w) mean(g) + sum_j w_j u^j) for ANY periods, i.e. the
    mean trajectory is synchronous DDP-SGDM on the mean gradient.  For N=1,
    omega=1 that is torch.optim.SGD on the mean gradient."""
    rng = np.random.default_rng(23)
    P, K, T = 20, 4, 30
    b, lr = f32(0.9), f32(0.05)
    cfg = _cfg("sgdm", (b,), (1.0,), period_x=7, period_u=(5,), period_v=0)
    x0 = rng.normal(0, 1, P)
    st = oracle.new_state(cfg, x0, K)
    p = torch.tensor(x0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=lr, momentum=b, dampening=b)
    opt.state[p]["momentum_buffer"] = torch.zeros(P, dtype=torch.float64)
    G = {s: rng.normal(0, 1, (K, P)) for s in range(1, T + 1)}
    masks = oracle.run(cfg, st, lambda s: G[s], range(1, T + 1), lambda s: lr)
    for s in range(1, T + 1):
        p.grad = torch.tensor(G[s].mean(axis=0), dtype=torch.float64)
        opt.step()
    assert masks.count(0) < T
    _close(st.x.mean(axis=0), p.detach().numpy(), 1e-12, 1e-14, "mean x")
    _close(st.u[0].mean(axis=0), opt.state[p]["momentum_buffer"].numpy(), 1e-12, 1e-15, "mean u")
    # N=2 with a gradient weight: the QH DDP recursion
    betas, omegas = (f32(0.6), f32(0.99)), (f32(0.25), f32(0.5))
    cfg = _cfg("sgdm", betas, omegas, period_x=4, period_u=(3, 11), period_v=0)
    st = oracle.new_state(cfg, x0, K)
    oracle.run(cfg, st, lambda s: G[s], range(1, T + 1), lambda s: lr)
    x, u = x0.copy(), [np.zeros(P), np.zeros(P)]
    for s in range(1, T + 1):
        gm = G[s].mean(axis=0)
        u = [bj * uj + (1 - bj) * gm for bj, uj in zip(betas, u)]
        x = x - lr * ((1 - sum(omegas)) * gm + sum(w * uj for w, uj in zip(omegas, u)))
    _close(st.x.mean(axis=0), x, 1e-12, 1e-14, "QH mean x")


def pin_virtual_average_adam_moments():
    """The same identity for the Adam form's moments: for any periods the
    worker mean of u^j is the EMA of the mean gradient and the worker mean
    of v is the EMA of the mean squared gradient."""
    rng = np.random.default_rng(24)
    P, K, T = 15, 3, 25
    betas, b2 = (f32(0.9), f32(0.999)), f32(0.95)
    cfg = _cfg("adam", betas, (f32(0.4), f32(0.4)), beta2=b2, eps=f32(1e-8), period_x=2,
               period_u=(3, 8), period_v=5)
    st = oracle.new_state(cfg, rng.normal(0, 1, P), K)
    G = {s: rng.normal(0, 1, (K, P)) for s in range(1, T + 1)}
    oracle.run(cfg, st, lambda s: G[s], range(1, T + 1), lambda s: 1e-3)
    u, v = [np.zeros(P), np.zeros(P)], np.zeros(P)
    for s in range(1, T + 1):
        u = [b * uj + (1 - b) * G[s].mean(axis=0) for b, uj in zip(betas, u)]
        v = b2 * v + (1 - b2) * (G[s] ** 2).mean(axis=0)
    for j in range(2):
        _close(st.u[j].mean(axis=0), u[j], 1e-12, 1e-15, f"mean u{j}")
    _close(st.v.mean(axis=0), v, 1e-12, 1e-15, "mean v")


def pin_all_periods_one_keeps_workers_identical():
    """All periods 1 (every state averaged after every step): all workers hold
    bit-identical states after every step, for every form; for SGDM without
    clip they follow DDP-SGDM on the mean gradient."""
    rng = np.random.default_rng(25)
    P, K, T = 19, 4, 10
    for form in ("adam", "adopt", "sgdm"):
        cfg = _cfg(form, (f32(0.9), f32(0.99)), (f32(0.3), f32(0.6)), beta2=f32(0.99),
                   eps=f32(1e-8), x_dtype="f32", g_dtype="f32", m_dtype="f32", period_x=1,
                   period_u=(1, 1), period_v=1)
        st = oracle.new_state(cfg, rng.normal(0, 1, P).astype(np.float32), K)
        for s in range(1, T + 1):
            oracle.run(cfg, st, lambda s_: rng.normal(0, 1, (K, P)).astype(np.float32), [s],
                       lambda s_: 1e-2, (lambda s_: 2.0) if form == "adopt" else (lambda s_: 0.0))
            for a in st.arrays():
                assert np.all(a == a[0]), (form, s)


def pin_model_only_equals_momenta_only():
    """Section 3, for the probabilistic variant (Algorithm 4, where an
    averaged momentum feeds the same step's direction): averaging only the
    model at every step (p_x = 1, p_j = 0) is algorithmically the same as
    averaging only the momenta at every step (p_x = 0, p_j = 1): from a
    common x_0 both keep every worker on the same x, which follows DDP-SGDM
    on the mean gradient."""
    rng = np.random.default_rng(28)
    P, K, T = 13, 4, 20
    betas, omegas = (0.0, f32(0.9)), (f32(0.3), f32(0.7))
    x0 = rng.normal(0, 1, P)
    G = {s: rng.normal(0, 1, (K, P)) for s in range(1, T + 1)}
    cfg = _cfg("sgdm", betas, omegas, period_x=0, period_u=(0, 0), period_v=0)
    a, b = oracle.new_state(cfg, x0, K), oracle.new_state(cfg, x0, K)
    oracle.run_probabilistic(cfg, a, lambda s: G[s], range(1, T + 1), lambda s: f32(0.05), lambda s: 0b001)
    oracle.run_probabilistic(cfg, b, lambda s: G[s], range(1, T + 1), lambda s: f32(0.05), lambda s: 0b110)
    x, u = x0.copy(), [np.zeros(P), np.zeros(P)]
    for s in range(1, T + 1):
        gm = G[s].mean(axis=0)
        u = [bj * uj + (1 - bj) * gm for bj, uj in zip(betas, u)]
        x = x - f32(0.05) * sum(w * uj for w, uj in zip(omegas, u))
    for m in range(K):
        _close(a.x[m], x, 1e-12, 1e-14, "model-only")
        _close(b.x[m], x, 1e-12, 1e-14, "momenta-only")
    # the deterministic order (Algorithm 3: the local momentum feeds the
    # step, the average is the next base) does not have this property
    c = oracle.new_state(cfg, x0, K)
    oracle.run(cfg, c, lambda s: G[s], range(1, T + 1), lambda s: f32(0.05), masks=lambda s: 0b110)
    assert np.abs(c.x - c.x[0]).max() > 1e-3


def pin_probabilistic_sync_virtual_average():
    """Algorithm 4 with drawn events (probabilities p_x, p_j; sum of omega =
    1; the gradient as a beta = 0 momentum): for any event sequence the
    worker mean of x follows DDP-SGDM on the mean gradient; with no events
    it is Algorithm 3 without averaging."""
    import synth

    rng = np.random.default_rng(29)
    P, K, T = 11, 3, 40
    betas, omegas = (0.0, f32(0.95)), (f32(0.25), f32(0.75))
    cfg = _cfg("sgdm", betas, omegas, period_x=0, period_u=(0, 0), period_v=0)
    masks = synth.bernoulli_masks(7, T, 2, 1 / 4, (1 / 2, 1 / 8))
    assert any(m & 1 for m in masks) and any(m & 6 for m in masks) and 0 in masks
    x0 = rng.normal(0, 1, P)
    G = {s: rng.normal(0, 1, (K, P)) for s in range(1, T + 1)}
    st = oracle.new_state(cfg, x0, K)
    applied = oracle.run_probabilistic(cfg, st, lambda s: G[s], range(1, T + 1), lambda s: f32(0.02),
                                       lambda s: masks[s - 1])
    assert applied == masks
    x, u = x0.copy(), [np.zeros(P), np.zeros(P)]
    for s in range(1, T + 1):
        gm = G[s].mean(axis=0)
        u = [b * uj + (1 - b) * gm for b, uj in zip(betas, u)]
        x = x - f32(0.02) * sum(w * uj for w, uj in zip(omegas, u))
    _close(st.x.mean(axis=0), x, 1e-12, 1e-14, "mean x")
    a, b = oracle.new_state(cfg, x0, K), oracle.new_state(cfg, x0, K)
    oracle.run_probabilistic(cfg, a, lambda s: G[s], range(1, T + 1), lambda s: f32(0.02), lambda s: 0)
    oracle.run(cfg, b, lambda s: G[s], range(1, T + 1), lambda s: f32(0.02))
    for p_, q_ in zip(a.arrays(), b.arrays()):
        assert np.array_equal(p_, q_)


def pin_outer_nesterov_unit_lr_no_momentum_is_averaging():
    """OuterOpt = Nesterov with outer_lr = 1, mu = 0 is the default
    averaging: the outer parameters become the worker mean."""
    rng = np.random.default_rng(30)
    P, K, T = 17, 3, 24
    kw = dict(beta2=f32(0.99), eps=f32(1e-8), period_x=4, period_u=(3, 0), period_v=5)
    a_cfg = _cfg("adam", (f32(0.9), f32(0.99)), (f32(0.3), f32(0.5)), **kw)
    b_cfg = _cfg("adam", (f32(0.9), f32(0.99)), (f32(0.3), f32(0.5)), outer="nesterov", outer_lr=1.0,
                 outer_momentum=0.0, **kw)
    x0 = rng.normal(0, 1, P)
    G = {s: rng.normal(0, 1, (K, P)) for s in range(1, T + 1)}
    a, b = oracle.new_state(a_cfg, x0, K), oracle.new_state(b_cfg, x0, K)
    oracle.run(a_cfg, a, lambda s: G[s], range(1, T + 1), lambda s: f32(1e-2))
    oracle.run(b_cfg, b, lambda s: G[s], range(1, T + 1), lambda s: f32(1e-2))
    # the outer parameters are kept in fp32: agreement to fp32 rounding
    _close(b.x, a.x, 3e-7, 1e-12, "nesterov(1, 0) vs averaging")
    _close(b.x_outer, b.x[0], 0, 0, "workers restart from the outer parameters")
    assert np.all(b.outer_mom == 0) or np.max(np.abs(b.outer_mom)) < 1.0


def pin_outer_nesterov_is_torch_sgd_nesterov():
    """At every averaging event of x the outer parameters take one step of
    torch.optim.SGD(lr, momentum, nesterov=True) on the outer gradient
    x_outer - mean_m(x^m), and every worker restarts from them."""
    rng = np.random.default_rng(31)
    P, K, T = 20, 3, 36
    lr_out, mu = f32(0.7), f32(0.9)
    cfg = _cfg("sgdm", (f32(0.9),), (f32(0.8),), period_x=4, period_u=(6,), period_v=0,
               outer="nesterov", outer_lr=lr_out, outer_momentum=mu)
    x0 = rng.normal(0, 1, P).astype(np.float32).astype(np.float64)  # fp32 outer copy holds x0 exactly
    st = oracle.new_state(cfg, x0, K)
    p = torch.tensor(x0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=lr_out, momentum=mu, nesterov=True)
    events = 0
    for s in range(1, T + 1):
        g = rng.normal(0, 1, (K, P))
        oracle.local_step(cfg, st, g, s, f32(0.05))
        mask = oracle.schedule(cfg, s)
        if mask & 1:
            mean = st.x.astype(np.float64).mean(axis=0)
            p.grad = p.detach() - torch.tensor(mean, dtype=torch.float64)
            opt.step()
            events += 1
        oracle.sync(cfg, st, mask)
        if mask & 1:
            _close(st.x_outer, p.detach().numpy(), 2e-6, 1e-9, f"outer params s={s}")
            _close(st.outer_mom, opt.state[p]["momentum_buffer"].numpy(), 2e-6, 1e-9, f"outer mom s={s}")
            for m in range(K):
                _close(st.x[m], st.x_outer, 0, 0, "restart")
            p.data = torch.tensor(st.x_outer.astype(np.float64))  # follow the fp32 outer copy
            opt.state[p]["momentum_buffer"] = torch.tensor(st.outer_mom.astype(np.float64))
    assert events == T // 4


def pin_state_stats_definitions():
    """Averaging diagnostics: a hand example, identical rows (variance 0,
    cosine 1), opposite rows (mean 0, variance = ||S^0||^2), and the
    identity var = mean_m ||c^m||^2 - ||cbar||^2 on random rows; with outer
    parameters the vectors are the pseudo-gradients x_outer - x^m."""
    a = np.array([[1.0, 2.0], [3.0, 4.0]])
    st = oracle.state_stats(a, "f64")
    assert np.allclose(st, [13.0, 2.0, 0.0, 0.0, 5.0, 25.0, 8.0, 18.0], rtol=0, atol=1e-12), st
    rng = np.random.default_rng(32)
    r = rng.normal(0, 1, 50)
    st = oracle.state_stats(np.tile(r, (3, 1)), "f64")
    _close(st[[4, 5, 6, 7, 8, 9]], [r @ r] * 6, 1e-12, 0, "identical rows")
    assert abs(st[1]) < 1e-12 * (r @ r)
    st = oracle.state_stats(np.stack([r, -r]), "f64")
    assert abs(st[0]) < 1e-20 and abs(st[1] - r @ r) < 1e-12 * (r @ r)
    b = rng.normal(0, 1, (5, 40))
    st = oracle.state_stats(b, "f64")
    _close(st[1], (b * b).sum(axis=1).mean() - st[0], 1e-10, 0, "variance identity")
    _close(st[4 + 5:], b @ b.mean(axis=0), 1e-12, 1e-14, "dots")
    xo = rng.normal(0, 1, 40).astype(np.float32)
    st = oracle.state_stats(b, "f64", xo)
    pg = xo.astype(np.float64) - b
    _close(st[0], ((xo - b.mean(axis=0)) ** 2).sum(), 1e-12, 0, "pseudo-gradient mean")
    _close(st[2], float(xo.astype(np.float64) @ xo.astype(np.float64)), 1e-12, 0, "outer norm")
    _close(st[4:9], (pg * pg).sum(axis=1), 1e-12, 0, "pseudo-gradient norms")
    _close(st[9:14], pg @ pg.mean(axis=0), 1e-12, 1e-14, "pseudo-gradient dots with their mean")
    _close(st[1], ((pg - pg.mean(axis=0)) ** 2).sum() / 5, 1e-12, 0, "pseudo-gradient variance")


def pin_cross_worker_variance_of_local_momentum():
    """Section 2.1 / Appendix derivation, measured with the diagnostic:
    from a synchronised momentum, K local steps of iid N(0, sigma^2)
    gradients (independent across workers) give a cross-worker variance of
    (1 - 1/M) P (1-b)/(1+b) (1 - b^{2K}) sigma^2 in expectation."""
    rng = np.random.default_rng(33)
    M, P, H, sigma, b = 8, 1 << 16, 32, 0.3, f32(0.9)
    cfg = _cfg("sgdm", (b,), (0.5,), x_dtype="f32", g_dtype="f32", m_dtype="f64", period_x=0,
               period_u=(0,), period_v=0)
    st = oracle.new_state(cfg, np.zeros(P, dtype=np.float32), M)
    for s in range(1, H + 1):
        oracle.local_step(cfg, st, (sigma * rng.standard_normal((M, P))).astype(np.float32), s, 0.0)
    stats = oracle.sync_stats(cfg, st, 0b10)
    want = (1 - 1 / M) * P * (1 - b) / (1 + b) * (1 - b ** (2 * H)) * sigma ** 2
    assert abs(stats[1][1] / want - 1) < 0.02, (stats[1][1], want)
    assert np.all(st.u[0] == st.u[0][0]), "averaged after the diagnostics"


# ----------------------------------------------------------------- P9, P11 (paper numbers)


def _paper_values():
    with open(os.path.join(GOLDEN, "paper_values.json")) as f:
        return json.load(f)


def pin_schedule_counts_and_comm_reduction():
    """The number of averaging events of state S in T steps is floor(T/H_S);
    the per-step communicated fraction sum_S 1/H_S is the inverse of the
    communication reduction of Section 2.3, which at K=32, N=1 is the
    paper's "10x less than DDP" (Section 5.3)."""
    pv = _paper_values()
    for (hx, hu, hv, n, T) in [(4, (8, 8), 16, 2, 32), (32, (64, 64, 64), 128, 3, 256),
                               (3, (5,), 7, 1, 100), (1, (1, 2), 0, 2, 9)]:
        cfg = _cfg("adam", (0.9,) * n, (0.1,) * n, period_x=hx, period_u=hu, period_v=hv)
        masks = [oracle.schedule(cfg, s) for s in range(1, T + 1)]
        assert sum(m & 1 for m in masks) == T // hx
        for j in range(n):
            assert sum((m >> (j + 1)) & 1 for m in masks) == T // hu[j]
        assert sum((m >> (n + 1)) & 1 for m in masks) == (T // hv if hv else 0)
        assert all(m >> (n + 2) == 0 for m in masks)
    sgdm = _cfg("sgdm", (0.9,), (0.5,), period_x=2, period_u=(2,), period_v=2)
    assert all(oracle.schedule(sgdm, s) >> 2 == 0 for s in range(1, 20)), "SGDM has no v"
    K = pv["comm_reduction"]["K"]
    cfg = _cfg("adam", (0.9,), (0.5,), period_x=K, period_u=(K,), period_v=K)
    T = 100 * K
    events = sum(bin(oracle.schedule(cfg, s)).count("1") for s in range(1, T + 1))
    # DDP sends one model-sized payload per step, MT-DAO one per averaging
    # event: the ratio is (1/K_x + 1/K_1 + 1/K_v)^-1
    reduction = T / events
    assert abs(reduction - pv["comm_reduction"]["closed_form"]) < 1e-9
    assert math.floor(reduction) == pv["comm_reduction"]["paper_statement"]


def pin_ema_decay_paper_numbers():
    """Section 2.1: with no new gradient a synchronised momentum keeps a
    beta^K share of itself -- about 0.03 for beta = 0.9, K = 32 -- and its
    half-life ln 0.5 / ln beta is about 6.6 steps at beta = 0.9; Table 5's
    half-life periods 69 / 693 / 6931 for beta = 0.99 / 0.999 / 0.9999."""
    pv = _paper_values()
    e = pv["ema_retention"]
    cfg = _cfg("sgdm", (f32(e["beta"]),), (0.5,), period_x=0, period_u=(0,), period_v=0)
    st = oracle.new_state(cfg, np.zeros(1), 1)
    st.u[0][:] = 1.0
    for s in range(1, e["K"] + 1):
        oracle.local_step(cfg, st, np.zeros((1, 1)), s, 0.0)
    assert round(float(st.u[0][0, 0]), 2) == e["paper_value"]
    for row in pv["half_life"]:
        b, periods = row["beta"], row["paper_steps"]
        tau = math.log(0.5) / math.log(b)
        assert round(tau, 1) == row.get("paper_tau", round(tau, 1))
        assert round(tau) == periods
        cfg = _cfg("sgdm", (f32(b),), (0.5,), period_x=0, period_u=(0,), period_v=0)
        st = oracle.new_state(cfg, np.zeros(1), 1)
        st.u[0][:] = 1.0
        for s in range(1, periods + 1):
            oracle.local_step(cfg, st, np.zeros((1, 1)), s, 0.0)
        assert abs(float(st.u[0][0, 0]) - 0.5) < 0.5 * (1 - b) + 1e-4, (b, st.u[0][0, 0])


# ----------------------------------------------------------------- P10


def pin_hand_worked_examples():
    """3-element, 2-worker examples computed by hand in decimal arithmetic
    under the readings of the oracle (Adam with bias correction and a
    mixed sync schedule; SGDM with the global-norm clip; ADOPT in both
    orders).  Tolerance 5e-5 relative: the oracle receives fp32 hyper-
    parameters while the hand calculation used exact decimals, and the
    fp32 rounding of 0.999 and 0.9999 moves 1 - beta by 1.3e-5 and 1.7e-5
    relative."""
    with open(os.path.join(GOLDEN, "hand_worked_examples.json")) as f:
        ex = json.load(f)
    for case in ex["cases"]:
        h = case["hyper"]
        cfg = _cfg(case["form"], [f32(b) for b in h["beta1"]], [f32(w) for w in h["omega"]],
                   beta2=f32(h.get("beta2", 0.0)), eps=f32(h.get("eps", 0.0)),
                   clip_rho=f32(h.get("clip_rho", 0.0)), adopt_order=h.get("adopt_order", "prev"),
                   period_x=h["period_x"], period_u=tuple(h["period_u"]), period_v=h.get("period_v", 0))
        st = oracle.new_state(cfg, np.array(ex["x0"]), 2)
        for step in case["steps"]:
            s = step["s"]
            g = np.array(step["grads"])
            c = 0.0
            if case["form"] == "adopt":
                t = s - 1 if cfg.adopt_order == "prev" else s
                c = f32(t ** 0.25) if t > 0 else 0.0
            sc = oracle.clip_scales(cfg, g)
            if "scales" in step:
                _close(sc, step["scales"], 1e-7, 0, f"{case['name']} s={s} clip scale")
            oracle.local_step(cfg, st, g, s, f32(h["lr"]), c, sc)
            for key, want in step.get("after_step", {}).items():
                r = int(key[1])
                _close(st.x[r], want, 5e-5, 1e-12, f"{case['name']} s={s} {key} x")
            mask = oracle.schedule(cfg, s)
            assert mask == step["mask"], (case["name"], s, mask)
            oracle.sync(cfg, st, mask)
            for name, want in step.get("after_sync", {}).items():
                arr = {"x": st.x, "v": st.v}.get(name)
                if arr is None:
                    arr = st.u[int(name[1:]) - 1]
                for r in range(2):
                    _close(arr[r], want, 5e-5, 1e-12, f"{case['name']} s={s} sync {name}")


# ----------------------------------------------------------------- P12 and storage


def _numpy_restatement(form, betas, omegas, b2, eps, order, bc, hx, hu, hv, rho, x0, G, lrs, cs):
    """Independent vectorised restatement of Algorithms 1-3 (float64, no
    storage rounding) used only by the brute-force pin."""
    K, P = G[1].shape
    N = len(betas)
    x = np.tile(x0, (K, 1)).astype(np.float64)
    u = np.zeros((N, K, P))
    v = np.zeros((K, P))
    wsum = sum(omegas)
    masks = []
    for s in sorted(G):
        g = G[s].astype(np.float64)
        if rho > 0 and form != "adopt":
            n = np.sqrt((g ** 2).sum(axis=1, keepdims=True))
            g = g * np.where(n > 0, np.minimum(1.0, rho / np.where(n > 0, n, 1.0)), 1.0)
        B = np.array(betas)[:, None, None]
        W = np.array(omegas)[:, None, None]
        if form == "adam":
            u = B * u + (1 - B) * g[None]
            v = b2 * v + (1 - b2) * g * g
            corr = (1 - B ** s) if bc else np.ones_like(B)
            vh = v / ((1 - b2 ** s) if bc else 1.0)
            x = x - lrs[s] * ((1 - wsum) * g + (W * u / corr).sum(0)) / (np.sqrt(vh) + eps)
        elif form == "adopt":
            if order == "prev" and s == 1:
                v = g * g
            else:
                if order == "prev":
                    n_ = g / (np.sqrt(v) + eps)
                    v = b2 * v + (1 - b2) * g * g
                else:
                    v = b2 * v + (1 - b2) * g * g
                    n_ = g / (np.sqrt(v) + eps)
                if cs[s] > 0:
                    n_ = np.clip(n_, -cs[s], cs[s])
                u = B * u + (1 - B) * n_[None]
                x = x - lrs[s] * ((1 - wsum) * n_ + (W * u).sum(0))
        else:
            u = B * u + (1 - B) * g[None]
            x = x - lrs[s] * ((1 - wsum) * g + (W * u).sum(0))
        mask = 0
        if hx and s % hx == 0:
            x[:] = x.mean(0)
            mask |= 1
        for j in range(N):
            if hu[j] and s % hu[j] == 0:
                u[j][:] = u[j].mean(0)
                mask |= 1 << (j + 1)
        if form != "sgdm" and hv and s % hv == 0:
            v[:] = v.mean(0)
            mask |= 1 << (N + 1)
        masks.append(mask)
    return x, u, v, masks


def pin_brute_force_tiny():
    """Random tiny problems (K <= 3, P <= 5, T <= 8) over every form and
    order, random hyper-parameters and periods: the oracle in fp64 storage
    equals an independent vectorised numpy restatement."""
    rng = np.random.default_rng(26)
    for trial in range(60):
        form = ["adam", "adopt", "sgdm"][trial % 3]
        N = int(rng.integers(1, 5))
        K = int(rng.integers(1, 4))
        P = int(rng.integers(1, 6))
        T = int(rng.integers(1, 9))
        betas = [f32(b) for b in rng.uniform(0, 0.999, N)]
        w = rng.uniform(0, 1, N)
        w = w / max(1.0, w.sum()) * rng.uniform(0.2, 1.0)
        omegas = [f32(a) for a in w]
        b2 = f32(rng.uniform(0.5, 0.9999))
        eps = f32(10.0 ** rng.uniform(-9, -3))
        order = ["prev", "cur"][int(rng.integers(0, 2))]
        bc = bool(rng.integers(0, 2))
        rho = f32(rng.uniform(0.1, 2.0)) if (form != "adopt" and rng.integers(0, 2)) else 0.0
        hx, hv = int(rng.integers(0, 4)), int(rng.integers(0, 4))
        hu = [int(a) for a in rng.integers(0, 4, N)]
        x0 = rng.normal(0, 1, P)
        G = {s: rng.normal(0, 1, (K, P)) * (rng.uniform(0, 3, (K, 1)) if rho else 1.0)
             for s in range(1, T + 1)}
        G[1][:, 0] = 0.0 if trial % 5 == 0 else G[1][:, 0]
        lrs = {s: f32(rng.uniform(1e-3, 0.1)) for s in G}
        cs = {s: (f32(rng.uniform(0.3, 2.0)) if rng.integers(0, 2) else 0.0) for s in G}
        cfg = _cfg(form, betas, omegas, beta2=b2, eps=eps, adopt_order=order, bias_correction=bc,
                   clip_rho=rho, period_x=hx, period_u=tuple(hu), period_v=hv)
        st = oracle.new_state(cfg, x0, K)
        masks = oracle.run(cfg, st, lambda s: G[s], range(1, T + 1), lambda s: lrs[s],
                           lambda s: cs[s])
        x, u, v, m2 = _numpy_restatement(form, betas, omegas, b2, eps, order, bc, hx, hu, hv, rho,
                                         x0, G, lrs, cs)
        assert masks == m2, (trial, masks, m2)
        _close(st.x, x, 1e-10, 1e-13, f"trial {trial} x")
        for j in range(N):
            _close(st.u[j], u[j], 1e-10, 1e-13, f"trial {trial} u{j}")
        if form != "sgdm":
            _close(st.v, v, 1e-10, 1e-16, f"trial {trial} v")


def _bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _bf16_by_fractions(v: float) -> float:
    """Independent bf16 rounding in exact rational arithmetic: 8
    significant bits, quantum never below 2^-133, ties to even (Python's
    round() on a Fraction rounds half to even), overflow to infinity."""
    from fractions import Fraction
    if v == 0:
        return 0.0
    a = Fraction(abs(v))
    e = 0
    while a >= Fraction(2) ** e:
        e += 1
    while a < Fraction(2) ** (e - 1):
        e -= 1
    q = Fraction(2) ** max(e - 8, -133)
    r = round(a / q) * q
    if r > 255 * Fraction(2) ** 120:
        return math.copysign(math.inf, v)
    return math.copysign(float(r), v)


def pin_storage_rounding():
    """Each store rounds once to its type with round-to-nearest-even:
    fp32 stores equal numpy's float32 cast of the fp64 value; bf16 stores
    keep 8 significant bits with ties to even, overflow to infinity and
    the bf16 subnormal range."""
    rng = np.random.default_rng(27)
    cfg = _cfg("sgdm", (0.0,), (0.0,), x_dtype="f32", g_dtype="f64", m_dtype="f64", period_x=0,
               period_u=(0,), period_v=0)
    x0 = rng.normal(0, 1, 1000).astype(np.float32)
    g = rng.normal(0, 1, (1, 1000))
    st = oracle.new_state(cfg, x0, 1)
    oracle.local_step(cfg, st, g, 1, f32(0.37))
    want = (x0.astype(np.float64) - f32(0.37) * g[0]).astype(np.float32)
    assert np.array_equal(st.x[0], want)
    # bf16: x = 0 - 1 * (-value) stores value rounded to bf16
    vals = [1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -30, -(1 + 2 ** -8),
            2.0 ** 127 * (1 + 2 ** -8), 255.5 * 2.0 ** 120, 3.4e38, 2.0 ** -130, 2.0 ** -134,
            2.0 ** -133 * 1.5, 2.0 ** -126 * (1 + 2 ** -8), 0.1, -7.77e-3]
    vals += list(rng.normal(0, 1, 200) * 10.0 ** rng.uniform(-40, 38, 200))
    vals = np.array(vals)
    want = np.array([_bf16_by_fractions(float(a)) for a in vals])
    assert want[0] == 1.0 and want[1] == 1.0 and want[2] == 1 + 2 ** -6 and np.isinf(want[6])
    cfg = _cfg("sgdm", (0.0,), (0.0,), x_dtype="bf16", g_dtype="f64", m_dtype="f64", period_x=0,
               period_u=(0,), period_v=0)
    st = oracle.new_state(cfg, np.zeros(vals.size, dtype=np.uint16), 1)
    oracle.local_step(cfg, st, -vals[None, :], 1, 1.0)
    got = _bits_to_f32(st.x[0]).astype(np.float64)
    assert np.array_equal(got, want), [(a, b, c) for a, b, c in zip(vals, got, want) if b != c][:5]


def pin_clip_scale():
    """clip(g, rho): per-worker global L2 norm, scale min(1, rho/||g||),
    1 for a zero norm or a disabled clip; computed over all elements."""
    g = np.array([[3.0, 4.0, 0.0], [0.0, 0.0, 0.0], [0.3, 0.0, 0.4]])
    cfg = _cfg("sgdm", (0.0,), (0.0,), clip_rho=1.0, period_x=0, period_u=(0,), period_v=0)
    sc = oracle.clip_scales(cfg, g)
    assert np.allclose(sc, [0.2, 1.0, 1.0], rtol=0, atol=1e-15)
    assert oracle.clip_scale(5.0, 0.0) == 1.0
    assert abs(oracle.sumsq(np.arange(10, dtype=np.float32)) - 285.0) < 1e-12


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]
