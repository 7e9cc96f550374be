"""Pins of the oracle's cart-pole step (CPU only).

Nothing here retypes the oracle's formula.  The step is checked against:

* hand-derived exact rational values of the first two steps from rest
  (tests/golden/cartpole_rational_steps.txt);
* the Euler-Lagrange equations of a cart carrying a uniform rod written in
  mass-matrix form and solved by a 50-digit linear solve (a different
  formulation from the oracle's closed-form elimination);
* the small-angle linearisation, a constant-coefficient linear system;
* conservation of horizontal momentum and of energy of the unforced system,
  whose explicit-Euler drift must vanish to first order in the time step;
* textbook sin/cos for the series the step uses;
* strict thresholds, including exact threshold values and NaN.
"""
import math
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))
P = oracle.make_params(**workloads.CARTPOLE)
F32 = np.float32


def _ulp(x):
    x = abs(float(F32(x)))
    return float(np.spacing(F32(max(x, 1e-30))))


def test_rational_first_steps():
    rows = []
    with open(os.path.join(HERE, "golden", "cartpole_rational_steps.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(line.split())
    assert len(rows) == 4
    for action in (1, 0):
        s = np.zeros(4, dtype=np.float32)
        for step in (1, 2):
            s = oracle.cartpole_step(P, s, action)
            want = next(r for r in rows if int(r[0]) == step and int(r[1]) == action)
            for c in range(4):
                exact = Fraction(want[2 + c])
                # fp32 constants (0.1f, 9.8f, 0.02f ...) differ from the exact
                # rationals by < 1 ulp each: allow 4 ulp of the exact value
                tol = 4 * _ulp(float(exact)) if exact != 0 else 0.0
                assert abs(float(s[c]) - float(exact)) <= tol, (action, step, c, s[c], exact)


def _exact_f32(v):
    return mpmath.mpf(float(F32(v)))


def _lagrange_step(state, action, params=workloads.CARTPOLE):
    """One Euler step from the Euler-Lagrange mass-matrix equations in 50 digits,
    with the fp32 values of the constants and exact sin/cos:
        [ M          m l cos th ] [xacc ]   [ F + m l thd^2 sin th ]
        [ m l cos th 4/3 m l^2  ] [thacc] = [ m g l sin th         ]"""
    with mpmath.workdps(50):
        g = _exact_f32(params["gravity"])
        mc = _exact_f32(params["masscart"])
        m = _exact_f32(params["masspole"])
        l = _exact_f32(params["half_length"])
        tau = _exact_f32(params["tau"])
        fm = _exact_f32(params["force_mag"])
        x, xd, th, thd = (mpmath.mpf(float(v)) for v in state)
        F = fm if action else -fm
        M = mc + m
        A = mpmath.matrix([[M, m * l * mpmath.cos(th)], [m * l * mpmath.cos(th), mpmath.mpf(4) / 3 * m * l * l]])
        rhs = mpmath.matrix([F + m * l * thd**2 * mpmath.sin(th), m * g * l * mpmath.sin(th)])
        xacc, thacc = mpmath.lu_solve(A, rhs)
        return [x + tau * xd, xd + tau * xacc, th + tau * thd, thd + tau * thacc], (xacc, thacc)


def test_one_step_matches_euler_lagrange():
    rng = np.random.Generator(np.random.PCG64(11))
    thr = workloads.CARTPOLE["theta_threshold_rad"]
    worst = 0.0
    for i in range(400):
        st = np.array([rng.uniform(-2.4, 2.4), rng.uniform(-3, 3),
                       rng.uniform(-thr, thr), rng.uniform(-4, 4)], dtype=np.float32)
        if i < 20:   # include tiny states near the origin
            st = (st * 1e-3).astype(np.float32)
        a = int(rng.integers(0, 2))
        got = oracle.cartpole_step(P, st, a)
        want, (xacc, thacc) = _lagrange_step(st, a)
        tau = float(F32(workloads.CARTPOLE["tau"]))
        for c in range(4):
            # the position/velocity update rounds once (0.5 ulp of the result);
            # the acceleration carries ~10 roundings relative to its own size
            # and enters scaled by tau.
            acc = float(xacc if c == 1 else thacc)
            bound = 0.5 * _ulp(got[c]) + tau * 12 * 2.0**-24 * (abs(acc) + 15.0)
            if c in (0, 2):
                bound = 0.5 * _ulp(got[c]) + 1e-30
            err = abs(float(got[c]) - float(want[c]))
            worst = max(worst, err / bound)
            assert err <= bound, (i, c, st, a, float(got[c]), float(want[c]))
    assert worst > 0.0


def test_sin_cos_series_match_textbook():
    thr = workloads.CARTPOLE["theta_threshold_rad"]
    xs = np.linspace(-math.pi / 4, math.pi / 4, 20001).astype(np.float32)
    for th in xs:
        s, c = oracle.sin_poly(th), oracle.cos_poly(th)
        ts, tc = math.sin(float(th)), math.cos(float(th))
        # within the fp32 threshold domain: 1 ulp; up to pi/4: 2 ulp + truncation 3e-8
        if abs(th) <= thr:
            assert abs(float(s) - ts) <= _ulp(ts), th
            assert abs(float(c) - tc) <= _ulp(tc), th
        else:
            assert abs(float(s) - ts) <= 2 * _ulp(ts) + 3e-8, th
            assert abs(float(c) - tc) <= 2 * _ulp(tc) + 3e-8, th
    assert oracle.sin_poly(0.0) == 0.0 and oracle.cos_poly(0.0) == 1.0
    # odd / even symmetry
    for th in (0.01, 0.1, 0.2):
        assert oracle.sin_poly(-th) == -oracle.sin_poly(th)
        assert oracle.cos_poly(-th) == oracle.cos_poly(th)


def test_small_angle_linearisation():
    """For |th|, |thd| small the step is the affine map z' = (I + tau A) z + tau c
    with kappa = g / (l (4/3 - m/M)):
        thacc = kappa th - F / (M l (4/3 - m/M)),  xacc = F/M - (m l / M) thacc."""
    c = workloads.CARTPOLE
    g, mc, m, l, tau, fm = (float(F32(c[k])) for k in ("gravity", "masscart", "masspole", "half_length", "tau", "force_mag"))
    M = mc + m
    denom = l * (4.0 / 3.0 - m / M)
    kappa = g / denom
    for action in (0, 1, None):
        F = 0.0 if action is None else (fm if action else -fm)
        params = P if action is not None else oracle.make_params(**workloads.cartpole(force_mag=0.0))
        a_in = 1 if action is None else action
        A = np.array([[0, 1, 0, 0],
                      [0, 0, -(m * l / M) * kappa, 0],
                      [0, 0, 0, 1],
                      [0, 0, kappa, 0]], dtype=np.float64)
        cvec = np.array([0, F / M + (m * l / M) * F / (M * denom), 0, -F / (M * denom)])
        z = np.array([1e-4, -2e-4, 3e-4, -1e-4])
        s = z.astype(np.float32)
        zl = s.astype(np.float64)
        # unforced: 5 steps stay in the linear regime; forced: one step (the
        # force drives thd to O(1) within a few steps)
        steps = 5 if action is None else 1
        for _ in range(steps):
            s = oracle.cartpole_step(params, s, a_in)
            zl = zl + tau * (A @ zl + cvec)
        err = np.abs(s.astype(np.float64) - zl)
        # neglected terms: O(th^3), O(th thd^2) and F th^2 ~ 1e-6 in the
        # acceleration (x tau); fp32 rounding: a few units of 2^-24 relative
        nonlin = 1e-12 if action is None else 3e-8
        assert np.all(err <= nonlin + 5 * 2.0**-24 * np.abs(zl)), (action, err)
        # and the linear map is not trivially satisfied: the state moved
        assert np.all(np.abs(zl - z.astype(np.float32)) > 0) or action is None


def _momentum(s, c):
    M = float(F32(c["masscart"])) + float(F32(c["masspole"]))
    ml = float(F32(c["masspole"])) * float(F32(c["half_length"]))
    return M * float(s[1]) + ml * float(s[3]) * math.cos(float(s[2]))


def _energy(s, c):
    mc, m, l, g = (float(F32(c[k])) for k in ("masscart", "masspole", "half_length", "gravity"))
    M = mc + m
    x, xd, th, thd = (float(v) for v in s)
    return 0.5 * M * xd * xd + m * l * xd * thd * math.cos(th) + (2.0 / 3.0) * m * l * l * thd * thd + m * g * l * math.cos(th)


@pytest.mark.parametrize("quantity", ["momentum", "energy"])
def test_unforced_conservation_first_order(quantity):
    """With F = 0 the continuous system conserves horizontal momentum and energy;
    explicit Euler drifts by O(tau) over a fixed time, so halving tau halves the
    drift.  A wrong or missing term leaves an O(1) drift as tau -> 0."""
    fn = _momentum if quantity == "momentum" else _energy
    horizon = 0.24     # seconds; keeps |theta| below pi/4 from this start
    drifts = []
    for tau in (0.004, 0.002, 0.001):
        c = workloads.cartpole(force_mag=0.0, tau=tau, no_termination=1, max_episode_steps=0)
        params = oracle.make_params(**c)
        s = np.array([0.0, 0.7, 0.15, -2.5], dtype=np.float32)
        e0 = fn(s, c)
        steps = int(round(horizon / tau))
        for _ in range(steps):
            s = oracle.cartpole_step(params, s, 1)
            assert abs(float(s[2])) < math.pi / 4
        drifts.append(fn(s, c) - e0)
    d = np.array(drifts)
    assert abs(d[0]) > 1e-4               # the drift is real at the coarse step ...
    r1, r2 = d[0] / d[1], d[1] / d[2]     # ... and first order in tau
    assert 1.7 < r1 < 2.3 and 1.7 < r2 < 2.3, d


def test_forced_energy_input():
    """With the force on, the work done per step is F xd tau to first order."""
    c = workloads.cartpole(tau=0.0005, no_termination=1, max_episode_steps=0)
    params = oracle.make_params(**c)
    s = np.array([0.0, 0.3, 0.05, 0.4], dtype=np.float32)
    work = 0.0
    e0 = _energy(s, c)
    for _ in range(200):
        work += 10.0 * float(s[1]) * 0.0005
        s = oracle.cartpole_step(params, s, 1)
    assert abs((_energy(s, c) - e0) - work) < 0.02 * abs(work)


def test_thresholds_strict_and_nan():
    thr_x = float(F32(2.4))
    thr_th = workloads.CARTPOLE["theta_threshold_rad"]
    assert F32(thr_th).view(np.uint32) == 0x3E567750
    on = lambda x, th: oracle.terminated(P, np.array([x, 0, th, 0], dtype=np.float32))  # noqa: E731
    assert not on(thr_x, 0.0) and not on(-thr_x, 0.0)
    assert on(float(np.nextafter(F32(thr_x), F32(10))), 0.0)
    assert on(-float(np.nextafter(F32(thr_x), F32(10))), 0.0)
    assert not on(0.0, thr_th) and not on(0.0, -thr_th)
    assert on(0.0, float(np.nextafter(F32(thr_th), F32(1)))) and on(0.0, -float(np.nextafter(F32(thr_th), F32(1))))
    assert not on(float("nan"), float("nan"))
    assert on(float("inf"), 0.0)
    noterm = oracle.make_params(**workloads.cartpole(no_termination=1))
    assert not oracle.terminated(noterm, np.array([100, 0, 3, 0], dtype=np.float32))


def test_compute_factor_one_is_the_plain_step():
    rng = np.random.Generator(np.random.PCG64(21))
    for _ in range(200):
        st = rng.uniform(-0.2, 0.2, 4).astype(np.float32)
        a = int(rng.integers(0, 2))
        assert np.array_equal(oracle.env_step(P, st, a), oracle.cartpole_step(P, st, a))


def test_compute_factor_converges_first_order():
    """C Euler iterations of tau / C approach the exact flow of the ODE over one
    step as C grows, with error halving when C doubles (first-order method).
    Reference: the same Euler-Lagrange mass-matrix ODE integrated with a
    50-digit classical Runge-Kutta method on a fine grid."""
    state0 = np.array([0.1, 0.5, 0.12, -1.5], dtype=np.float32)

    def rk4_flow(y0, F, tau, steps=400):
        c = workloads.CARTPOLE
        with mpmath.workdps(40):
            g, mc, m, l = (mpmath.mpf(float(F32(c[k]))) for k in ("gravity", "masscart", "masspole", "half_length"))
            M = mc + m

            def f(y):
                x, xd, th, thd = y
                A = mpmath.matrix([[M, m * l * mpmath.cos(th)], [m * l * mpmath.cos(th), mpmath.mpf(4) / 3 * m * l * l]])
                rhs = mpmath.matrix([F + m * l * thd**2 * mpmath.sin(th), m * g * l * mpmath.sin(th)])
                xa, ta = mpmath.lu_solve(A, rhs)
                return [xd, xa, thd, ta]
            y = [mpmath.mpf(float(v)) for v in y0]
            h = mpmath.mpf(float(F32(tau))) / steps
            for _ in range(steps):
                k1 = f(y)
                k2 = f([a + h / 2 * b for a, b in zip(y, k1)])
                k3 = f([a + h / 2 * b for a, b in zip(y, k2)])
                k4 = f([a + h * b for a, b in zip(y, k3)])
                y = [a + h / 6 * (b1 + 2 * b2 + 2 * b3 + b4) for a, b1, b2, b3, b4 in zip(y, k1, k2, k3, k4)]
            return np.array([float(v) for v in y])

    # a long step (tau = 0.2) so that the discretisation error dominates rounding
    c = workloads.cartpole(tau=0.2, no_termination=1, max_episode_steps=0)
    exact = rk4_flow(state0, float(F32(c["force_mag"])), c["tau"])
    errs = []
    for C in (4, 8, 16, 32):
        params = oracle.make_params(**dict(c, compute_factor=C))
        got = oracle.env_step(params, state0, 1).astype(np.float64)
        errs.append(np.abs(got - exact).max())
    errs = np.array(errs)
    ratios = errs[:-1] / errs[1:]
    assert np.all((ratios > 1.7) & (ratios < 2.3)), (errs, ratios)
