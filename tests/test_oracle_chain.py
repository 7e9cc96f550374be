"""Pins of the oracle's full-range sin/cos and of its second simulator, the cart
carrying a chain of N uniform rods (CPU only).

Nothing here retypes the oracle's formulas.  They are checked against:

* textbook sin/cos (math.sin / math.cos) at angles far outside the series'
  domain, and the exact identity of the reduction on the series' domain;
* the cart-pole Euler-Lagrange mass-matrix solve at large angles;
* for the chain, the equations of motion assembled independently from the
  geometry of the links: rod-centre Jacobians give the mass matrix
  M = sum_i (m_i J_i^T J_i + I_i e_i e_i^T), Christoffel symbols of M
  (differentiated numerically in 50 digits) give the velocity terms, and the
  gradient of the potential gives the gravity terms, solved by a 50-digit
  linear solve (the oracle uses closed-form coupling constants instead);
* conservation of energy and horizontal momentum of the unforced chain, whose
  explicit-Euler drift must be first order in the time step;
* the small-angle linearisation (a constant-coefficient linear system);
* the one-link chain against the (separately pinned) cart-pole step;
* exact mirror symmetry, the reset draw's counters, and the episode loop's
  invariants.
"""
import math

import mpmath
import numpy as np
import pytest

import oracle
import workloads

F32 = np.float32
P = oracle.make_params(**workloads.CARTPOLE)


def _ulp(x):
    return float(np.spacing(F32(max(abs(float(F32(x))), 1e-30))))


# ---------------------------------------------------------------------------
# full-range sin / cos
# ---------------------------------------------------------------------------
def test_sincos_is_the_series_on_its_domain():
    """|theta| <= fp32(pi/4): no reduction, the series' bits exactly."""
    q = float(F32(math.pi / 4))
    xs = np.concatenate([np.linspace(-q, q, 4001, dtype=np.float32),
                         np.array([q, -q, 0.0, -0.0, 1e-30, -1e-38], dtype=np.float32)])
    for th in xs:
        s, c = oracle.sincos(th)
        assert s.view(np.uint32) == oracle.sin_series(th).view(np.uint32), th
        assert c.view(np.uint32) == oracle.cos_series(th).view(np.uint32), th
    # the series maps -0 to +0 (th + th^3 q with q < 0 rounds (-0)(q) to +0): a
    # defined property of the operation order, kept by the reduction
    assert oracle.sincos(-0.0)[0].view(np.uint32) == 0


def test_sincos_matches_textbook_at_large_angles():
    """Error bound: series truncation <= 2.5e-8 on |r| <= pi/4 (the degree-10
    cosine remainder), a few fp32 roundings of values <= 1 (<= 1.2e-7), the
    reduction's rounding of r (<= 3e-8) and |k| |pi/2 - hi - lo| (< 2e-11 for
    |theta| <= 2e4): 2.5e-7 in all."""
    rng = np.random.Generator(np.random.PCG64(3))
    xs = np.concatenate([rng.uniform(-20, 20, 20000), rng.uniform(-2e4, 2e4, 5000),
                         [k * math.pi / 2 + d for k in range(-40, 41) for d in (-1e-6, 0.0, 1e-6)],
                         [k * math.pi / 4 for k in range(-81, 82, 2)]]).astype(np.float32)
    worst = 0.0
    for th in xs:
        s, c = oracle.sincos(th)
        ts, tc = math.sin(float(th)), math.cos(float(th))
        err = max(abs(float(s) - ts), abs(float(c) - tc))
        worst = max(worst, err)
        assert err <= 2.5e-7, (th, s, ts, c, tc)
    assert worst > 1e-9        # the comparison is not vacuous


def test_sincos_quadrants_odd_even_and_special_values():
    rng = np.random.Generator(np.random.PCG64(4))
    for th in rng.uniform(-50, 50, 2000).astype(np.float32):
        s, c = oracle.sincos(th)
        sm, cm = oracle.sincos(-th)
        assert sm.view(np.uint32) == (-s).view(np.uint32) and cm.view(np.uint32) == c.view(np.uint32), th
    for v in (float("inf"), float("-inf"), float("nan")):
        s, c = oracle.sincos(v)
        assert math.isnan(s) and math.isnan(c)
    # continuity across the series' edge and across a quadrant boundary
    q = F32(math.pi / 4)
    above = np.nextafter(q, F32(1))
    assert abs(float(oracle.sincos(above)[0]) - float(oracle.sincos(q)[0])) < 3e-7
    assert abs(float(oracle.sincos(F32(3 * math.pi / 4))[0]) - math.sin(float(F32(3 * math.pi / 4)))) < 2.5e-7


def _exact(v):
    return mpmath.mpf(float(F32(v)))


def test_cartpole_step_any_angle_matches_euler_lagrange():
    """The cart-pole step with the pole anywhere on the circle (termination
    disabled) against the 50-digit mass-matrix solve with exact sin/cos."""
    c = workloads.cartpole(no_termination=1)
    params = oracle.make_params(**c)
    rng = np.random.Generator(np.random.PCG64(12))
    g, mc, m, l, tau, fm = (_exact(c[k]) for k in ("gravity", "masscart", "masspole", "half_length", "tau",
                                                   "force_mag"))
    for i in range(300):
        st = np.array([rng.uniform(-3, 3), rng.uniform(-5, 5), rng.uniform(-12, 12), rng.uniform(-8, 8)],
                      dtype=np.float32)
        a = int(rng.integers(0, 2))
        got = oracle.env_step(params, st, a)
        with mpmath.workdps(50):
            x, xd, th, thd = (mpmath.mpf(float(v)) for v in st)
            F = fm if a else -fm
            A = mpmath.matrix([[mc + m, m * l * mpmath.cos(th)], [m * l * mpmath.cos(th), mpmath.mpf(4) / 3 * m * l * l]])
            rhs = mpmath.matrix([F + m * l * thd**2 * mpmath.sin(th), m * g * l * mpmath.sin(th)])
            xacc, thacc = mpmath.lu_solve(A, rhs)
            want = [x + tau * xd, xd + tau * xacc, th + tau * thd, thd + tau * thacc]
        for q in range(4):
            acc = float(xacc if q == 1 else thacc)
            # sin/cos are now within 2.5e-7 absolute (not 1 ulp): the
            # acceleration's error scales with its inputs' size
            bound = 0.5 * _ulp(got[q]) + (0 if q in (0, 2) else float(tau) * (3e-6 * (abs(acc) + 60.0)))
            assert abs(float(got[q]) - float(want[q])) <= bound + 1e-30, (i, q, st, a, got[q], float(want[q]))


# ---------------------------------------------------------------------------
# the chain: an independent assembly of its equations of motion
# ---------------------------------------------------------------------------
def _chain_eom(c, N, state, force):
    """(qdd, M, f) in 50 digits from the links' geometry.  Rod i (0-based) has
    its centre at (x + sum_{j<i} L sin phi_j + l sin phi_i,
    sum_{j<i} L cos phi_j + l cos phi_i) and inertia m L^2 / 12 about it."""
    with mpmath.workdps(50):
        mc, m, l, g = (_exact(c[k]) for k in ("masscart", "masspole", "half_length", "gravity"))
        L = 2 * l
        I = m * L * L / 12
        n = N + 1
        q = [mpmath.mpf(float(state[0]))] + [mpmath.mpf(float(state[2 * j])) for j in range(1, N + 1)]
        qd = [mpmath.mpf(float(state[1]))] + [mpmath.mpf(float(state[2 * j + 1])) for j in range(1, N + 1)]

        def jac(qq, i):
            """2 x n Jacobian of rod i's centre."""
            Jx = [mpmath.mpf(1)] + [mpmath.mpf(0)] * N
            Jy = [mpmath.mpf(0)] * n
            for j in range(i + 1):
                arm = L if j < i else l
                Jx[1 + j] = arm * mpmath.cos(qq[1 + j])
                Jy[1 + j] = -arm * mpmath.sin(qq[1 + j])
            return Jx, Jy

        def mass(qq):
            Mm = mpmath.zeros(n, n)
            Mm[0, 0] += mc
            for i in range(N):
                Jx, Jy = jac(qq, i)
                for a in range(n):
                    for b in range(n):
                        Mm[a, b] += m * (Jx[a] * Jx[b] + Jy[a] * Jy[b])
                Mm[1 + i, 1 + i] += I
            return Mm

        def potential(qq):
            V = mpmath.mpf(0)
            for i in range(N):
                y = sum(L * mpmath.cos(qq[1 + j]) for j in range(i)) + l * mpmath.cos(qq[1 + i])
                V += m * g * y
            return V

        M = mass(q)
        # dM/dq_k by central differences in 50 digits
        h = mpmath.mpf(10) ** -20
        dM = []
        for k in range(n):
            qp, qm = list(q), list(q)
            qp[k] += h
            qm[k] -= h
            dM.append((mass(qp) - mass(qm)) / (2 * h))
        rhs = mpmath.zeros(n, 1)
        for i in range(n):
            cor = mpmath.mpf(0)
            for j in range(n):
                for k in range(n):
                    gam = (dM[k][i, j] + dM[j][i, k] - dM[i][j, k]) / 2
                    cor += gam * qd[j] * qd[k]
            qp, qm = list(q), list(q)
            qp[i] += h
            qm[i] -= h
            dV = (potential(qp) - potential(qm)) / (2 * h)
            rhs[i] = (force if i == 0 else 0) - cor - dV
        qdd = mpmath.lu_solve(M, rhs)
        return [qdd[i] for i in range(n)], M, rhs


def _random_chain_state(rng, N, angle=math.pi, vel=4.0):
    st = np.empty(2 * (N + 1), dtype=np.float32)
    st[0] = rng.uniform(-2, 2)
    st[1] = rng.uniform(-3, 3)
    for j in range(1, N + 1):
        st[2 * j] = rng.uniform(-angle, angle)
        st[2 * j + 1] = rng.uniform(-vel, vel)
    return st


@pytest.mark.parametrize("N", [1, 2, 3, 4])
@pytest.mark.parametrize("consts", ["default", "other"])
def test_chain_accelerations_match_independent_equations(N, consts):
    """Default constants, and constants with no unit length or simple ratio
    (L = 1 at the default half-length would hide a factor L)."""
    over = {} if consts == "default" else dict(masscart=0.8, masspole=0.23, half_length=0.35, gravity=9.81)
    c = workloads.cartpole(no_termination=1, **over)
    params = oracle.make_params(**c)
    rng = np.random.Generator(np.random.PCG64(100 + N + (0 if consts == "default" else 50)))
    worst = 0.0
    for i in range(40 if N < 4 else 25):
        st = _random_chain_state(rng, N, angle=(0.2 if i < 5 else 4.0))
        force = float(rng.choice([-10.0, 10.0]))
        got = oracle.chain_accel(params, N, st, force).astype(np.float64)
        want, M, f = _chain_eom(c, N, st, force)
        want = np.array([float(v) for v in want])
        # fp32 assembly and elimination: relative 2^-24 per operation, about
        # 10 N operations deep, amplified by the conditioning of M (the
        # oracle's sin/cos add 2.5e-7 absolute to each trig value)
        Minv = mpmath.inverse(M)
        cond = float(mpmath.mnorm(M, 1) * mpmath.mnorm(Minv, 1))
        scale = float(mpmath.mnorm(Minv, 1)) * (float(mpmath.mnorm(f, 1)) + 30.0) + np.abs(want).max()
        bound = (40 * N * 2.0**-24 + 2.5e-7) * cond * scale
        err = np.abs(got - want).max()
        worst = max(worst, err / bound)
        assert err <= bound, (N, i, st, force, got, want, bound)
    assert worst > 0


def test_one_link_chain_is_the_cartpole():
    """N = 1 is the cart-pole; the two fp32 operation orders differ, so the
    states agree to within a few ulps (rounding), never more."""
    c = workloads.cartpole(no_termination=1)
    params = oracle.make_params(**c)
    rng = np.random.Generator(np.random.PCG64(7))
    for _ in range(2000):
        st = _random_chain_state(rng, 1, angle=3.0)
        a = int(rng.integers(0, 2))
        ch = oracle.chain_step(params, 1, st, a)
        cp = oracle.env_step(params, st, a)
        for q in range(4):
            tol = 8 * _ulp(cp[q]) + (2e-6 if q in (1, 3) else 0.0)
            assert abs(float(ch[q]) - float(cp[q])) <= tol, (st, a, q, ch, cp)


def _chain_energy_momentum(c, N, st):
    """Energy and horizontal momentum in double from the links' geometry."""
    mc, m, l, g = (float(F32(c[k])) for k in ("masscart", "masspole", "half_length", "gravity"))
    L = 2 * l
    I = m * L * L / 12
    x, xd = float(st[0]), float(st[1])
    phi = [float(st[2 * j]) for j in range(1, N + 1)]
    phid = [float(st[2 * j + 1]) for j in range(1, N + 1)]
    T = 0.5 * mc * xd * xd
    V = 0.0
    px = mc * xd
    for i in range(N):
        vx = xd + sum(L * math.cos(phi[j]) * phid[j] for j in range(i)) + l * math.cos(phi[i]) * phid[i]
        vy = -sum(L * math.sin(phi[j]) * phid[j] for j in range(i)) - l * math.sin(phi[i]) * phid[i]
        y = sum(L * math.cos(phi[j]) for j in range(i)) + l * math.cos(phi[i])
        T += 0.5 * m * (vx * vx + vy * vy) + 0.5 * I * phid[i] ** 2
        V += m * g * y
        px += m * vx
    return T + V, px


@pytest.mark.parametrize("N", [2, 3])
@pytest.mark.parametrize("quantity", [0, 1])
def test_unforced_chain_conserves_energy_and_momentum_to_first_order(N, quantity):
    """With F = 0 the continuous chain conserves energy and horizontal momentum;
    explicit Euler drifts by O(tau) over a fixed time, so halving tau halves the
    drift.  A wrong coupling or sign leaves an O(1) drift."""
    horizon = 0.2
    drifts = []
    st0 = np.zeros(2 * (N + 1), dtype=np.float32)
    st0[1] = 0.4
    for j in range(1, N + 1):
        st0[2 * j] = 0.3 * (-1) ** j
        st0[2 * j + 1] = 0.8 * j
    for tau in (0.002, 0.001, 0.0005):
        c = workloads.cartpole(force_mag=0.0, tau=tau, no_termination=1, max_episode_steps=0)
        params = oracle.make_params(**c)
        s = st0.copy()
        q0 = _chain_energy_momentum(c, N, s)[quantity]
        for _ in range(int(round(horizon / tau))):
            s = oracle.chain_step(params, N, s, 1)
        drifts.append(_chain_energy_momentum(c, N, s)[quantity] - q0)
    d = np.array(drifts)
    assert abs(d[0]) > 1e-5
    r1, r2 = d[0] / d[1], d[1] / d[2]
    assert 1.7 < r1 < 2.3 and 1.7 < r2 < 2.3, d


@pytest.mark.parametrize("N", [1, 2, 4])
def test_chain_small_angle_linearisation(N):
    """Near the upright state the accelerations are M0^-1 (F e_0 + g H phi),
    with M0 the mass matrix at phi = 0 and H the gravity moments: an affine
    function of phi whose error is O(phi^2) (phid^2 terms included)."""
    c = workloads.cartpole(no_termination=1)
    params = oracle.make_params(**c)
    zero = np.zeros(2 * (N + 1), dtype=np.float32)
    _, M0, _ = _chain_eom(c, N, zero, 0.0)
    M0 = np.array(M0.tolist(), dtype=np.float64)
    mc, m, l, g = (float(F32(c[k])) for k in ("masscart", "masspole", "half_length", "gravity"))
    # gravity moment of link j: g (m l + (N - j) m L), j = 1..N
    H = np.array([g * (m * l + (N - j) * m * 2 * l) for j in range(1, N + 1)])
    rng = np.random.Generator(np.random.PCG64(55 + N))
    for _ in range(50):
        st = _random_chain_state(rng, N, angle=1e-3, vel=1e-3)
        F = float(rng.choice([-10.0, 10.0, 0.0]))
        phi = np.array([float(st[2 * j]) for j in range(1, N + 1)])
        lin = np.linalg.solve(M0, np.concatenate([[F], H * phi]))
        got = oracle.chain_accel(params, N, st, F).astype(np.float64)
        # neglected: phi^2 (cos), phi phid^2, F phi^2 ~ 1e-5 relative of |F|
        tol = 5e-5 * (abs(F) + 1.0) * np.abs(np.linalg.inv(M0)).max() + 64 * 2.0**-24 * np.abs(lin).max()
        assert np.abs(got - lin).max() <= tol, (N, st, F, got, lin)


@pytest.mark.parametrize("N", [1, 2, 3, 4])
def test_chain_mirror_symmetry_exact(N):
    """Negating every state word and the force negates the step's result bit
    for bit: every operation is odd or even in the right arguments and fp32
    rounding is symmetric."""
    c = workloads.cartpole(no_termination=1)
    params = oracle.make_params(**c)
    rng = np.random.Generator(np.random.PCG64(9 + N))
    for _ in range(300):
        st = _random_chain_state(rng, N, angle=6.0)
        a = int(rng.integers(0, 2))
        out = oracle.chain_step(params, N, st, a)
        neg = oracle.chain_step(params, N, -st, 1 - a)
        assert np.array_equal((-out).view(np.uint32), neg.view(np.uint32)), (st, a)


@pytest.mark.parametrize("N", [1, 2, 3, 4])
def test_chain_reset_draw_counters(N):
    """Words 4j .. 4j+3 of an episode starting at t come from Philox of counter
    (env, t / 8, RESET, j) mapped to the reset box; N = 1 is the cart-pole's
    reset draw."""
    for env, t, seed in ((0, 0, 0), (12345, 77, 1), (2**31 + 5, 2**32 - 9, 2**40 + 7)):
        got = oracle.chain_reset_draw(P, N, seed, env, t)
        key = [seed & 0xFFFFFFFF, seed >> 32]
        S = 2 * (N + 1)
        want = []
        for j in range((S + 3) // 4):
            w = oracle.philox4x32_10([env, t >> 3, 0, j], key)
            want += [oracle.uniform(int(v), workloads.CARTPOLE["reset_low"], workloads.CARTPOLE["reset_high"])
                     for v in w]
        assert np.array_equal(got, np.array(want[:S], dtype=np.float32))
        if N == 1:
            assert np.array_equal(got, oracle.reset_draw(P, seed, env, t))


def test_chain_thresholds():
    N = 3
    thr = F32(workloads.CARTPOLE["theta_threshold_rad"])
    st = np.zeros(8, dtype=np.float32)
    for j in range(1, N + 1):
        s = st.copy()
        s[2 * j] = thr
        assert not oracle.chain_terminated(P, N, s)
        s[2 * j] = -np.nextafter(thr, F32(1))
        assert oracle.chain_terminated(P, N, s)
        s[2 * j + 1] = 100.0          # velocities never terminate
        s[2 * j] = 0.0
        assert not oracle.chain_terminated(P, N, s)
    s = st.copy()
    s[0] = np.nextafter(F32(2.4), F32(3))
    assert oracle.chain_terminated(P, N, s)
    s[0] = float("nan")
    assert not oracle.chain_terminated(P, N, s)
    noterm = oracle.make_params(**workloads.cartpole(no_termination=1))
    assert not oracle.chain_terminated(noterm, N, np.full(8, 50.0, dtype=np.float32))


# ---------------------------------------------------------------------------
# the chain's episode loop
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N", [1, 3])
def test_chain_rows_chain_and_done_semantics(N):
    sim = oracle.ChainSim(300, N, P, env0=77)
    sim.reset(11)
    T = 80
    tr = sim.step(T)
    S = 2 * (N + 1)
    obs, act, done = tr["obs"], tr["action"], tr["done"]
    assert np.all(tr["reward"] == 1.0)
    for i in range(0, 300, 7):
        env = 77 + i
        assert np.array_equal(obs[0, :, i], oracle.chain_reset_draw(P, N, 11, env, 0))
        for k in range(T):
            assert act[k, i] == oracle.action_bit(11, env, k)
            nxt = oracle.chain_step(P, N, obs[k, :, i], int(act[k, i]))
            term = oracle.chain_terminated(P, N, nxt)
            assert bool(done[k, i] & 1) == term
            if k + 1 < T:
                want = oracle.chain_reset_draw(P, N, 11, env, k + 1) if done[k, i] else nxt
                assert np.array_equal(obs[k + 1, :, i].view(np.uint32), want.view(np.uint32))
    assert obs.shape == (T, S, 300)
    assert int(done.astype(bool).sum()) > 300          # episodes ended and restarted


def test_chain_partition_and_slice_invariance_and_resume():
    N = 2
    a = oracle.ChainSim(200, N, P)
    a.reset(5)
    whole = a.step(64)
    b = oracle.ChainSim(200, N, P)
    b.reset(5)
    parts = [b.step(k) for k in (1, 7, 20, 36)]
    for key in ("obs", "action", "reward", "done"):
        assert np.array_equal(np.concatenate([p[key] for p in parts]), whole[key]), key
    sa, ea, ta = a.get_state()
    sb, eb, tb = b.get_state()
    assert np.array_equal(sa, sb) and np.array_equal(ea, eb) and ta == tb == 64
    # a slice of envs 50..149 is the same as columns 50..149
    c = oracle.ChainSim(100, N, P, env0=50)
    c.reset(5)
    sl = c.step(64)
    assert np.array_equal(sl["obs"], whole["obs"][:, :, 50:150])
    # resume from a saved state
    d = oracle.ChainSim(200, N, P)
    d.reset(5)
    d.step(10)
    st, ep, t = d.get_state()
    e = oracle.ChainSim(200, N, P)
    e.reset(99)
    e.set_state(st, ep, t)
    e.reset  # noqa: B018
    r1 = d.step(30)
    r2 = oracle.ChainSim(200, N, P)
    r2.reset(5)
    r2.step(10)
    assert np.array_equal(r2.step(30)["obs"], r1["obs"])


def test_chain_block_stats_brute_force_and_time_limit():
    N = 2
    params = oracle.make_params(**workloads.cartpole(max_episode_steps=12))
    sim = oracle.ChainSim(700, N, params, env0=200)
    sim.reset(3)
    sim.step(5)
    st_before, ep_before, _ = sim.get_state()
    tr = sim.step(40)
    done, stats = tr["done"], tr["stats"]
    assert stats.shape == (sim.n_blocks, 4)
    want = np.zeros(stats.shape, dtype=np.int64)
    ep = ep_before.astype(np.int64).copy()
    for k in range(40):
        for i in range(700):
            ep[i] += 1
            if done[k, i]:
                blk = (200 + i) // 256 - 200 // 256
                want[blk] += [1, ep[i], done[k, i] & 1, (done[k, i] >> 1) & 1]
                ep[i] = 0
    assert np.array_equal(stats, want)
    assert np.any(done == 2) and np.any(done & 1)
    _, ep_end, _ = sim.get_state()
    assert ep_end.max() < 12


@pytest.mark.parametrize("N", [1, 2, 3, 4])
def test_chain_episodes_sampled_last_at_least_eight_steps(N):
    """Random pushes from the reset box: no sampled episode ends before step 8,
    so two episodes of one env never begin in the same 8-step reset block."""
    sim = oracle.ChainSim(2000, N, P)
    sim.reset(N)
    d = sim.step(200)["done"].astype(bool)
    for i in range(2000):
        idx = np.flatnonzero(d[:, i])
        if len(idx):
            assert idx[0] + 1 >= 8
            assert len(idx) == 1 or np.diff(idx).min() >= 8


@pytest.mark.parametrize("N", [1, 2])
def test_chain_row_checker_accepts_oracle_rows_and_finds_planted_errors(N):
    sim = oracle.ChainSim(90, N, P, env0=500)
    sim.reset(8)
    tr = sim.step(50)
    st, ep, t = sim.get_state()
    keys = ("obs", "action", "reward", "done")
    assert oracle.chain_check_rows(P, N, 8, 500, 0, *[tr[k] for k in keys], final_state=st, final_ep=ep) == (0, None)
    for field, k, i in (("obs", 20, 33), ("obs", 0, 5), ("action", 3, 89), ("done", 30, 13), ("final", 49, 61),
                        ("final_ep", 49, 2)):
        bad = {key: tr[key].copy() for key in keys}
        fs, fe = st.copy(), ep.copy()
        if field == "obs":
            bad["obs"][k, 2, i] = np.nextafter(bad["obs"][k, 2, i], F32(1))
        elif field == "action":
            bad["action"][k, i] ^= 1
        elif field == "done":
            bad["done"][k, i] ^= 2
        elif field == "final":
            fs[3, i] = np.nextafter(fs[3, i], F32(1))
        else:
            fe[i] += 1
        count, first = oracle.chain_check_rows(P, N, 8, 500, 0, *[bad[key] for key in keys], final_state=fs,
                                               final_ep=fe)
        want_k = k - 1 if (field == "obs" and k > 0) else k
        assert count >= 1 and first == (want_k, i), (field, count, first)
