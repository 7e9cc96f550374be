"""Pins of the oracle's vectorised data-collection loop (CPU only).

Invariants and closed forms the loop must satisfy whatever its internals:

* every trajectory row continues the previous one: the next obs is the Euler
  step of (obs, action), or, after done, the reset draw of the next step;
* done bit 0 <=> the post-step state crossed a threshold; bit 1 <=> the
  episode reached the time limit; stored episode counters stay below it;
* results do not depend on how K steps are split into calls, or on which
  slice of environments is simulated (counter-based RNG keyed by global id);
* the padding words follow the closed form of their linear recurrence;
* block statistics equal a brute-force recount from the trajectory;
* random-action episode lengths have the cart-pole's known scale.
"""
import math
from fractions import Fraction

import mpmath
import numpy as np
import pytest

import oracle
import workloads

P = oracle.make_params(**workloads.CARTPOLE)


def _run(n, T, K, D=0, seed=0, env0=0, params=P, policy=None):
    sim = oracle.Sim(n, D, params, env0=env0)
    sim.reset(seed)
    parts = []
    done_steps = 0
    while done_steps < T:
        k = min(K, T - done_steps)
        parts.append(sim.step(k, policy=policy))
        done_steps += k
    traj = {key: np.concatenate([p[key] for p in parts], axis=0) for key in ("obs", "action", "reward", "done")}
    traj["stats"] = [p["stats"] for p in parts]
    return sim, traj


def test_reset_state_in_box_and_counters_zero():
    sim = oracle.Sim(1000, 3, P)
    sim.reset(5)
    st, ep, t = sim.get_state()
    assert t == 0 and np.all(ep == 0)
    assert np.all(st[:4] >= np.float32(-0.05)) and np.all(st[:4] <= np.float32(0.05))
    assert np.all(st[4:] == 0) and not np.any(np.signbit(st[4:]))
    a, b = sim.pad_params()
    assert np.all(a >= np.float32(0.9)) and np.all(a <= np.float32(0.99))
    assert np.all(b >= np.float32(-1)) and np.all(b <= np.float32(1))


def test_trajectory_rows_chain_and_done_semantics():
    n, T = 64, 300
    sim, tr = _run(n, T, K=T, seed=1)
    obs, act, rew, done = tr["obs"], tr["action"], tr["reward"], tr["done"]
    assert np.all(rew == 1.0)
    assert set(np.unique(act)) <= {0, 1}
    assert set(np.unique(done)) <= {0, 1, 2, 3}
    final, _, t = sim.get_state()
    assert t == T
    for e in range(n):
        for t in range(T):
            post = oracle.cartpole_step(P, obs[t, :, e], int(act[t, e]))
            term = oracle.terminated(P, post)
            assert (done[t, e] & 1) == int(term)
            nxt = obs[t + 1, :, e] if t + 1 < T else final[:4, e]
            if done[t, e]:
                assert np.array_equal(nxt, oracle.reset_draw(P, 1, e, t + 1))
            else:
                assert np.array_equal(nxt, post)
            assert act[t, e] == oracle.action_bit(1, e, t)


def test_time_limit_and_counters():
    params = oracle.make_params(**workloads.cartpole(max_episode_steps=5, x_threshold=1e9, theta_threshold_rad=1e9))
    sim, tr = _run(8, 23, K=23, params=params)
    done = tr["done"]
    # only truncations, every 5th step
    expect = np.zeros(23, dtype=np.uint8)
    expect[4::5] = 2
    assert np.array_equal(done, np.repeat(expect[:, None], 8, axis=1))
    _, ep, _ = sim.get_state()
    assert np.all(ep == 23 % 5)
    # default limit: no run of more than 500 steps without done, counters < 500
    params = oracle.make_params(**workloads.cartpole(no_termination=1))
    sim, tr = _run(2, 1200, K=600, params=params)
    d = tr["done"]
    assert np.array_equal(np.nonzero(d[:, 0])[0], np.array([499, 999]))
    assert np.all(d[[499, 999]] == 2)
    _, ep, _ = sim.get_state()
    assert np.all(ep < 500)


def test_terminated_and_truncated_together():
    # a threshold that is crossed exactly on the 3rd step of every episode
    params = oracle.make_params(**workloads.cartpole(max_episode_steps=3, x_threshold=1e9, theta_threshold_rad=1e9))
    _, tr = _run(4, 9, K=9, params=params)
    assert np.all(tr["done"][2::3] == 2)
    tight = oracle.make_params(**workloads.cartpole(max_episode_steps=1, theta_threshold_rad=0.0))
    _, tr = _run(4, 4, K=4, params=tight)
    # every step terminates (any nonzero angle) and is truncated (limit 1), unless theta' == 0 exactly
    assert np.all(tr["done"] == 3)


@pytest.mark.parametrize("D", [0, 5])
def test_partition_invariance(D):
    n, T = 37, 130
    base_sim, base = _run(n, T, K=T, D=D, seed=3)
    for K in (1, 7, 64):
        sim, tr = _run(n, T, K=K, D=D, seed=3)
        for key in ("obs", "action", "reward", "done"):
            assert np.array_equal(tr[key], base[key]), (K, key)
        s1, e1, t1 = sim.get_state()
        s0, e0, t0 = base_sim.get_state()
        assert np.array_equal(s1, s0) and np.array_equal(e1, e0) and t1 == t0


def test_slice_invariance():
    # env e behaves the same whether simulated alone or inside a larger batch
    n, T = 300, 80
    _, full = _run(n, T, K=40, D=2, seed=workloads.PARITY_SEEDS[2])
    for e in (0, 17, 255, 256, 299):
        _, one = _run(1, T, K=T, D=2, seed=workloads.PARITY_SEEDS[2], env0=e)
        for key in ("obs", "action", "done"):
            assert np.array_equal(one[key][..., 0], full[key][..., e]), (e, key)


def test_get_set_state_resume():
    n, T = 50, 120
    _, whole = _run(n, T, K=T, D=3, seed=9)
    sim = oracle.Sim(n, 3, P)
    sim.reset(9)
    first = sim.step(T // 2)
    st, ep, t = sim.get_state()
    sim2 = oracle.Sim(n, 3, P)
    sim2.reset(9)                      # same padding parameters
    sim2.set_state(st, ep, t)
    second = sim2.step(T - T // 2)
    for key in ("obs", "action", "done"):
        assert np.array_equal(np.concatenate([first[key], second[key]]), whole[key])


def test_step_before_reset_and_overflow():
    sim = oracle.Sim(4, 0, P)
    with pytest.raises(RuntimeError):
        sim.step(1)
    sim.reset(0)
    st, ep, _ = sim.get_state()
    sim.set_state(st, ep, 2**32 - 10)
    sim.step(9)
    with pytest.raises(RuntimeError):
        sim.step(2)


def test_block_stats_brute_force():
    n, T = 700, 150
    env0 = 200      # a slice straddling block boundaries
    sim = oracle.Sim(n, 0, P, env0=env0)
    sim.reset(2)
    pre = sim.step(37)                  # stats are per call
    _, ep_start, _ = sim.get_state()
    out = sim.step(T)
    done = out["done"]
    nblk = sim.n_blocks
    want = np.zeros((nblk, 4), dtype=np.int64)
    for i in range(n):
        blk = (env0 + i) // 256 - env0 // 256
        length = int(ep_start[i])
        for t in range(T):
            length += 1
            if done[t, i]:
                want[blk] += [1, length, done[t, i] & 1, (done[t, i] >> 1) & 1]
                length = 0
    assert np.array_equal(out["stats"].astype(np.int64), want)
    assert want[:, 0].sum() > 0 and pre["stats"].sum() > 0


def test_episode_length_scale():
    """Random pushes topple the pole in about 22 steps on average (at least 8)."""
    n, T = 2000, 400
    _, tr = _run(n, T, K=T, seed=0)
    d = tr["done"]
    lengths = []
    for e in range(n):
        idx = np.nonzero(d[:, e])[0]
        lengths.extend(np.diff(np.concatenate([[-1], idx])).tolist())
    lengths = np.array(lengths)
    assert 20.0 < lengths.mean() < 25.0
    assert lengths.min() >= 8
    assert np.all(d & 2 == 0)        # no episode reaches 500 steps here


def _forced_action_policy(action):
    """Zero weights and output biases that put all mass on one action."""
    z = lambda *s: np.zeros(s, dtype=np.float32)  # noqa: E731
    b3 = np.array([50.0, -50.0] if action == 0 else [-50.0, 50.0], dtype=np.float32)
    return oracle.Policy(z(64, 4), z(64), z(64, 64), z(64), z(2, 64), b3)


def test_padding_closed_form_constant_action():
    """With a_t = 1 throughout an episode, s_n = b (1 - a^n) / (1 - a); fp32
    rounding adds at most ~n ulp-sized errors, bounded by n eps |b| / (1 - a).
    Gravity and force are off so that the cart-pole stays finite without
    termination (a NaN observation would make the policy's p0 NaN)."""
    params = oracle.make_params(**workloads.cartpole(no_termination=1, max_episode_steps=0,
                                                     gravity=0.0, force_mag=0.0))
    D, n, T = 6, 8, 60
    sim = oracle.Sim(n, D, params)
    sim.reset(4)
    a, b = sim.pad_params()
    sim.step(T, policy=_forced_action_policy(1))
    st, _, _ = sim.get_state()
    for j in range(D):
        for e in range(n):
            aa, bb = Fraction(float(a[j, e])), Fraction(float(b[j, e]))
            exact = bb * (1 - aa**T) / (1 - aa)
            bound = T * 2.0**-24 * abs(float(bb)) / (1 - float(aa))
            assert abs(float(st[4 + j, e]) - float(exact)) <= bound
    # action 0 throughout: the words stay exactly +0
    sim.reset(4)
    sim.step(T, policy=_forced_action_policy(0))
    st, _, _ = sim.get_state()
    assert np.all(st[4:] == 0) and not np.any(np.signbit(st[4:]))


def test_padding_closed_form_random_actions():
    """Within an episode that starts at t0, s_t = sum_{i<t} a^(t-1-i) b u_i."""
    D, n, T = 3, 16, 90
    sim = oracle.Sim(n, D, P)
    sim.reset(6)
    a, b = sim.pad_params()
    tr = sim.step(T)
    st, _, _ = sim.get_state()
    act, done = tr["action"], tr["done"]
    with mpmath.workdps(40):
        for e in range(n):
            last_done = np.nonzero(done[:, e])[0]
            t0 = int(last_done[-1]) + 1 if len(last_done) else 0
            for j in range(D):
                aa, bb = mpmath.mpf(float(a[j, e])), mpmath.mpf(float(b[j, e]))
                exact = mpmath.fsum(aa ** (T - 1 - i) * bb * int(act[i, e]) for i in range(t0, T))
                bound = (T - t0) * 2.0**-24 * abs(float(bb)) / (1 - float(aa)) + 1e-30
                assert abs(float(st[4 + j, e]) - float(exact)) <= bound, (e, j)
                if t0 == T:
                    assert st[4 + j, e] == 0


def test_episodes_last_at_least_eight_steps():
    """With the default constants no episode ends within 7 steps: from every
    point of a grid over the initial-state box (corners included) and under all
    2^7 action sequences the post-step state stays inside the thresholds for 7
    steps.  So two episodes of one environment never begin in the same 8-step
    block and never share a reset draw."""
    import itertools
    grid = np.linspace(-0.05, 0.05, 3, dtype=np.float32)
    for st in itertools.product(grid, repeat=4):
        for acts in itertools.product((0, 1), repeat=7):
            s = np.array(st, dtype=np.float32)
            for a in acts:
                s = oracle.cartpole_step(P, s, a)
                assert not oracle.terminated(P, s), (st, acts)
    # and 8 steps can suffice: the fastest fall from a corner ends at step 8
    s = np.array([0.0, 0.05, 0.05, 0.05], dtype=np.float32)
    for _ in range(7):
        s = oracle.cartpole_step(P, s, 0)
    assert oracle.terminated(P, oracle.cartpole_step(P, s, 0))


@pytest.mark.parametrize("over", [{}, {"max_episode_steps": 7}, {"x_threshold": 0.3}, {"compute_factor": 3}])
def test_row_checker_accepts_oracle_rows_and_finds_planted_errors(over):
    """orc_check_rows (the teacher-forced check GPU tests run at full size) passes
    the oracle's own trajectory and flags a corrupted obs (row 0, which must be
    the reset draw, included), action, reward or done at the row and env where it
    was planted, and a final state or episode counter that is not the last
    row's successor."""
    params = oracle.make_params(**workloads.cartpole(**over))
    n, T, env0, seed = 97, 60, 1000, 5
    sim = oracle.Sim(n, 0, params, env0=env0)
    sim.reset(seed)
    tr = sim.step(T)
    fin, fin_ep, _ = sim.get_state()
    assert oracle.check_rows(params, seed, env0, 0, tr["obs"], tr["action"], tr["reward"], tr["done"],
                             final_state=fin, final_ep=fin_ep) == (0, None)
    for field, k, i in (("obs", 17, 40), ("obs", 0, 9), ("action", 3, 96), ("reward", 59, 0), ("done", 30, 13),
                        ("final", T - 1, 50), ("final_ep", T - 1, 3)):
        bad = {key: tr[key].copy() for key in ("obs", "action", "reward", "done")}
        fs, fe = fin.copy(), fin_ep.copy()
        if field == "obs":
            bad["obs"][k, 2, i] = np.nextafter(bad["obs"][k, 2, i], np.float32(1))
        elif field == "action":
            bad["action"][k, i] ^= 1
        elif field == "reward":
            bad["reward"][k, i] = 0.5
        elif field == "done":
            bad["done"][k, i] ^= 2
        elif field == "final":
            fs[0, i] = np.nextafter(fs[0, i], np.float32(-1))
        else:
            fe[i] += 1
        count, first = oracle.check_rows(params, seed, env0, 0, bad["obs"], bad["action"], bad["reward"], bad["done"],
                                         final_state=fs, final_ep=fe)
        # an obs error shows at the step that produced it (row k - 1 predicts
        # row k); row 0 is compared with the reset draw
        want_k = k - 1 if (field == "obs" and k > 0) else k
        assert count >= 1 and first == (want_k, i), (field, count, first)
    # a later start: rows from step t0 with the episode counters at t0
    st, ep, t = sim.get_state()
    tr2 = sim.step(25)
    assert oracle.check_rows(params, seed, env0, t, tr2["obs"], tr2["action"], tr2["reward"], tr2["done"],
                             ep0=ep) == (0, None)


@pytest.mark.parametrize("bf16", [False, True])
def test_policy_row_checker_accepts_oracle_rows_and_finds_planted_errors(bf16):
    """orc_check_policy_rows passes the oracle's own policy trajectory (p0, log pi
    and value rounded to fp32, as a device records them), accepts a recorded
    value at the edge of its enclosure and rejects one just past it, flags a
    planted error in the trajectory at its row and env, and admits an action
    that differs from the oracle's only when u lies inside the p0 enclosure."""
    import policy_bounds
    params = oracle.make_params(**workloads.cartpole(max_episode_steps=9))
    w = workloads.mlp_weights(7)
    rng = np.random.Generator(np.random.PCG64(8))
    for k in ("b1", "b2", "b3", "bv"):
        w[k] = (rng.standard_normal(w[k].shape) * 0.3).astype(np.float32)
    pol = oracle.Policy(**w, bf16=bf16)
    n, T, env0, seed = 61, 40, 300, 9
    sim = oracle.Sim(n, 0, params, env0=env0)
    sim.reset(seed)
    tr = sim.step(T, policy=pol)
    f = {k: tr[k].astype(np.float32) for k in ("p0", "logp", "value")}
    rows = dict(obs=tr["obs"], action=tr["action"], reward=tr["reward"], done=tr["done"])

    def check(errs=None, **repl):
        r = dict(rows, p0=f["p0"], logp=f["logp"], value=f["value"])
        r.update(repl)
        return oracle.check_policy_rows(params, pol, seed, env0, 0, r["obs"], r["action"], r["reward"], r["done"],
                                        r["p0"], errs or policy_bounds.errs(), logp=r["logp"], value=r["value"])

    bad, first, st = check()
    assert (bad, first, st["exempt"]) == (0, None, 0) and st["worst"] <= 6e-8
    assert 0.0 < st["mean_width"] <= st["max_width"] < 0.01
    assert int(tr["done"].max()) >= 1                    # episode ends are crossed
    # the enclosure's edge passes, the next float past it fails
    u_all = np.array([[oracle.policy_u(seed, env0 + i, k) for i in range(n)] for k in range(T)])
    gap = np.abs(u_all - tr["p0"])
    k, i = np.unravel_index(int(np.argmax(gap)), gap.shape)      # a row where u is far from p0
    obs_ki = tr["obs"][k, :, i]
    b = pol.bounds(obs_ki, policy_bounds.errs())
    a = int(tr["action"][k, i])
    for field, (lo, hi) in (("p0", b["p0"]), ("logp", b["logp1" if a else "logp0"]), ("value", b["value"])):
        for edge, outward in ((lo, -1.0), (hi, 1.0)):
            inside = np.float32(edge)
            if (float(inside) - edge) * outward > 0:                  # fp32 rounding moved it outside
                inside = np.nextafter(inside, np.float32(-outward * 10))
            arr = f[field].copy()
            arr[k, i] = inside
            assert check(**{field: arr})[0] == 0, (field, edge)
            arr[k, i] = np.nextafter(inside, np.float32(outward * 10))
            while (float(arr[k, i]) - edge) * outward <= 0:
                arr[k, i] = np.nextafter(arr[k, i], np.float32(outward * 10))
            bad, first, _ = check(**{field: arr})
            assert bad == 1 and first == (k, i), (field, edge, bad, first)
    for field, kk, ii in (("action", 11, 30), ("obs", 25, 7), ("obs", 0, 60), ("reward", 2, 2), ("done", 30, 44)):
        arr = rows[field].copy()
        if field == "action":
            arr[kk, ii] ^= 1
        elif field == "obs":
            arr[kk, 1, ii] = np.nextafter(arr[kk, 1, ii], np.float32(-1))
        elif field == "reward":
            arr[kk, ii] = 0.0
        else:
            arr[kk, ii] ^= 1
        bad, first, _ = check(**{field: arr})
        want_k = kk - 1 if (field == "obs" and kk > 0) else kk
        assert bad >= 1 and first == (want_k, ii), (field, bad, first)
    # the state after the last row, and the per-step |p0 - oracle p0| output
    fin, fin_ep, _ = sim.get_state()
    r = oracle.check_policy_rows(params, pol, seed, env0, 0, rows["obs"], rows["action"], rows["reward"],
                                 rows["done"], f["p0"], policy_bounds.errs(), logp=f["logp"], value=f["value"],
                                 final_state=fin, final_ep=fin_ep)
    assert r[0] == 0
    fs = fin.copy()
    fs[2, 17] = np.nextafter(fs[2, 17], np.float32(1))
    r = oracle.check_policy_rows(params, pol, seed, env0, 0, rows["obs"], rows["action"], rows["reward"],
                                 rows["done"], f["p0"], policy_bounds.errs(), final_state=fs, final_ep=fin_ep)
    assert r[:2] == (1, (T - 1, 17))
    dp0 = np.zeros((T, n), dtype=np.float32)
    oracle.check_policy_rows(params, pol, seed, env0, 0, rows["obs"], rows["action"], rows["reward"], rows["done"],
                             f["p0"], policy_bounds.errs(), dp0_out=dp0)
    assert np.array_equal(dp0, np.abs(f["p0"].astype(np.float64) - tr["p0"]).astype(np.float32))
    # an action flip on the last row (nothing after it to diverge): record p0
    # just across u with the flipped action, its done byte and its log pi
    k = T - 1
    i = int(np.argmin(gap[k]))
    u = float(u_all[k, i])
    a = 1 - int(tr["action"][k, i])
    p0g, act, done, logp = f["p0"].copy(), tr["action"].copy(), tr["done"].copy(), f["logp"].copy()
    p0g[k, i] = np.nextafter(np.float32(u), np.float32(2)) if a == 0 else np.float32(u)
    act[k, i] = a
    logit, _, _ = pol.eval(tr["obs"][k, :, i])
    post = oracle.env_step(params, tr["obs"][k, :, i], a)
    done[k, i] = int(oracle.terminated(params, post)) | (tr["done"][k, i] & 2)    # the time limit: action-free
    logp[k, i] = np.float32(oracle.log_prob(logit, a))
    flip = dict(action=act, done=done, p0=p0g, logp=logp)
    wide = policy_bounds.errs(scale=4.0 * (gap[k, i] + 1e-6) / policy_bounds.E_P0)    # enclosure holds u
    bad, first, st = check(errs=wide, **flip)
    assert (bad, st["exempt"]) == (0, 1), (bad, first, st, gap[k, i])
    bad, first, st = check(**flip)                        # the true enclosure does not
    assert (bad, first) == (1, (k, i)), (bad, first, gap[k, i])
    # the recorded action must follow the recorded p0 exactly, whatever the enclosure
    bad, first, _ = check(errs=wide, p0=p0g)
    assert (bad, first) == (1, (k, i))
