"""GPU parity of the fused MLP-policy kernels (fp32 and bf16) against the oracle.

The policy's arithmetic need not match the oracle's bit for bit, so the rules
are:
* the GPU's own consistency is exact: action = (u < p0_gpu ? 0 : 1), with u the
  POLICY-stream uniform of (seed, env, step) and p0_gpu the recorded policy_p0;
* teacher-forced, at every recorded step, p0_gpu, and the recorded log pi of
  the GPU's action and value, lie in the oracle's enclosures for the recorded
  obs (orc_mlp_bounds under the error model of tests/policy_bounds.py: fp32
  accumulation, and the kernel's tanh, p0 and log pi errors measured over all
  fp32 inputs; in bf16 mode it follows every hidden-unit rounding those errors
  could flip).  An action can then differ from the oracle's own choice only
  where u lies inside the p0 enclosure;
* fp32 also keeps a fixed gate |p0_gpu - p0_oracle| <= 1e-5 (the enclosures are
  worst-case sums, ~1e-4 wide; observed differences are ~1e-7), so a defect
  smaller than the enclosure would still show;
* the next observation, the done byte and the reward follow from
  (obs_t, action_t) bit for bit (Euler step or the reset draw);
* free-running: an environment's trajectory equals the oracle's up to its first
  action disagreement, which must be one whose u lies in the p0 enclosure.
"""
import os

import numpy as np
import pytest

import oracle
import policy_bounds
import workloads
from gpu_helpers import F32_P0_GATE, device_policy, policy_weights

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401


def _gpu_policy_run(n, T, K, w, dtype, seed, cfg=None, slices=None, learner=None):
    import paper_2207_07736_amd as p
    if learner is None:
        learner = "wv" in w
    st, keep = device_policy(w, dtype)
    sim = p.Simulator(n, 0, cfg or workloads.CARTPOLE)
    try:
        sim.reset(seed)
        tr = p.Trajectory(T, n, p0=True, learner=learner)
        stats = []
        for k0 in range(0, T, K):
            sim.step(min(K, T - k0), tr.rows(k0, min(K, T - k0)), policy=st)
            stats.append(tr.block_stats.clone())
        torch.cuda.synchronize()

        def cols(x):
            if slices is None:
                return x.cpu().numpy()
            return np.concatenate([x[..., a:b].cpu().numpy() for a, b in slices], axis=-1)

        out = dict(obs=cols(tr.obs), action=cols(tr.action), reward=cols(tr.reward), done=cols(tr.done),
                   p0=cols(tr.policy_p0), stats=[s.cpu().numpy().view(np.uint32) for s in stats])
        if learner:
            out["logp"], out["value"] = cols(tr.logp), cols(tr.value)
        state, ep, t = sim.get_state()
        out["t"] = t
        del tr, keep
        return out
    finally:
        sim.close()


def _check_teacher_forced(g, w, dtype, seed, env_ids, cfg=None):
    """Every recorded step of every listed env, against the oracle's enclosures."""
    params = oracle.make_params(**(cfg or workloads.CARTPOLE))
    pol = oracle.Policy(**w, bf16=(dtype == "bf16"))
    errs = policy_bounds.errs()
    T = g["action"].shape[0]
    worst, exempt = 0.0, 0
    for col, env in enumerate(env_ids):
        for t in range(T):
            obs = g["obs"][t, :, col]
            u = float(oracle.policy_u(seed, env, t))
            p_gpu = float(g["p0"][t, col])
            a = int(g["action"][t, col])
            assert a == (0 if u < p_gpu else 1), (env, t, u, p_gpu, a)
            logit, p_ref, v_ref = pol.eval(obs)
            b = pol.bounds(obs, errs)
            worst = max(worst, abs(p_gpu - p_ref))
            assert b["p0"][0] <= p_gpu <= b["p0"][1], (env, t, p_gpu, p_ref, b["p0"])
            if dtype == "f32":
                assert abs(p_gpu - p_ref) <= F32_P0_GATE, (env, t, p_gpu, p_ref)
            if "logp" in g:
                lo, hi = b["logp1" if a else "logp0"]
                assert lo <= float(g["logp"][t, col]) <= hi, (env, t, g["logp"][t, col], lo, hi)
                lo, hi = b["value"]
                assert lo <= float(g["value"][t, col]) <= hi, (env, t, g["value"][t, col], lo, hi)
            if a != (0 if u < p_ref else 1):
                assert b["p0"][0] <= u <= b["p0"][1], (env, t, u, p_ref)     # implied by the two checks above
                exempt += 1
            post = oracle.cartpole_step(params, obs, a)
            term = oracle.terminated(params, post)
            assert (g["done"][t, col] & 1) == int(term)
            assert g["reward"][t, col] == 1.0
            if t + 1 < T:
                nxt = g["obs"][t + 1, :, col]
                want = oracle.reset_draw(params, seed, env, t + 1) if g["done"][t, col] else post
                assert np.array_equal(nxt.view(np.uint32), want.view(np.uint32)), (env, t)
    return worst, exempt


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("bias_scale", [0.0, 0.3])
def test_policy_teacher_forced(dtype, bias_scale):
    n, T, K, seed = 300, 64, 16, 5
    w = policy_weights(11, bias_scale)
    g = _gpu_policy_run(n, T, K, w, dtype, seed)
    worst, exempt = _check_teacher_forced(g, w, dtype, seed, list(range(n)))
    assert worst > 0.0 or dtype == "f32"
    # the compiled checker the full-size tests use reaches the same verdict
    bad, first, st = oracle.check_policy_rows(
        oracle.make_params(**workloads.CARTPOLE), oracle.Policy(**w, bf16=(dtype == "bf16")), seed, 0, 0, g["obs"],
        g["action"], g["reward"], g["done"], g["p0"], policy_bounds.errs(), logp=g["logp"], value=g["value"])
    assert (bad, first, st["exempt"]) == (0, None, exempt) and abs(st["worst"] - worst) <= 1e-12 * max(1.0, worst)
    # the p0 values are not degenerate
    assert 0.05 < float(g["p0"].std()) and np.all((g["p0"] > 0) & (g["p0"] < 1))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_free_running_until_exempt_divergence(dtype):
    n, T, K, seed = 256, 48, 16, 2
    w = policy_weights(3)
    g = _gpu_policy_run(n, T, K, w, dtype, seed)
    sim = oracle.Sim(n, 0, oracle.make_params(**workloads.CARTPOLE))
    sim.reset(seed)
    pol = oracle.Policy(**w, bf16=(dtype == "bf16"))
    r = {k: [] for k in ("obs", "action", "done")}
    for _ in range(T // K):
        o = sim.step(K, policy=pol)
        for k in r:
            r[k].append(o[k])
    r = {k: np.concatenate(v) for k, v in r.items()}
    errs = policy_bounds.errs()
    diverged = 0
    for e in range(n):
        mism = np.nonzero(g["action"][:, e] != r["action"][:, e])[0]
        upto = int(mism[0]) if len(mism) else T
        assert np.array_equal(g["obs"][:upto + 1 if upto < T else T, :, e].view(np.uint32),
                              r["obs"][:upto + 1 if upto < T else T, :, e].view(np.uint32)), e
        assert np.array_equal(g["done"][:upto, e], r["done"][:upto, e])
        if upto < T:
            u = float(oracle.policy_u(seed, e, upto))
            lo, hi = pol.bounds(r["obs"][upto, :, e], errs)["p0"]
            assert lo <= u <= hi, (e, upto, u, lo, hi)
            diverged += 1
    assert diverged <= n // 10


def test_policy_zero_weights_is_coin_flip():
    """All-zero weights: p0 = 1/2 exactly on the GPU too, so the actions are
    exactly (u >= 1/2) and the trajectory equals the oracle's bit for bit."""
    z = {k: np.zeros_like(v) for k, v in workloads.mlp_weights(0).items()}
    n, T, seed = 200, 40, 9
    for dtype in ("f32", "bf16"):
        g = _gpu_policy_run(n, T, 8, z, dtype, seed)
        assert np.all(g["p0"] == 0.5)
        assert np.all(np.abs(g["logp"] + np.log(2.0)) <= 1e-7) and np.all(g["value"] == 0.0)
        sim = oracle.Sim(n, 0, oracle.make_params(**workloads.CARTPOLE))
        sim.reset(seed)
        r = sim.step(T, policy=oracle.Policy(**z))
        for k in ("obs", "action", "done"):
            assert np.array_equal(np.asarray(g[k]).view(np.uint8), np.asarray(r[k]).view(np.uint8)), (dtype, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_workload_full_size_sampled(dtype):
    """1,048,576 envs x 256 steps in 16 launches of K = 16 (the bench shape):
    teacher-forced checks on sampled slices, properties on the whole batch."""
    w = workloads.WORKLOADS[workloads.MLP]
    n, T, K, seed = w["n"], w["T"], w["K"][0], w["seed"]
    wts = workloads.mlp_weights(seed)
    slices = [(0, 64), (n - 64, n)]
    g = _gpu_policy_run(n, T, K, wts, dtype, seed, slices=slices)
    env_ids = list(range(0, 64)) + list(range(n - 64, n))
    # teacher-forced on the first 32 steps of the sampled envs (oracle cost)
    gs = {k: (v[:32] if isinstance(v, np.ndarray) else v) for k, v in g.items()}
    _check_teacher_forced(gs, wts, dtype, seed, env_ids)
    assert g["t"] == T
    assert np.all(g["reward"] == 1.0) and int(g["action"].max()) <= 1 and int(g["done"].max()) <= 3


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_without_value_head_or_learner_outputs(dtype):
    """No value head, or no learner planes: p0 and the trajectory are what they
    are with them (the extra outputs change nothing else)."""
    n, T, K, seed = 300, 32, 16, 4
    w = policy_weights(12, 0.3)
    full = _gpu_policy_run(n, T, K, w, dtype, seed, learner=True)
    bare = _gpu_policy_run(n, T, K, w, dtype, seed, learner=False)
    nov = {k: v for k, v in w.items() if k not in ("wv", "bv")}
    nohead = _gpu_policy_run(n, T, K, nov, dtype, seed, learner=False)
    for o in (bare, nohead):
        for k in ("obs", "action", "done", "p0"):
            assert np.array_equal(np.asarray(o[k]).view(np.uint8), np.asarray(full[k]).view(np.uint8)), k
    _check_teacher_forced(full, w, dtype, seed, list(range(n)))


def test_learner_batch_is_zero_copy_and_consistent():
    """The learner reads the kernel's own buffers: views, not copies.  A plain
    fp32 torch re-evaluation of the policy on those views reproduces the
    recorded log pi and value (the first-epoch importance ratio of a PPO-style
    learner is 1)."""
    import paper_2207_07736_amd as p
    n, T, K, seed = 4096, 64, 16, 3
    w = policy_weights(5, 0.3)
    st, keep = device_policy(w, "f32")
    sim = p.Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(seed)
        tr = p.Trajectory(T, n, learner=True)
        for k0 in range(0, T, K):
            sim.step(K, tr.rows(k0, K), policy=st)
        torch.cuda.synchronize()
        b = tr.learner_batch()
        assert b["obs"].data_ptr() == tr.obs.data_ptr() and b["obs"].shape == (T, n, 4)
        for k in ("action", "reward", "done", "logp", "value"):
            assert b[k].data_ptr() == getattr(tr, k).data_ptr()
        x = b["obs"].reshape(-1, 4)
        W = {k: torch.from_numpy(w[k]).cuda() for k in w}
        h = torch.tanh(x @ W["w1"].T + W["b1"])
        h = torch.tanh(h @ W["w2"].T + W["b2"])
        logits = h @ W["w3"].T + W["b3"]
        value = (h @ W["wv"].T + W["bv"])[:, 0]
        logp = torch.log_softmax(logits, dim=1).gather(1, b["action"].reshape(-1, 1).long())[:, 0]
        ratio = torch.exp(logp - b["logp"].reshape(-1))
        assert float((ratio - 1).abs().max()) < 1e-4
        assert float((value - b["value"].reshape(-1)).abs().max()) < 1e-4
        del tr, b
    finally:
        sim.close()
    del keep


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_env_results_independent_of_n(dtype):
    """The MLP mixes 64 environments per wave in its matrix tiles, but each
    environment's outputs are its own column: the first 300 environments of a
    1,000-env run equal a 300-env run bit for bit (p0, log pi, value, actions)."""
    w = policy_weights(4, 0.3)
    small = _gpu_policy_run(300, 32, 16, w, dtype, 6)
    big = _gpu_policy_run(1000, 32, 16, w, dtype, 6, slices=[(0, 300)])
    for k in ("obs", "action", "done", "p0", "logp", "value"):
        assert np.array_equal(np.asarray(small[k]).view(np.uint8), np.asarray(big[k]).view(np.uint8)), k


def test_policy_errors():
    import paper_2207_07736_amd as p
    w = workloads.mlp_weights(0)
    st, keep = device_policy(w, "f32")
    sim = p.Simulator(100, 2, workloads.CARTPOLE)
    try:
        sim.reset(0)
        with pytest.raises(p.RlsimError) as e:
            sim.step(4, None, policy=st)
        assert e.value.code == p.RLSIM_EUNSUPPORTED
    finally:
        sim.close()
    sim = p.Simulator(100, 0, workloads.CARTPOLE)
    try:
        sim.reset(0)
        bad = p.rlsim_policy(7, st.w1, st.b1, st.w2, st.b2, st.w3, st.b3)
        with pytest.raises(p.RlsimError) as e:
            sim.step(4, None, policy=bad)
        assert e.value.code == p.RLSIM_EINVAL
        bad = p.rlsim_policy(p.RLSIM_F32, None, st.b1, st.w2, st.b2, st.w3, st.b3)
        with pytest.raises(p.RlsimError) as e:
            sim.step(4, None, policy=bad)
        assert e.value.code == p.RLSIM_EINVAL
        tr = p.Trajectory(4, 100, learner=True)
        with pytest.raises(p.RlsimError) as e:                     # learner planes without a policy
            sim.step(4, tr.rows(0, 4))
        assert e.value.code == p.RLSIM_EINVAL
        nohead = p.rlsim_policy(p.RLSIM_F32, st.w1, st.b1, st.w2, st.b2, st.w3, st.b3, None, None)
        with pytest.raises(p.RlsimError) as e:                     # value plane without a value head
            sim.step(4, tr.rows(0, 4), policy=nohead)
        assert e.value.code == p.RLSIM_EINVAL
        mis = p.rlsim_policy(p.RLSIM_F32, st.w1, st.b1, st.w2, st.b2, st.w3, st.b3, st.wv + 2, st.bv)
        with pytest.raises(p.RlsimError) as e:
            sim.step(4, None, policy=mis)
        assert e.value.code == p.RLSIM_EINVAL
        sim.step(4, tr.rows(0, 4), policy=st)                      # the handle still works
        torch.cuda.synchronize()
        del tr
    finally:
        sim.close()
    del keep


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 63, 65, 257])
def test_policy_tiny_and_ragged_env_counts(dtype, n):
    """Env counts that leave most of a wave's matrix columns, or a workgroup's
    waves, empty: every recorded step still follows the teacher-forced rules."""
    w = policy_weights(31, 0.2)
    g = _gpu_policy_run(n, 24, 8, w, dtype, 13)
    _check_teacher_forced(g, w, dtype, 13, list(range(n)))
    assert g["t"] == 24


def _policy_case(i):
    rng = np.random.Generator(np.random.PCG64(5000 + i))
    dtype = ("f32", "bf16")[i % 2]
    n = int(rng.choice([1, 64, 100, 257, 1000, 3000]))
    T = int(rng.integers(1, 65))
    cuts = sorted(set(int(c) for c in rng.integers(1, T, size=int(rng.integers(0, 4)))) if T > 1 else [])
    bounds = [0] + cuts + [T]
    sched = [b - a for a, b in zip(bounds[:-1], bounds[1:])]
    w = policy_weights(int(rng.integers(0, 1000)), float(rng.choice([0.0, 0.3, 1.0])))
    scale = float(rng.choice([0.25, 1.0, 3.0]))          # from nearly linear to saturated units
    for k in ("w1", "w2", "w3", "wv"):
        w[k] = (w[k] * scale).astype(np.float32)
    seed = int(rng.integers(0, 2**63))
    return dtype, n, sched, w, seed


@pytest.mark.parametrize("i", range(int(os.environ.get("RLSIM_POLICY_CASES", "16"))))
def test_policy_random_cases(i):
    """Seeded draws of precision, env count, K schedule, weight scale (nearly
    linear to saturated hidden units), biases and seed; every recorded step
    against the oracle's enclosures with the compiled checker."""
    import paper_2207_07736_amd as p
    dtype, n, sched, w, seed = _policy_case(i)
    T = sum(sched)
    print(f"policy case {i}: {dtype} n={n} sched={sched} seed={seed}", flush=True)
    st, keep = device_policy(w, dtype)
    sim = p.Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(seed)
        tr = p.Trajectory(T, n, p0=True, learner=True)
        k0 = 0
        for k in sched:
            sim.step(k, tr.rows(k0, k), policy=st)
            k0 += k
        torch.cuda.synchronize()
        g = {key: getattr(tr, key).cpu().numpy() for key in ("obs", "action", "reward", "done", "policy_p0", "logp",
                                                             "value")}
        del tr
    finally:
        sim.close()
    del keep
    bad, first, stats = oracle.check_policy_rows(
        oracle.make_params(**workloads.CARTPOLE), oracle.Policy(**w, bf16=(dtype == "bf16")), seed, 0, 0, g["obs"],
        g["action"], g["reward"], g["done"], g["policy_p0"], policy_bounds.errs(), logp=g["logp"], value=g["value"])
    assert bad == 0, (i, bad, first, stats)
    if dtype == "f32":
        assert stats["worst"] <= F32_P0_GATE, stats


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_last_steps_below_the_global_step_limit(dtype):
    """The policy kernel's final K steps before the global step reaches
    2^32 - 1 (the sampling uniforms' counter block t >> 2 at its largest), from
    a mid-episode state: every step inside the enclosures, the episode counters
    continue from the state that was set, and one further step is rejected."""
    import paper_2207_07736_amd as p
    n, K, seed = 300, 48, 77
    t_start = (1 << 32) - 1 - K
    w = policy_weights(8, 0.3)
    st, keep = device_policy(w, dtype)
    sim = p.Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(seed)
        state, _, _ = sim.get_state()
        ep0 = np.random.default_rng(9).integers(0, 500, n).astype(np.uint32)
        sim.set_state(state, ep0, t_start)
        tr = p.Trajectory(K, n, p0=True, learner=True)
        sim.step(16, tr.rows(0, 16), policy=st)
        sim.step(K - 16, tr.rows(16, K - 16), policy=st)
        torch.cuda.synchronize()
        g = {key: getattr(tr, key).cpu().numpy() for key in ("obs", "action", "reward", "done", "policy_p0", "logp",
                                                             "value")}
        _, ep_end, t_end = sim.get_state()
        assert t_end == (1 << 32) - 1
        with pytest.raises(p.RlsimError) as e:
            sim.step(1, policy=st)
        assert e.value.code == p.RLSIM_EINVAL
        del tr
    finally:
        sim.close()
    del keep
    assert np.array_equal(g["obs"][0], state)
    assert (g["done"] & 2).any()
    bad, first, stats = oracle.check_policy_rows(
        oracle.make_params(**workloads.CARTPOLE), oracle.Policy(**w, bf16=(dtype == "bf16")), seed, 0, t_start,
        g["obs"], g["action"], g["reward"], g["done"], g["policy_p0"], policy_bounds.errs(), logp=g["logp"],
        value=g["value"], ep0=ep0)
    assert bad == 0, (bad, first, stats)
    if dtype == "f32":
        assert stats["worst"] <= F32_P0_GATE, stats
    # the episode counters: ep0 plus the steps since the last done (0 after it)
    done_any = (g["done"] != 0)
    last = np.where(done_any.any(axis=0), K - 1 - np.argmax(done_any[::-1], axis=0), -1)
    want = np.where(last >= 0, K - 1 - last, ep0 + K).astype(np.uint32)
    assert np.array_equal(ep_end, want)
