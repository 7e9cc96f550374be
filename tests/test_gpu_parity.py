"""GPU parity: the HIP library against the CPU oracle, through the C ABI.

Random-action runs are compared bit for bit: observations, actions, rewards,
done bytes, block statistics, the final state (cart-pole and padding words),
the episode counters and the global step.  Sizes span several 256-env tiles
and ragged tails; the full-size workloads are compared on sampled env slices
(oracle on the same global env ids) plus properties that hold at any size.
"""
import numpy as np
import pytest

import workloads
from gpu_helpers import assert_bit_equal, gpu_run, oracle_run

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401  (fails loudly if the library is missing)


def _stats_equal(g, r):
    assert len(g) == len(r)
    for a, b in zip(g, r):
        assert np.array_equal(a, b)


def test_small_workload_full_bit_exact():
    """1,024 envs, 100 steps, one launch per step (the unfused form), seed 0."""
    w = workloads.WORKLOADS[workloads.SMALL]
    sched = [1] * w["T"]
    g = gpu_run(w["n"], w["T"], sched, seed=w["seed"])
    r = oracle_run(w["n"], w["T"], sched, seed=w["seed"])
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])
    assert r["done"].any()          # episodes do end within the run


@pytest.mark.parametrize("seed", workloads.PARITY_SEEDS)
@pytest.mark.parametrize("n", [1, 257, 1000])
def test_ragged_sizes_and_seeds(n, seed):
    T = 150
    sched = [1, 6, 57, 86]                       # unaligned call boundaries
    g = gpu_run(n, T, sched, seed=seed)
    r = oracle_run(n, T, sched, seed=seed)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("sched", [[300], [1] * 300, [7] * 42 + [6], [128, 129, 43]])
def test_k_partitions_match_oracle(sched):
    n, T = 700, 300
    g = gpu_run(n, T, sched, seed=1)
    r = oracle_run(n, T, [T], seed=1)
    assert_bit_equal(g, r)


@pytest.mark.parametrize("D", [1, 4, 5, 16])
def test_padding_words_bit_exact(D):
    n, T = 513, 260
    sched = [100, 160]
    g = gpu_run(n, T, sched, D=D, seed=2)
    r = oracle_run(n, T, sched, D=D, seed=2)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("overrides", [
    dict(max_episode_steps=5),
    dict(max_episode_steps=0, no_termination=1),
    dict(max_episode_steps=3, x_threshold=0.01),        # terminated and truncated together
    dict(max_episode_steps=1),
    dict(force_mag=0.0, gravity=0.0),
])
def test_edge_configs(overrides):
    """Edge configurations; with termination disabled the pole swings through
    every angle (the quadrant-reduced sin/cos), and every state stays finite."""
    cfg = workloads.cartpole(**overrides)
    n, T = 300, 120
    g = gpu_run(n, T, [50, 70], D=2, seed=3, cfg=cfg)
    r = oracle_run(n, T, [50, 70], D=2, seed=3, cfg=cfg)
    assert_bit_equal(g, r)
    assert np.isfinite(g["obs"]).all() and np.isfinite(g["state"]).all()
    if overrides.get("no_termination"):
        assert np.abs(g["obs"][:, 2]).max() > 4.0        # far past the series' own domain
    _stats_equal(g["stats"], r["stats"])


def test_k_sweep_workload_full_size():
    """65,536 envs x 1,000 steps: K = 1, 10, 100 and 1,000 give the identical
    trajectory; sampled slices equal the oracle."""
    w = workloads.WORKLOADS[workloads.K_SWEEP]
    n, T = w["n"], w["T"]
    slices = [(0, 256), (30000, 30100), (n - 256, n)]
    outs = {K: gpu_run(n, T, [K] * (T // K), seed=w["seed"], slices=slices) for K in w["K"]}
    base = outs[1000]
    for K, o in outs.items():
        assert_bit_equal(o, base)
    ref = [oracle_run(b - a, T, [T], seed=w["seed"], env0=a) for a, b in slices]
    merged = {key: np.concatenate([x[key] for x in ref], axis=-1) for key in ("obs", "action", "reward", "done", "state")}
    merged["ep"] = np.concatenate([x["ep"] for x in ref])
    merged["t"] = T
    assert_bit_equal(base, merged)


def test_headline_sampled_and_properties():
    """4,194,304 envs x 200 steps in one launch (K = 200), as the bench times it."""
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T = w["n"], w["T"]
    slices = [(0, 256), (2097152, 2097152 + 256), (n - 512, n)]
    g = gpu_run(n, T, [T], seed=w["seed"], slices=slices)
    ref = [oracle_run(b - a, T, [T], seed=w["seed"], env0=a) for a, b in slices]
    merged = {key: np.concatenate([x[key] for x in ref], axis=-1) for key in ("obs", "action", "reward", "done", "state")}
    merged["ep"] = np.concatenate([x["ep"] for x in ref])
    merged["t"] = T
    assert_bit_equal(g, merged)
    # block statistics of the sampled blocks
    blocks = [0, 2097152 // 256, n // 256 - 2, n // 256 - 1]
    want = np.concatenate([ref[0]["stats"][0], ref[1]["stats"][0], ref[2]["stats"][0]])
    assert np.array_equal(g["stats"][0][blocks], want)


def test_headline_whole_batch_properties():
    """Properties of the full headline trajectory that hold at any size: every
    reward is 1, actions are bits, done bytes are in {0..3}, the block statistics
    count exactly the done bytes, and stored episode counters stay below 500."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T = w["n"], w["T"]
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(w["seed"])
        traj = Trajectory(T, n)
        sim.step(T, traj.rows(0, T))
        torch.cuda.synchronize()
        assert bool((traj.reward == 1.0).all())
        assert int(traj.action.max()) <= 1
        assert int(traj.done.max()) <= 3
        dn = traj.done.to(torch.int64)
        per_env = (dn != 0).sum(dim=0)
        per_block = per_env.view(-1, 256).sum(dim=1)
        stats = traj.block_stats.to(torch.int64)
        assert torch.equal(stats[:, 0], per_block)
        # column 1, the summed lengths of the episodes that ended: each env's
        # ended episodes span from its first step to its last episode end
        # (episodes start at the reset, t = 0), so their lengths add up to
        # 1 + the step index of the env's last done byte (0 without one)
        steps = torch.arange(1, T + 1, device=dn.device, dtype=torch.int64).view(T, 1)
        last_end = ((dn != 0).to(torch.int64) * steps).max(dim=0).values
        assert torch.equal(stats[:, 1], last_end.view(-1, 256).sum(dim=1))
        assert torch.equal(stats[:, 2], (dn & 1).sum(dim=0).view(-1, 256).sum(dim=1))
        assert torch.equal(stats[:, 3], (dn >> 1).sum(dim=0).view(-1, 256).sum(dim=1))
        _, ep, t = sim.get_state()
        assert t == T and int(ep.max()) < 500
        # fraction of env-steps that end an episode: ~1/22 for random pushes
        frac = float(per_env.sum()) / (n * T)
        assert 0.035 < frac < 0.055
        del traj
    finally:
        sim.close()


def test_rerun_deterministic_and_stream():
    n, T = 4096, 64
    s = torch.cuda.Stream()
    a = gpu_run(n, T, [T], seed=5, stream=s)
    b = gpu_run(n, T, [32, 32], seed=5)
    assert_bit_equal(a, b)


def test_no_trajectory_and_stats_only():
    from paper_2207_07736_amd import Simulator, stats_only
    n, T = 1000, 90
    r = oracle_run(n, T, [T], seed=4)
    sim = Simulator(n, 3, workloads.CARTPOLE)
    try:
        sim.reset(4)
        sim.step(T, None)                       # traj NULL: pure simulation
        st_a, ep_a, t_a = sim.get_state()
        sim.reset(4)
        stats = torch.zeros(((n + 255) // 256, 4), dtype=torch.int32, device="cuda")
        sim.step(T, stats_only(stats, n))
        st_b, ep_b, _ = sim.get_state()
    finally:
        sim.close()
    r3 = oracle_run(n, T, [T], D=3, seed=4)
    assert np.array_equal(st_a.view(np.uint32), r3["state"].view(np.uint32)) and np.array_equal(ep_a, r3["ep"])
    assert np.array_equal(st_b.view(np.uint32), r3["state"].view(np.uint32)) and t_a == T
    assert np.array_equal(stats.cpu().numpy().view(np.uint32), r3["stats"][0])
    assert r["done"].any()


def test_get_set_state_resume():
    from paper_2207_07736_amd import Simulator, Trajectory
    n, T, D = 777, 140, 4
    whole = gpu_run(n, T, [T], D=D, seed=8)
    sim = Simulator(n, D, workloads.CARTPOLE)
    sim2 = Simulator(n, D, workloads.CARTPOLE)
    try:
        sim.reset(8)
        tr1 = Trajectory(T // 2, n)
        sim.step(T // 2, tr1.rows(0, T // 2))
        st, ep, t = sim.get_state()
        sim2.reset(8)                              # same padding parameters
        sim2.set_state(st, ep, t)
        tr2 = Trajectory(T - T // 2, n)
        sim2.step(T - T // 2, tr2.rows(0, T - T // 2))
        torch.cuda.synchronize()
        obs = np.concatenate([tr1.obs.cpu().numpy(), tr2.obs.cpu().numpy()])
        done = np.concatenate([tr1.done.cpu().numpy(), tr2.done.cpu().numpy()])
        assert np.array_equal(obs.view(np.uint32), whole["obs"].view(np.uint32))
        assert np.array_equal(done, whole["done"])
        st2, ep2, t2 = sim2.get_state()
        assert np.array_equal(st2.view(np.uint32), whole["state"].view(np.uint32)) and t2 == T
    finally:
        sim.close()
        sim2.close()


def test_nan_state_propagates_like_oracle():
    """A NaN injected through set_state never crosses a threshold (NaN compares
    false), so the env runs to the time limit; both sides agree on NaN-ness."""
    import oracle
    from paper_2207_07736_amd import Simulator, Trajectory
    n, T = 300, 40
    cfg = workloads.cartpole(max_episode_steps=30)
    sim = Simulator(n, 0, cfg)
    osim = oracle.Sim(n, 0, oracle.make_params(**cfg))
    try:
        sim.reset(1)
        osim.reset(1)
        st, ep, t = sim.get_state()
        st[2, 5] = np.nan
        st[0, 100] = np.inf
        sim.set_state(st, ep, t)
        osim.set_state(st, ep, t)
        tr = Trajectory(T, n)
        sim.step(T, tr.rows(0, T))
        torch.cuda.synchronize()
        ref = osim.step(T)
        g_done = tr.done.cpu().numpy()
        assert np.array_equal(g_done, ref["done"])
        g_obs = tr.obs.cpu().numpy()
        assert np.array_equal(np.isnan(g_obs), np.isnan(ref["obs"]))
        fin = ~np.isnan(g_obs)
        assert np.array_equal(g_obs[fin].view(np.uint32), ref["obs"][fin].view(np.uint32))
    finally:
        sim.close()


@pytest.mark.parametrize("D", [0, 4, 100])
def test_last_steps_below_the_global_step_limit(D):
    """The final K steps before the global step reaches 2^32 - 1: the Philox
    counter blocks (t >> 3, t >> 7) take their largest values and nothing wraps;
    one further step is rejected.  Episode counters near the time limit make the
    truncation path run there too."""
    import oracle
    from paper_2207_07736_amd import RLSIM_EINVAL, RlsimError, Simulator, Trajectory
    n, K, seed = 300, 40, (1 << 40) + 7
    t_start = (1 << 32) - 1 - K
    sim = Simulator(n, D, workloads.CARTPOLE)
    osim = oracle.Sim(n, D, oracle.make_params(**workloads.CARTPOLE))
    try:
        sim.reset(seed)
        osim.reset(seed)
        st, ep, _ = sim.get_state()
        ep = np.random.default_rng(5).integers(0, 500, n).astype(np.uint32)
        sim.set_state(st, ep, t_start)
        osim.set_state(st, ep, t_start)
        tr = Trajectory(K, n)
        sim.step(K, tr.rows(0, K))
        torch.cuda.synchronize()
        ref = osim.step(K)
        for key in ("obs", "action", "reward", "done"):
            g = getattr(tr, key).cpu().numpy()
            assert np.array_equal(g.view(np.uint8), ref[key].view(np.uint8)), key
        assert (tr.done.cpu().numpy() & 2).any()
        g_st, g_ep, g_t = sim.get_state()
        r_st, r_ep, r_t = osim.get_state()
        assert np.array_equal(g_st.view(np.uint32), r_st.view(np.uint32))
        assert np.array_equal(g_ep, r_ep) and g_t == r_t == (1 << 32) - 1
        with pytest.raises(RlsimError) as e:
            sim.step(1)
        assert e.value.code == RLSIM_EINVAL
    finally:
        sim.close()


@pytest.mark.parametrize("n", [1, 63, 65, 257, 1000])
def test_warp_specialised_chunk_tails_and_ragged_blocks(n):
    """Trajectory calls of K >= 16 steps without padding words run the
    warp-specialised kernel (rows handed from stepping to storing waves in
    4-step chunks): K on and off the chunk size around the threshold, blocks
    whose stepping waves are partly or wholly past n, with and without the
    block statistics."""
    sched = [15, 16, 17, 18, 19, 20, 33, 64]
    T = sum(sched)
    r = oracle_run(n, T, sched, seed=12)
    for stats in (True, False):
        g = gpu_run(n, T, sched, seed=12, stats=stats)
        assert_bit_equal(g, r)
        if stats:
            _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("D", [1, 3, 4])
@pytest.mark.parametrize("n", [1, 257, 1000])
def test_warp_specialised_padding_words(D, n):
    """Calls of K >= 64 steps with 1-4 padding words run the warp-specialised
    kernel with the words in the stepping waves' registers; K = 63 does not.
    Chunk tails, blocks past n and the padding state against the oracle."""
    sched = [64, 65, 130, 63, 66]
    T = sum(sched)
    g = gpu_run(n, T, sched, D=D, seed=14)
    r = oracle_run(n, T, sched, D=D, seed=14)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("overrides", [
    dict(max_episode_steps=5),
    dict(max_episode_steps=0, no_termination=1),
    dict(max_episode_steps=3, x_threshold=0.01),
    dict(max_episode_steps=1),
    dict(force_mag=0.0, gravity=0.0),
    dict(compute_factor=7),
])
def test_warp_specialised_edge_configs(overrides):
    """The edge configurations and a compute factor through the
    warp-specialised kernel (D = 0, K >= 16)."""
    cfg = workloads.cartpole(**overrides)
    n, T = 300, 120
    g = gpu_run(n, T, [50, 70], seed=3, cfg=cfg)
    r = oracle_run(n, T, [50, 70], seed=3, cfg=cfg)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("C", [2, 7, 64])
def test_compute_factor_bit_exact(C):
    """The paper's compute factor: C Euler iterations of tau / C per step."""
    cfg = workloads.cartpole(compute_factor=C)
    n, T = 300, 90
    g = gpu_run(n, T, [1, 40, 49], D=3, seed=6, cfg=cfg)
    r = oracle_run(n, T, [1, 40, 49], D=3, seed=6, cfg=cfg)
    assert_bit_equal(g, r)
    for a, b in zip(g["stats"], r["stats"]):
        assert np.array_equal(a, b)


def test_max_envs_sampled():
    """The largest handle the ABI allows, 2^30 environments, 2 steps in one launch
    with trajectory and statistics: sampled env slices (first, middle, last) equal
    the oracle bit for bit, including the byte offsets near 2^32 of the last envs."""
    from paper_2207_07736_amd import Simulator, Trajectory
    torch.cuda.empty_cache()
    n, T = 1 << 30, 2
    slices = [(0, 256), (1 << 29, (1 << 29) + 256), (n - 512, n)]
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(7)
        traj = Trajectory(T, n)
        sim.step(T, traj.rows(0, T))
        torch.cuda.synchronize()
        cols = lambda x: np.concatenate([x[..., a:b].cpu().numpy() for a, b in slices], axis=-1)  # noqa: E731
        g = dict(obs=cols(traj.obs), action=cols(traj.action), reward=cols(traj.reward), done=cols(traj.done))
        blocks = [0, (1 << 29) // 256, n // 256 - 2, n // 256 - 1]
        g_stats = traj.block_stats[blocks].cpu().numpy().view(np.uint32)
        del traj
        state, ep, t = sim.get_state()
        g["state"] = np.concatenate([state[:, a:b] for a, b in slices], axis=1)
        g["ep"] = np.concatenate([ep[a:b] for a, b in slices])
        g["t"] = t
        del state, ep
    finally:
        sim.close()
        torch.cuda.empty_cache()
    ref = [oracle_run(b - a, T, [T], seed=7, env0=a) for a, b in slices]
    merged = {key: np.concatenate([x[key] for x in ref], axis=-1) for key in ("obs", "action", "reward", "done", "state")}
    merged["ep"] = np.concatenate([x["ep"] for x in ref])
    merged["t"] = T
    assert_bit_equal(g, merged)
    want = np.concatenate([ref[0]["stats"][0], ref[1]["stats"][0], ref[2]["stats"][0]])
    assert np.array_equal(g_stats, want)


@pytest.mark.parametrize("D", [0, 5, 20])
def test_env_results_independent_of_n(D):
    """Environment e's trajectory, statistics row and final state do not depend on
    how many environments the handle holds (kernel mapping, tiles, tails)."""
    T, sched = 120, [50, 70]
    small = gpu_run(300, T, sched, D=D, seed=12)
    big = gpu_run(2000, T, sched, D=D, seed=12, slices=[(0, 300)])
    assert_bit_equal(small, big)
    # the first statistics row covers envs 0..255 in both runs
    for a, b in zip(small["stats"], big["stats"]):
        assert np.array_equal(a[0], b[0])


def test_concurrent_handles_on_two_streams_match_solo_runs():
    """Two handles (different sizes, padding words and seeds) stepped in
    interleaved calls on two streams, with the streams overlapping: each
    handle's trajectory and final state equal its solo run bit for bit (the
    library keeps no state outside the handle)."""
    from paper_2207_07736_amd import Simulator, Trajectory
    specs = [(3000, 0, 11, [40, 1, 39]), (1500, 24, 12, [1] * 20 + [60])]
    solo = [gpu_run(n, sum(sch), sch, D=D, seed=seed, stats=False) for n, D, seed, sch in specs]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    sims, trajs = [], []
    try:
        for (n, D, seed, sch), s in zip(specs, streams):
            sim = Simulator(n, D, workloads.CARTPOLE, stream=s)
            sim.reset(seed)
            sims.append(sim)
            trajs.append(Trajectory(sum(sch), n, stats=False))
        torch.cuda.synchronize()
        k0 = [0, 0]
        queues = [list(sch) for _, _, _, sch in specs]
        while queues[0] or queues[1]:
            for h in (0, 1):
                if queues[h]:
                    k = queues[h].pop(0)
                    sims[h].step(k, trajs[h].rows(k0[h], k))
                    k0[h] += k
        torch.cuda.synchronize()
        for h in (0, 1):
            got = {key: getattr(trajs[h], key).cpu().numpy() for key in ("obs", "action", "reward", "done")}
            state, ep, t = sims[h].get_state()
            got.update(state=state, ep=ep, t=t)
            for key in ("obs", "action", "reward", "done", "state", "ep"):
                assert np.array_equal(np.asarray(got[key]).view(np.uint8), np.asarray(solo[h][key]).view(np.uint8)), (h, key)
            assert got["t"] == solo[h]["t"]
    finally:
        for sim in sims:
            sim.close()


@pytest.mark.parametrize("D", [0, 5, 20])
def test_env0_handle_equals_oracle_slice(D):
    """A handle holding global environments env0 .. env0 + n - 1 draws the
    random numbers of those environments: bit-exact against the oracle's slice
    with the same global ids (trajectory, statistics rows, final state)."""
    env0, n, T = 3 * 2**20, 700, 90
    sched = [40, 50]
    g = gpu_run(n, T, sched, D=D, seed=6, env0=env0)
    r = oracle_run(n, T, sched, D=D, seed=6, env0=env0)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("D", [0, 3, 40])
def test_shards_equal_the_single_handle(D):
    """Two handles of 1,024 environments at env0 = 0 and 1,024 record exactly
    the columns of one 2,048-env handle (the sharding of the path over GPUs,
    here on one GPU), for random actions, and the last one's statistics rows
    are rows 4 .. 7 of the whole handle's."""
    T, sched = 100, [30, 70]
    whole = gpu_run(2048, T, sched, D=D, seed=12)
    for env0 in (0, 1024):
        part = gpu_run(1024, T, sched, D=D, seed=12, env0=env0)
        cols = {k: (whole[k][..., env0:env0 + 1024] if k != "ep" else whole[k][env0:env0 + 1024])
                for k in ("obs", "action", "reward", "done", "state", "ep")}
        cols["t"] = whole["t"]
        assert_bit_equal(part, cols)
        for a, b in zip(part["stats"], whole["stats"]):
            assert np.array_equal(a, b[env0 // 256:env0 // 256 + 4])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_shards_equal_the_single_handle_with_policy(dtype):
    """As above with the MLP policy sampling the actions (its uniforms are
    keyed by global env ids too): bit-identical shards."""
    from gpu_helpers import device_policy, policy_weights
    st, keep = device_policy(policy_weights(3, bias_scale=0.2), dtype)
    T, sched = 48, [16, 32]
    whole = gpu_run(1024, T, sched, seed=4, policy=st, p0=True)
    part = gpu_run(512, T, sched, seed=4, policy=st, p0=True, env0=512)
    cols = {k: whole[k][..., 512:] for k in ("obs", "action", "reward", "done", "p0", "state")}
    cols["ep"], cols["t"] = whole["ep"][512:], whole["t"]
    assert_bit_equal(part, cols, keys=("obs", "action", "reward", "done", "p0", "state", "ep"))
    del keep


def test_step_rejects_rows_cut_for_another_call():
    """Rows cut for another K, another environment count or another state size
    raise before anything is enqueued: the handle's step counter is unchanged
    and a correct call afterwards matches the oracle."""
    from paper_2207_07736_amd import Simulator, Trajectory
    n = 300
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(2)
        tr = Trajectory(200, n)
        other_n = Trajectory(10, n + 1)
        other_s = Trajectory(10, n, S=6)
        for K, rows in ((200, tr.rows(0, 100)), (5, tr.rows(0, 10)), (10, other_n.rows(0, 10)),
                        (10, other_s.rows(0, 10))):
            with pytest.raises(ValueError):
                sim.step(K, rows)
        with pytest.raises(TypeError):
            sim.step(10, rows.struct)
        assert sim.get_state()[2] == 0
        sim.step(10, tr.rows(0, 10))
        torch.cuda.synchronize()
        r = oracle_run(n, 10, [10], seed=2)
        assert np.array_equal(tr.obs[:10].cpu().numpy().view(np.uint32), r["obs"].view(np.uint32))
        del tr, other_n, other_s
    finally:
        sim.close()


@pytest.mark.parametrize("n", [4, 260, 1028, 4096])
def test_warp_specialised_more_shapes(n):
    """The warp-specialised kernel at environment counts that are multiples of
    4 (a full block, a few lanes of a second one), over chunk tails (K = 17, 18,
    19, 65) and long calls."""
    sched = [16, 17, 18, 19, 65, 200]
    T = sum(sched)
    g = gpu_run(n, T, sched, seed=21)
    r = oracle_run(n, T, sched, seed=21)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])


def test_warp_specialised_planes_only_4_byte_aligned():
    """Trajectory planes that are 4- but not 16-byte aligned (a buffer offset by
    one float, which the ABI allows) record the oracle's trajectory bit for
    bit."""
    from paper_2207_07736_amd import Simulator, TrajRows, traj_struct
    n, K = 1024, 40
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(3)
        obs_buf = torch.empty(K * 4 * n + 1, dtype=torch.float32, device="cuda")
        rew_buf = torch.empty(K * n + 1, dtype=torch.float32, device="cuda")
        obs, rew = obs_buf[1:].view(K, 4, n), rew_buf[1:].view(K, n)
        act = torch.empty((K, n), dtype=torch.uint8, device="cuda")
        done = torch.empty((K, n), dtype=torch.uint8, device="cuda")
        assert obs.data_ptr() % 16 != 0
        sim.step(K, TrajRows(traj_struct(obs, act, rew, done), K, n, 4))
        torch.cuda.synchronize()
        r = oracle_run(n, K, [K], seed=3)
        assert np.array_equal(obs.cpu().numpy().view(np.uint32), r["obs"].view(np.uint32))
        assert np.array_equal(act.cpu().numpy(), r["action"]) and np.array_equal(done.cpu().numpy(), r["done"])
        assert bool((rew == 1.0).all())
    finally:
        sim.close()
