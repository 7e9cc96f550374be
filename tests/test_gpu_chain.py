"""GPU parity of the second simulator, the cart carrying a chain of N uniform
rods, against the CPU oracle through the C ABI: bit for bit (observations,
actions, rewards, done bytes, block statistics, final state, counters, step),
for N = 1 .. 4, ragged environment counts, K partitions, seeds, edge
configurations (termination off, so the links swing through every angle),
compute factors, global env offsets and resume; the full-size chain workload
(1,048,576 envs x 200 steps in one launch) sampled, and every env-step of it
for N = 2 checked teacher-forced."""
import concurrent.futures as cf
import os

import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import assert_bit_equal, gpu_run, oracle_run

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401


def _stats_equal(g, r):
    assert len(g) == len(r)
    for a, b in zip(g, r):
        assert np.array_equal(a, b)


def _both(n, T, sched, N, seed=0, cfg=None, env0=0):
    print(f"chain N={N} n={n} T={T} sched={sched} seed={seed} env0={env0} cfg={cfg}", flush=True)
    g = gpu_run(n, T, sched, seed=seed, cfg=cfg, links=N, env0=env0)
    r = oracle_run(n, T, sched, seed=seed, cfg=cfg, links=N, env0=env0)
    assert_bit_equal(g, r)
    _stats_equal(g["stats"], r["stats"])
    return g, r


@pytest.mark.parametrize("N", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 257, 1000])
def test_chain_ragged_sizes(N, n):
    g, r = _both(n, 150, [1, 6, 57, 86], N, seed=N + n)
    assert g["obs"].shape == (150, 2 * N + 2, n)
    if n > 1:
        assert r["done"].any()


@pytest.mark.parametrize("N", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 63, 65, 257, 1000])
def test_chain_warp_specialised_shapes(N, n):
    """Trajectory calls of K >= 16 steps run the warp-specialised chain kernel
    (rows handed from stepping to storing waves in 2-step chunks): K on and
    off the chunk size around the threshold, blocks whose stepping waves are
    partly or wholly past n, with and without the block statistics."""
    sched = [15, 16, 17, 18, 33, 2, 64]
    T = sum(sched)
    print(f"chain split N={N} n={n} sched={sched}", flush=True)
    r = oracle_run(n, T, sched, seed=40 + N, links=N)
    for stats in (True, False):
        g = gpu_run(n, T, sched, seed=40 + N, stats=stats, links=N)
        assert_bit_equal(g, r)
        if stats:
            _stats_equal(g["stats"], r["stats"])


@pytest.mark.parametrize("N", [2, 4])
@pytest.mark.parametrize("seed", workloads.PARITY_SEEDS)
def test_chain_seeds(N, seed):
    _both(512, 100, [100], N, seed=seed)


@pytest.mark.parametrize("sched", [[200], [1] * 200, [7] * 28 + [4], [128, 72]])
def test_chain_k_partitions(sched):
    n, T = 600, 200
    g = gpu_run(n, T, sched, seed=1, links=3)
    r = oracle_run(n, T, [T], seed=1, links=3)
    assert_bit_equal(g, r)


@pytest.mark.parametrize("N", [1, 2, 4])
@pytest.mark.parametrize("overrides", [
    dict(max_episode_steps=5),
    dict(max_episode_steps=0, no_termination=1),
    dict(max_episode_steps=3, x_threshold=0.01),
    dict(max_episode_steps=1),
    dict(force_mag=0.0, gravity=0.0),
    dict(compute_factor=3),
    dict(masscart=0.7, masspole=0.23, half_length=0.35, gravity=9.81, tau=0.01),
])
def test_chain_edge_configs(N, overrides):
    """With termination off the links swing through every angle, which runs
    the quadrant reduction of sin/cos; every state stays finite.  (The free
    four-link chain's explicit-Euler integration diverges within about 75
    steps of tau = 0.02, on both sides alike; that case runs four Euler
    iterations per step instead.)"""
    if N == 4 and overrides.get("no_termination"):
        overrides = dict(overrides, compute_factor=4)
    cfg = workloads.cartpole(**overrides)
    g, _ = _both(300, 120, [50, 70], N, seed=3, cfg=cfg)
    assert np.isfinite(g["obs"]).all()
    if overrides.get("no_termination"):
        assert np.abs(g["obs"][:, 2]).max() > 1.0


@pytest.mark.parametrize("N", [1, 4])
def test_chain_env0(N):
    _both(700, 90, [40, 50], N, seed=6, env0=5 * 2**20)


def test_chain_get_set_state_resume():
    from paper_2207_07736_amd import Simulator, Trajectory
    n, T, N = 777, 140, 3
    whole = gpu_run(n, T, [T], seed=8, links=N)
    sim = Simulator(n, 0, workloads.CARTPOLE, links=N)
    sim2 = Simulator(n, 0, workloads.CARTPOLE, links=N)
    try:
        sim.reset(8)
        tr1 = Trajectory(T // 2, n, S=sim.S)
        sim.step(T // 2, tr1.rows(0, T // 2))
        st, ep, t = sim.get_state()
        assert st.shape == (2 * N + 2, n)
        sim2.reset(8)                              # the seed's Philox key
        sim2.set_state(st, ep, t)
        tr2 = Trajectory(T - T // 2, n, S=sim.S)
        sim2.step(T - T // 2, tr2.rows(0, T - T // 2))
        torch.cuda.synchronize()
        obs = np.concatenate([tr1.obs.cpu().numpy(), tr2.obs.cpu().numpy()])
        assert np.array_equal(obs.view(np.uint32), whole["obs"].view(np.uint32))
        st2, ep2, t2 = sim2.get_state()
        assert np.array_equal(st2.view(np.uint32), whole["state"].view(np.uint32)) and t2 == T
        assert np.array_equal(ep2, whole["ep"])
    finally:
        sim.close()
        sim2.close()


def test_chain_rejects_policy():
    import paper_2207_07736_amd as p
    from gpu_helpers import device_policy, policy_weights
    st, keep = device_policy(policy_weights(1), "f32")
    sim = p.Simulator(64, 0, workloads.CARTPOLE, links=2)
    try:
        sim.reset(0)
        with pytest.raises(p.RlsimError) as e:
            sim.step(4, None, policy=st)
        assert e.value.code == p.RLSIM_EUNSUPPORTED
    finally:
        sim.close()
    del keep


def _random_case(i):
    rng = np.random.Generator(np.random.PCG64(5000 + i))
    N = int(rng.integers(1, 5))
    n = int(rng.choice([1, 63, 65, 256, 300, 777, 1024, 1500]))
    T = int(rng.integers(1, 121))
    cuts = sorted(set(int(c) for c in rng.integers(1, T, size=int(rng.integers(0, 4)))) if T > 1 else [])
    bounds = [0] + cuts + [T]
    sched = [b - a for a, b in zip(bounds[:-1], bounds[1:])]
    seed = int(rng.integers(0, 2**63))
    over = {}
    if rng.random() < 0.4:
        over["max_episode_steps"] = int(rng.choice([0, 2, 9, 40]))
    if rng.random() < 0.3:
        over["force_mag"] = float(np.float32(rng.uniform(0.0, 25.0)))
    if rng.random() < 0.3:
        over["compute_factor"] = int(rng.choice([2, 4]))
    if rng.random() < 0.3:
        over["masscart"] = float(np.float32(rng.uniform(0.2, 3.0)))
        over["masspole"] = float(np.float32(rng.uniform(0.02, 0.5)))
        over["half_length"] = float(np.float32(rng.uniform(0.1, 1.0)))
        over["tau"] = float(np.float32(rng.uniform(0.002, 0.03)))
    if over.get("max_episode_steps") == 0 and rng.random() < 0.5:
        over["no_termination"] = 1
    env0 = 256 * int(rng.integers(0, 2**20)) if rng.random() < 0.3 else 0
    return N, n, T, sched, seed, over, env0


@pytest.mark.parametrize("i", range(int(os.environ.get("RLSIM_CHAIN_CASES", "24"))))
def test_chain_random_case(i):
    N, n, T, sched, seed, over, env0 = _random_case(i)
    _both(n, T, sched, N, seed=seed, cfg=workloads.cartpole(**over), env0=env0)


def _check_slice(N, seed, a, tr):
    params = oracle.make_params(**workloads.CARTPOLE)
    n = tr["action"].shape[1]
    bounds = np.linspace(0, n, THREADS + 1).astype(int)

    def one(j):
        lo, hi = int(bounds[j]), int(bounds[j + 1])
        if lo == hi:
            return 0, None
        bad, first = oracle.chain_check_rows(params, N, seed, a + lo, 0, tr["obs"][:, :, lo:hi],
                                             tr["action"][:, lo:hi], tr["reward"][:, lo:hi], tr["done"][:, lo:hi],
                                             final_state=tr["state"][:, lo:hi], final_ep=tr["ep"][lo:hi])
        return bad, (None if first is None else (first[0], first[1] + lo))

    with cf.ThreadPoolExecutor(max_workers=THREADS) as ex:
        res = list(ex.map(one, range(THREADS)))
    return sum(r[0] for r in res), [r[1] for r in res if r[1] is not None]


@pytest.mark.parametrize("N", [1, 2, 3, 4])
def test_chain_workload_full_size(N):
    """The chain workload as the bench times it (1,048,576 envs x 200 steps in
    one K = 200 launch): sampled slices against the oracle bit for bit; for
    N = 2 every env-step teacher-forced (row 0 against the reset draw, the final
    state against the last row's successor); whole-batch properties."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.CHAIN_SWEEP
    n, T, seed = w["n"], w["T"], w["seed"]
    sim = Simulator(n, 0, workloads.CARTPOLE, links=N)
    try:
        sim.reset(seed)
        tr = Trajectory(T, n, S=sim.S)
        sim.step(T, tr.rows(0, T))
        torch.cuda.synchronize()
        state, ep, t = sim.get_state()
        assert t == T
        assert bool((tr.reward == 1.0).all()) and int(tr.action.max()) <= 1 and int(tr.done.max()) <= 3
        assert bool(torch.isfinite(tr.obs).all())
        dn = tr.done.to(torch.int64)
        stats = tr.block_stats.to(torch.int64)
        assert torch.equal(stats[:, 0], (dn != 0).sum(dim=0).view(-1, 256).sum(dim=1))
        assert torch.equal(stats[:, 2], (dn & 1).sum(dim=0).view(-1, 256).sum(dim=1))
        keys = ("obs", "action", "reward", "done")
        slices = [(0, 256), (n // 2 + 512, n // 2 + 768), (n - 256, n)]
        for a, b in slices:
            cols = {k: getattr(tr, k)[..., a:b].cpu().numpy() for k in keys}
            cols["state"], cols["ep"], cols["t"] = state[:, a:b], ep[a:b], t
            ref = oracle_run(b - a, T, [T], seed=seed, links=N, env0=a)
            assert_bit_equal(cols, ref)
        if N == 2:
            S = n // 4
            for a in range(0, n, S):
                cols = {k: getattr(tr, k)[..., a:a + S].cpu().numpy() for k in keys}
                cols["state"], cols["ep"] = state[:, a:a + S], ep[a:a + S]
                bad, firsts = _check_slice(N, seed, a, cols)
                assert bad == 0, (a, bad, firsts[:4])
        del tr
    finally:
        sim.close()
