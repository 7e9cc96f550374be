"""Every recorded step of large GPU runs, teacher-forced against the oracle.

From the GPU's own obs at step t, the oracle (orc_check_rows) recomputes the
random action bit, the simulation step, the done byte (episode lengths tracked
from the reset) and the next row -- the reset draw after an episode end -- and
requires the recorded row to match bit for bit, for every environment and every
step: the whole 65,536-env x 1,000-step workload in its fused and unfused forms,
and every environment of the 4,194,304-env headline launch and of the
262,144-env state-size launch (D = 4,096; the other state sizes must record the
same trajectory).
The MLP-policy workload (1,048,576 envs x 256 steps in K = 16 launches) is
checked the same way on 32,768 of its environments, every step, by
orc_check_policy_rows: p0, log pi and the value inside the oracle's enclosures
(tests/policy_bounds.py), the action following the recorded p0 exactly, the
rest bit for bit."""
import concurrent.futures as cf
import os

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401


def _run(n, T, K, seed, cols=None):
    from paper_2207_07736_amd import Simulator, Trajectory
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(seed)
        tr = Trajectory(T, n, stats=False)
        for k0 in range(0, T, K):
            sim.step(K, tr.rows(k0, K))
        torch.cuda.synchronize()
        a, b = cols if cols else (0, n)
        out = {key: getattr(tr, key)[..., a:b].cpu().numpy() for key in ("obs", "action", "reward", "done")}
        del tr
        return out
    finally:
        sim.close()


def _check_all(tr, seed, env0):
    """Split the env columns over host threads; returns total mismatches."""
    params = oracle.make_params(**workloads.CARTPOLE)
    n = tr["action"].shape[1]
    bounds = np.linspace(0, n, THREADS + 1).astype(int)

    def one(j):
        a, b = int(bounds[j]), int(bounds[j + 1])
        if a == b:
            return 0, None
        bad, first = oracle.check_rows(params, seed, env0 + a, 0, tr["obs"][:, :, a:b], tr["action"][:, a:b],
                                       tr["reward"][:, a:b], tr["done"][:, a:b])
        return bad, (None if first is None else (first[0], first[1] + a))

    with cf.ThreadPoolExecutor(max_workers=THREADS) as ex:
        res = list(ex.map(one, range(THREADS)))
    total = sum(r[0] for r in res)
    firsts = [r[1] for r in res if r[1] is not None]
    return total, (firsts[0] if firsts else None)


@pytest.mark.parametrize("K", [1000, 1])
def test_k_sweep_workload_every_step(K):
    w = workloads.WORKLOADS[workloads.K_SWEEP]
    tr = _run(w["n"], w["T"], K, w["seed"])
    bad, first = _check_all(tr, w["seed"], 0)
    assert bad == 0, (K, bad, first)
    assert int(tr["done"].astype(bool).sum()) > w["n"]       # many episodes ended and restarted


def test_headline_launch_every_env_every_step():
    """All 4,194,304 x 200 env-steps of the bench's single K = 200 launch,
    checked in sixteen slices of 262,144 environments."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, T = w["n"], w["T"]
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(w["seed"])
        tr = Trajectory(T, n, stats=False)
        sim.step(T, tr.rows(0, T))                     # the bench's single K = 200 launch
        torch.cuda.synchronize()
        S = n // 16
        ends = 0
        for a in range(0, n, S):
            cols = {key: getattr(tr, key)[..., a:a + S].cpu().numpy() for key in ("obs", "action", "reward", "done")}
            bad, first = _check_all(cols, w["seed"], a)
            assert bad == 0, (a, bad, first)
            ends += int(cols["done"].astype(bool).sum())
        assert ends > n * T // 30                      # episodes end about once per 22 steps
        del tr
    finally:
        sim.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_workload_32k_envs_every_step(dtype):
    import policy_bounds
    from gpu_helpers import BF16_P0_MEAN_GATE, BF16_P0_Q9999_GATE, F32_P0_GATE, device_policy

    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.MLP]
    n, T, K, seed = w["n"], w["T"], w["K"][0], w["seed"]
    wts = workloads.mlp_weights(seed)
    S = 8192                                             # envs per slice, four slices
    st, keep = device_policy(wts, dtype)
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(seed)
        tr = Trajectory(T, n, stats=False, p0=True, learner=True)
        for k0 in range(0, T, K):
            sim.step(K, tr.rows(k0, K), policy=st)     # the bench's launch shape
        torch.cuda.synchronize()
        starts = (0, n // 3 + 5, 2 * n // 3, n - S)
        keys = ("obs", "action", "reward", "done", "policy_p0", "logp", "value")
        cols = {key: np.concatenate([getattr(tr, key)[..., a:a + S].cpu().numpy() for a in starts], axis=-1)
                for key in keys}
        del tr
    finally:
        sim.close()
    del keep
    env_ids = np.concatenate([np.arange(a, a + S) for a in starts])
    params = oracle.make_params(**workloads.CARTPOLE)
    pol = oracle.Policy(**wts, bf16=(dtype == "bf16"))
    errs = policy_bounds.errs()

    dp0 = np.zeros((T, 4 * S), dtype=np.float32)          # |p0 - oracle p0| of every checked env-step

    def one(a, b):
        # each column range lies inside one slice of consecutive env ids
        if a == b:
            return None
        assert env_ids[b - 1] - env_ids[a] == b - 1 - a
        c = {key: v[..., a:b] for key, v in cols.items()}
        part = np.zeros((T, b - a), dtype=np.float32)
        bad, first, stats = oracle.check_policy_rows(
            params, pol, seed, int(env_ids[a]), 0, c["obs"], c["action"], c["reward"], c["done"], c["policy_p0"],
            errs, logp=c["logp"], value=c["value"], dp0_out=part)
        dp0[:, a:b] = part
        stats["width_sum"] = stats["mean_width"] * (b - a) * T
        return bad, (None if first is None else (first[0], int(env_ids[a + first[1]]))), stats

    ranges = []
    for j in range(4):                                   # split each slice on its own
        per = max(1, THREADS // 4)
        edges = np.linspace(j * S, (j + 1) * S, per + 1).astype(int)
        ranges += [(int(edges[m]), int(edges[m + 1])) for m in range(per)]
    with cf.ThreadPoolExecutor(max_workers=THREADS) as ex:
        res = [r for r in ex.map(lambda ab: one(*ab), ranges) if r is not None]
    bad = sum(r[0] for r in res)
    firsts = [r[1] for r in res if r[1] is not None]
    worst = max(r[2]["worst"] for r in res)
    exempt = sum(r[2]["exempt"] for r in res)
    max_width = max(r[2]["max_width"] for r in res)
    mean_width = sum(r[2]["width_sum"] for r in res) / (4 * S * T)
    mean_dp0, p9999 = float(dp0.astype(np.float64).mean()), float(np.quantile(dp0, 0.9999))
    print(f"{dtype}: worst |p0 - oracle| {worst:.3g}, mean {mean_dp0:.3g}, 99.99th percentile {p9999:.3g}, "
          f"p0 enclosure width mean {mean_width:.3g} max {max_width:.3g}, "
          f"{exempt} actions differ from the oracle's", flush=True)
    if bad:
        k, env = firsts[0]
        col = int(np.nonzero(env_ids == env)[0][0])
        logit, p_ref, v_ref = pol.eval(cols["obs"][k, :, col])
        enc = pol.bounds(cols["obs"][k, :, col], errs)
        a = int(cols["action"][k, col])
        detail = dict(step=k, env=env, u=float(oracle.policy_u(seed, env, k)), action=a,
                      p0=(float(cols["policy_p0"][k, col]), p_ref), logp=(float(cols["logp"][k, col]),
                                                                        oracle.log_prob(logit, a)),
                      value=(float(cols["value"][k, col]), v_ref), logits=tuple(logit), enclosures=enc)
        raise AssertionError(f"{dtype}: {bad} failing env-steps; first {detail}; firsts {firsts[:4]}")
    assert exempt <= 4 * S * T // 10000, exempt
    if dtype == "f32":
        assert worst <= F32_P0_GATE, worst
    else:
        assert mean_dp0 <= BF16_P0_MEAN_GATE and p9999 <= BF16_P0_Q9999_GATE, (mean_dp0, p9999)
    assert int(cols["done"].astype(bool).sum()) > 0


def test_state_size_workload_every_step():
    """262,144 envs x 500 steps in one K = 500 launch with D = 4,096 padding
    words: every recorded step teacher-forced against the oracle.  The padding
    words never feed back into the cart-pole, so the trajectories of D = 4, 64
    and 512 must equal it bit for bit (compared on the device)."""
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS[workloads.STATE_SWEEP]
    n, T, seed = w["n"], w["T"], w["seed"]
    keys = ("obs", "action", "reward", "done")
    ref = None
    for D in sorted(w["D"], reverse=True):
        sim = Simulator(n, D, workloads.CARTPOLE)
        try:
            sim.reset(seed)
            tr = Trajectory(T, n, stats=False)
            sim.step(T, tr.rows(0, T))
            torch.cuda.synchronize()
            if ref is None:
                ref = {key: getattr(tr, key) for key in keys}
                S = n // 4
                for a in range(0, n, S):
                    cols = {key: ref[key][..., a:a + S].cpu().numpy() for key in keys}
                    bad, first = _check_all(cols, seed, a)
                    assert bad == 0, (D, a, bad, first)
            else:
                for key in keys:
                    assert torch.equal(getattr(tr, key), ref[key]), (D, key)
                del tr
        finally:
            sim.close()
