"""Every recorded step of large GPU runs, teacher-forced against the oracle.

From the GPU's own obs at step t, the oracle (orc_check_rows) recomputes the
random action bit, the simulation step, the done byte (episode lengths tracked
from the reset) and the next row -- the reset draw after an episode end -- and
requires the recorded row to match bit for bit, for every environment and every
step: the whole 65,536-env x 1,000-step workload in its fused and unfused forms,
and a quarter of a million environments of the 4,194,304-env headline launch."""
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
    w = workloads.WORKLOADS["C2"]
    tr = _run(w["n"], w["T"], K, w["seed"])
    bad, first = _check_all(tr, w["seed"], 0)
    assert bad == 0, (K, bad, first)
    assert int(tr["done"].astype(bool).sum()) > w["n"]       # many episodes ended and restarted


def test_headline_launch_quarter_million_envs_every_step():
    from paper_2207_07736_amd import Simulator, Trajectory
    w = workloads.WORKLOADS["C3"]
    n, T = w["n"], w["T"]
    sim = Simulator(n, 0, workloads.CARTPOLE)
    try:
        sim.reset(w["seed"])
        tr = Trajectory(T, n, stats=False)
        sim.step(T, tr.rows(0, T))                     # the bench's single K = 200 launch
        torch.cuda.synchronize()
        for a in (0, n // 3, 2 * n // 3 + 17, n - 65536):
            cols = {key: getattr(tr, key)[..., a:a + 65536].cpu().numpy() for key in ("obs", "action", "reward", "done")}
            bad, first = _check_all(cols, w["seed"], a)
            assert bad == 0, (a, bad, first)
        del tr
    finally:
        sim.close()
