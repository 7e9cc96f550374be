"""Randomised GPU parity: seeded draws of environment count, padding words, K
schedule, seed and simulator constants, each run compared with the oracle bit
for bit (trajectory, statistics, final state, counters).  The draws are fixed by
the test's own generator seed, so every run checks the same cases.  The
RLSIM_RANDOM_CASES environment variable raises the case count for a longer
campaign (default 96)."""
import os

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
    import paper_2207_07736_amd  # noqa: F401


def _case(i):
    rng = np.random.Generator(np.random.PCG64(1000 + i))
    n = int(rng.choice([1, 63, 64, 65, 255, 256, 257, 511, 777, 1024, 1500, 2049]))
    D = int(rng.choice([0, 0, 1, 3, 8, 16, 17, 40, 64, 65, 130, 300]))
    T = int(rng.integers(1, 161))
    cuts = sorted(set(int(c) for c in rng.integers(1, T, size=int(rng.integers(0, 4)))) if T > 1 else [])
    bounds = [0] + cuts + [T]
    sched = [b - a for a, b in zip(bounds[:-1], bounds[1:])]
    seed = int(rng.integers(0, 2**63))
    over = {}
    if rng.random() < 0.4:
        over["max_episode_steps"] = int(rng.choice([0, 1, 2, 7, 30]))
    if rng.random() < 0.3:
        over["x_threshold"] = float(np.float32(rng.uniform(0.05, 2.4)))
    if rng.random() < 0.3:
        over["force_mag"] = float(np.float32(rng.uniform(0.0, 30.0)))
    if rng.random() < 0.2:
        over["compute_factor"] = int(rng.choice([2, 3, 5]))
    if rng.random() < 0.2:
        over["reset_low"], over["reset_high"] = -0.2, 0.2
    if rng.random() < 0.25:
        over["gravity"] = float(np.float32(rng.uniform(0.0, 20.0)))
        over["masspole"] = float(np.float32(rng.uniform(0.01, 1.0)))
        over["half_length"] = float(np.float32(rng.uniform(0.1, 2.0)))
        over["tau"] = float(np.float32(rng.uniform(0.001, 0.05)))
    if over.get("max_episode_steps") == 0 and rng.random() < 0.5:
        over["no_termination"] = 1
    return n, D, T, sched, seed, over


@pytest.mark.parametrize("i", range(int(os.environ.get("RLSIM_RANDOM_CASES", "96"))))
def test_random_case_bit_exact(i):
    n, D, T, sched, seed, over = _case(i)
    cfg = workloads.cartpole(**over)
    print(f"case {i}: n={n} D={D} T={T} sched={sched} seed={seed} cfg={over}", flush=True)
    g = gpu_run(n, T, sched, D=D, seed=seed, cfg=cfg)
    r = oracle_run(n, T, sched, D=D, seed=seed, cfg=cfg)
    assert_bit_equal(g, r)
    assert len(g["stats"]) == len(r["stats"])
    for a, b in zip(g["stats"], r["stats"]):
        assert np.array_equal(a, b)
