"""K unfused launches captured in a HIP graph (the decomposition of the fusion
speedup into launch overhead and register residency).

rlsim_step_fused issues exactly one kernel launch and no memset or allocation,
so a sequence of calls on a capturing stream records one kernel node per call.
Every replay is checked against the eager run, with eager work (a reset) and a
synchronisation between replays.
"""
import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401


@pytest.mark.parametrize("D", [0, 5, 40])
def test_graph_of_unfused_launches_matches_eager(D):
    from paper_2207_07736_amd import Simulator, Trajectory
    n, T, seed = 3000, 60, 4
    s = torch.cuda.Stream()
    sim = Simulator(n, D, workloads.CARTPOLE, stream=s)
    try:
        tr = Trajectory(T, n)
        rows = [tr.rows(k, 1) for k in range(T)]
        with torch.cuda.stream(s):
            # eager reference
            sim.reset(seed)
            for k in range(T):
                sim.step(1, rows[k])
            s.synchronize()
            ref = {k: getattr(tr, k).clone() for k in ("obs", "action", "reward", "done")}
            ref_state = sim.get_state()
            # capture the same T launches (t = 0 .. T-1 are baked into the nodes)
            sim.reset(seed)
            s.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                for k in range(T):
                    sim.step(1, rows[k])
            for rep in range(3):
                for k in ("obs", "action", "reward", "done"):
                    getattr(tr, k).zero_()
                sim.reset(seed)                 # eager work between replays
                s.synchronize()
                g.replay()
                s.synchronize()
                for k in ("obs", "action", "reward", "done"):
                    assert torch.equal(getattr(tr, k), ref[k]), (rep, k)
                st, ep, _ = sim.get_state()
                assert np.array_equal(st.view(np.uint32), ref_state[0].view(np.uint32)) and np.array_equal(ep, ref_state[1])
        del g, tr
    finally:
        sim.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_graph_of_policy_launches_matches_eager(dtype):
    """The MLP-policy kernel in a graph: 8 launches of K = 4 with p0, log pi and
    value recorded, replayed three times; every output plane equals the eager
    run bit for bit."""
    from gpu_helpers import device_policy, policy_weights

    from paper_2207_07736_amd import Simulator, Trajectory
    n, T, K, seed = 2000, 32, 4, 6
    st, keep = device_policy(policy_weights(21, 0.2), dtype)
    s = torch.cuda.Stream()
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=s)
    planes = ("obs", "action", "reward", "done", "policy_p0", "logp", "value")
    try:
        tr = Trajectory(T, n, p0=True, learner=True)
        rows = [tr.rows(k0, K) for k0 in range(0, T, K)]
        with torch.cuda.stream(s):
            sim.reset(seed)
            for r in rows:
                sim.step(K, r, policy=st)
            s.synchronize()
            ref = {k: getattr(tr, k).clone() for k in planes}
            ref_state = sim.get_state()
            sim.reset(seed)
            s.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                for r in rows:
                    sim.step(K, r, policy=st)
            for rep in range(3):
                for k in planes:
                    getattr(tr, k).zero_()
                sim.reset(seed)
                s.synchronize()
                g.replay()
                s.synchronize()
                for k in planes:
                    assert torch.equal(getattr(tr, k), ref[k]), (rep, k)
                st_, ep, _ = sim.get_state()
                assert np.array_equal(st_.view(np.uint32), ref_state[0].view(np.uint32))
                assert np.array_equal(ep, ref_state[1])
        del g, tr
    finally:
        sim.close()
    del keep
