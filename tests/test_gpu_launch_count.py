"""One kernel launch per rlsim_step_fused call, whatever K is (the fused
design's defining property), and the launch counts of rlsim_reset.

Each call is recorded with the HIP runtime's stream capture on the handle's
stream, and the captured graph's nodes are counted and typed (nothing is
replayed).  The graph holds exactly what the call enqueued."""
import ctypes

import pytest

import workloads

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

HIP_CAPTURE_RELAXED = 2
HIP_NODE_KERNEL = 0


@pytest.fixture(scope="module")
def hip():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2207_07736_amd  # noqa: F401
    torch.cuda.init()
    L = ctypes.CDLL("libamdhip64.so.7")      # the runtime torch and librlsim already share
    vp = ctypes.c_void_p
    L.hipStreamBeginCapture.argtypes = [vp, ctypes.c_int]
    L.hipStreamEndCapture.argtypes = [vp, ctypes.POINTER(vp)]
    L.hipGraphGetNodes.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_size_t)]
    L.hipGraphNodeGetType.argtypes = [vp, ctypes.POINTER(ctypes.c_int)]
    L.hipGraphDestroy.argtypes = [vp]
    return L


def _captured_node_types(hip, stream, fn):
    s = ctypes.c_void_p(stream.cuda_stream)
    assert hip.hipStreamBeginCapture(s, HIP_CAPTURE_RELAXED) == 0
    g = ctypes.c_void_p()
    try:
        fn()
    finally:
        rc = hip.hipStreamEndCapture(s, ctypes.byref(g))
    assert rc == 0
    try:
        n = ctypes.c_size_t(0)
        assert hip.hipGraphGetNodes(g, None, ctypes.byref(n)) == 0
        nodes = (ctypes.c_void_p * max(n.value, 1))()
        assert hip.hipGraphGetNodes(g, ctypes.cast(nodes, ctypes.c_void_p), ctypes.byref(n)) == 0
        types = []
        for i in range(n.value):
            t = ctypes.c_int(-1)
            assert hip.hipGraphNodeGetType(ctypes.c_void_p(nodes[i]), ctypes.byref(t)) == 0
            types.append(t.value)
        return types
    finally:
        hip.hipGraphDestroy(g)


@pytest.mark.parametrize("D", [0, 3, 8, 20, 40])
def test_one_launch_per_step_call(hip, D):
    from paper_2207_07736_amd import Simulator, Trajectory
    s = torch.cuda.Stream()
    n = 5000
    sim = Simulator(n, D, workloads.CARTPOLE, stream=s)
    try:
        sim.reset(1)
        tr = Trajectory(1000, n)
        torch.cuda.synchronize()
        for K in (1, 7, 200, 1000):
            types = _captured_node_types(hip, s, lambda: sim.step(K, tr.rows(0, K)))
            assert types == [HIP_NODE_KERNEL], (D, K, types)
        types = _captured_node_types(hip, s, lambda: sim.step(300, None))
        assert types == [HIP_NODE_KERNEL]
        # reset: the initial state, plus the padding parameters when D > 0
        types = _captured_node_types(hip, s, lambda: sim.reset(2))
        assert types == [HIP_NODE_KERNEL] * (2 if D else 1)
        del tr
    finally:
        sim.close()


def test_one_launch_per_policy_step_call(hip):
    import numpy as np
    from paper_2207_07736_amd import RLSIM_F32, Simulator, Trajectory, policy_struct
    w = workloads.mlp_weights(0)
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in w.items()}
    pol = policy_struct(RLSIM_F32, dev["w1"], dev["b1"], dev["w2"], dev["b2"], dev["w3"], dev["b3"],
                        dev["wv"], dev["bv"])
    s = torch.cuda.Stream()
    sim = Simulator(3000, 0, workloads.CARTPOLE, stream=s)
    try:
        sim.reset(0)
        tr = Trajectory(64, 3000, p0=True, learner=True)
        torch.cuda.synchronize()
        for K in (1, 16, 64):
            types = _captured_node_types(hip, s, lambda: sim.step(K, tr.rows(0, K), policy=pol))
            assert types == [HIP_NODE_KERNEL], (K, types)
        del tr
    finally:
        sim.close()
    del dev


@pytest.mark.parametrize("N", [1, 4])
def test_one_launch_per_chain_step_call(hip, N):
    """The chain model: one launch per call for K below and above the
    warp-specialised kernel's threshold, with and without a trajectory."""
    from paper_2207_07736_amd import Simulator, Trajectory
    s = torch.cuda.Stream()
    n = 3000
    sim = Simulator(n, 0, workloads.CARTPOLE, stream=s, links=N)
    try:
        sim.reset(1)
        tr = Trajectory(300, n, S=sim.S)
        torch.cuda.synchronize()
        for K in (1, 15, 16, 300):
            types = _captured_node_types(hip, s, lambda: sim.step(K, tr.rows(0, K)))
            assert types == [HIP_NODE_KERNEL], (N, K, types)
        types = _captured_node_types(hip, s, lambda: sim.step(300, None))
        assert types == [HIP_NODE_KERNEL]
        types = _captured_node_types(hip, s, lambda: sim.reset(2))
        assert types == [HIP_NODE_KERNEL]
        del tr
    finally:
        sim.close()
