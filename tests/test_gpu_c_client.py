"""The C ABI from plain C: tests/c_client/rlsim_client.c creates a handle,
resets it, runs one fused launch with a trajectory in hipMalloc'd buffers and
reads the state back, with no Python or torch in the process.  Its output must
equal the oracle bit for bit; it also checks two error statuses and messages."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c_client", "rlsim_client")


def _ensure_built():
    if not os.path.exists(EXE):
        import sys
        sys.path.insert(0, os.path.join(HERE, "c_client"))
        import build_client
        build_client.build()


def test_client_builds_links_and_rejects_a_bad_command_line():
    _ensure_built()
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=60)      # no device call
    assert r.returncode == 1 and "usage" in r.stderr


@pytest.mark.gpu
@pytest.mark.parametrize("n,K,seed", [(1000, 50, (1 << 40) + 7), (70000, 13, 3)])
def test_c_client_run_matches_oracle(tmp_path, n, K, seed):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _ensure_built()                 # normally built by __graft_entry__.build(); gcc takes well under a second
    out = tmp_path / "run.bin"
    r = subprocess.run([EXE, str(n), str(K), str(seed), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    buf = out.read_bytes()
    sizes = [("obs", np.float32, K * 4 * n), ("action", np.uint8, K * n), ("reward", np.float32, K * n),
             ("done", np.uint8, K * n), ("state", np.float32, 4 * n), ("ep", np.uint32, n), ("t", np.uint64, 1)]
    got, off = {}, 0
    for name, dt, count in sizes:
        nbytes = np.dtype(dt).itemsize * count
        got[name] = np.frombuffer(buf, dtype=dt, count=count, offset=off)
        off += nbytes
    assert off == len(buf)
    sim = oracle.Sim(n, 0, oracle.make_params(**workloads.CARTPOLE))
    sim.reset(seed)
    want = sim.step(K, stats=False)
    st, ep, t = sim.get_state()
    for name in ("obs", "action", "reward", "done"):
        assert np.array_equal(got[name].view(np.uint8), np.ascontiguousarray(want[name]).reshape(-1).view(np.uint8)), name
    assert np.array_equal(got["state"].view(np.uint32), st.reshape(-1).view(np.uint32))
    assert np.array_equal(got["ep"], ep) and int(got["t"][0]) == t == K
