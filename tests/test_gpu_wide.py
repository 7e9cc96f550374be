"""GPU parity of the wide-padding kernels (the paper's state-size factor S).

Beyond 32 padding words per environment the library switches to the two-phase
kernel (the cart-pole pass leaves action/done bits in LDS, then waves replay
the padding recurrence with the words in registers, pipelined across the
256-env blocks of a persistent workgroup; up to 64 words, one word per lane and
eight environments per step through a jump table); up to 32 words stay in each
thread's registers.  Everything is compared
bit for bit with the oracle: trajectory, block statistics, cart-pole state,
all padding words and episode counters.
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
    import paper_2207_07736_amd  # noqa: F401


# D values cover every kernel shape: register-resident words (<= 32), one word
# per lane for eight envs at a time (33-64), 4/8/16 words per lane (four or two
# envs per scalar decision up to 512 words, one above), ragged rows (D not a
# multiple of 4 or of the chunk) and several 1,024-word chunks per env
# (D > 1,024).
@pytest.mark.parametrize("D", [17, 32, 33, 63, 64, 65, 100, 256, 512, 777, 1024, 2048, 4096, 5000])
def test_wide_padding_bit_exact(D):
    n = 260                                   # two stats blocks, ragged tail
    T = 140 if D > 1024 else 300
    sched = [1, T - 1]
    g = gpu_run(n, T, sched, D=D, seed=7)
    r = oracle_run(n, T, sched, D=D, seed=7)
    assert_bit_equal(g, r)
    for a, b in zip(g["stats"], r["stats"]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("n", [1, 63, 65])
@pytest.mark.parametrize("D", [48, 300, 1100])
def test_wide_tiny_populations(n, D):
    """A grid of one persistent workgroup whose only block is partial (one env,
    a partial wave, a wave and one lane), for the jump-table, 8- and
    16-words-per-lane shapes: trajectory, state, every padding word and the
    statistics row equal the oracle's."""
    T = 300
    sched = [37, T - 37]
    g = gpu_run(n, T, sched, D=D, seed=11)
    r = oracle_run(n, T, sched, D=D, seed=11)
    assert_bit_equal(g, r)
    for a, b in zip(g["stats"], r["stats"]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("D", [20, 64, 512])
def test_wide_long_launch_crosses_chunks(D):
    """K larger than the 512-step LDS round: the padding words are carried over
    between rounds inside one launch."""
    n, T = 300, 1100
    g = gpu_run(n, T, [T], D=D, seed=workloads.PARITY_SEEDS[2])
    r = oracle_run(n, T, [T], D=D, seed=workloads.PARITY_SEEDS[2])
    assert_bit_equal(g, r)


@pytest.mark.parametrize("D", [48, 72, 300, 700, 1100])
def test_wide_pipeline_several_blocks_per_workgroup(D):
    """More 256-env blocks than the persistent grid has workgroups (two per CU
    on 256 CUs): 514 blocks, the last one partial, so workgroup 0 runs blocks 0
    and 512 one after the other, and K = 800 takes two 512-step rounds
    per block, so several items of one block pass through the pipeline; a second
    call of K = 300 follows.  The columns of blocks 0, 256, 512 and the partial
    last one -- the trajectory, the cart-pole state and every padding word --
    and their statistics rows equal the oracle's slices at the same global ids
    (D = 48, 72, 300, 700 and 1,100 take the jump-table, 4-, 8- and
    16-words-per-lane shapes, the last in two 1,024-word chunks)."""
    n = 256 * 513 + 100
    T, sched = 1100, [800, 300]
    slices = [(0, 256), (256 * 256, 256 * 257), (256 * 512, 256 * 513), (256 * 513, n)]
    print(f"wide pipeline D={D} n={n} sched={sched}", flush=True)
    g = gpu_run(n, T, sched, D=D, seed=21, slices=slices)
    refs = [oracle_run(b - a, T, sched, D=D, seed=21, env0=a) for a, b in slices]
    want = {k: np.concatenate([r[k] for r in refs], axis=-1) for k in ("obs", "action", "reward", "done", "state")}
    want["ep"] = np.concatenate([r["ep"] for r in refs])
    want["t"] = refs[0]["t"]
    assert_bit_equal(g, want, keys=("obs", "action", "reward", "done", "state", "ep"))
    for call, gs in enumerate(g["stats"]):
        for (a, b), r in zip(slices, refs):
            rows = r["stats"][call]
            assert np.array_equal(gs[a // 256:a // 256 + len(rows)], rows), (call, a)


@pytest.mark.parametrize("D", [48, 300])
def test_wide_pipeline_without_trajectory(D):
    """The wide kernel's forms without a trajectory, at the multi-block size of
    the test above: a call with traj = NULL and a statistics-only call leave the
    same state as the recording call, the statistics equal the recording call's,
    and both match the oracle's slices of the first block, of block 512 (the
    second block of workgroup 0 on the two-per-CU grid) and of the last block."""
    from paper_2207_07736_amd import Simulator, Trajectory, stats_only
    n, T, seed = 256 * 513 + 100, 700, 23
    states, stats = [], []
    for form in ("traj", "none", "stats"):
        sim = Simulator(n, D, workloads.CARTPOLE)
        try:
            sim.reset(seed)
            if form == "traj":
                tr = Trajectory(T, n)
                sim.step(T, tr.rows(0, T))
                stats.append(tr.block_stats.clone())
                del tr
            elif form == "none":
                sim.step(T, None)
            else:
                st = torch.zeros(((n + 255) // 256, 4), dtype=torch.int32, device="cuda")
                sim.step(T, stats_only(st, n))
                stats.append(st)
            torch.cuda.synchronize()
            states.append(sim.get_state())
        finally:
            sim.close()
    for st, ep, t in states[1:]:
        assert np.array_equal(st.view(np.uint32), states[0][0].view(np.uint32))
        assert np.array_equal(ep, states[0][1]) and t == T
    assert torch.equal(stats[0], stats[1])
    for a, b in ((0, 256), (256 * 512, 256 * 513), (256 * 513, n)):
        r = oracle_run(b - a, T, [T], D=D, seed=seed, env0=a)
        assert np.array_equal(states[0][0][:, a:b].view(np.uint32), r["state"].view(np.uint32))
        assert np.array_equal(stats[1].cpu().numpy().view(np.uint32)[a // 256:a // 256 + len(r["stats"][0])],
                              r["stats"][0])


def test_wide_edge_configs():
    cfg = workloads.cartpole(max_episode_steps=7, no_termination=1)
    g = gpu_run(200, 60, [13, 47], D=70, seed=1, cfg=cfg)
    r = oracle_run(200, 60, [13, 47], D=70, seed=1, cfg=cfg)
    assert_bit_equal(g, r)


def test_wide_set_state_round_trip():
    from paper_2207_07736_amd import Simulator
    n, D = 333, 130
    sim = Simulator(n, D, workloads.CARTPOLE)
    try:
        sim.reset(3)
        sim.step(20)
        st, ep, t = sim.get_state()
        rng = np.random.Generator(np.random.PCG64(0))
        st2 = rng.standard_normal(st.shape).astype(np.float32)
        sim.set_state(st2, ep, t)
        back, ep2, t2 = sim.get_state()
        assert np.array_equal(back.view(np.uint32), st2.view(np.uint32)) and np.array_equal(ep2, ep) and t2 == t
    finally:
        sim.close()


@pytest.mark.parametrize("D", workloads.WORKLOADS[workloads.STATE_SWEEP]["D"])
def test_state_size_workload_fused_equals_unfused(D):
    """262,144 envs x 500 steps: one K=500 launch equals 500 K=1 launches bit for
    bit (trajectory on sampled slices, the full final state), and the sampled
    slices equal the oracle."""
    w = workloads.WORKLOADS[workloads.STATE_SWEEP]
    n, T = w["n"], w["T"]
    slices = [(0, 256), (n - 256, n)]
    fused = gpu_run(n, T, [T], D=D, seed=w["seed"], slices=slices)
    unfused = gpu_run(n, T, [1] * T, D=D, seed=w["seed"], slices=slices)
    assert_bit_equal(fused, unfused)
    ref = [oracle_run(b - a, T, [T], D=D, seed=w["seed"], env0=a) for a, b in slices]
    merged = {key: np.concatenate([x[key] for x in ref], axis=-1) for key in ("obs", "action", "reward", "done", "state")}
    merged["ep"] = np.concatenate([x["ep"] for x in ref])
    merged["t"] = T
    assert_bit_equal(fused, merged)
