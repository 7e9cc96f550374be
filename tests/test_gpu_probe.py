"""The store-only probe (include/rlsim_probe.h) writes every byte it claims,
in the trajectory layout, at a ragged size and at the headline size the bench
times it at (4,194,304 envs x 200 rows), checked in full on the device."""
import pytest

import workloads

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _expected_ok(tr, n, K):
    e = torch.arange(n, device="cuda", dtype=torch.int64)
    k = torch.arange(K, device="cuda", dtype=torch.int64)[:, None]
    base = ((e & 0xFFFF)[None, :] + k).to(torch.float32)              # [K][n], exact
    for c in range(4):
        if not torch.equal(tr.obs[:, c, :], base + float(c)):
            return f"obs component {c}"
    if not torch.equal(tr.action, ((e[None, :] + k) & 1).to(torch.uint8)):
        return "action"
    if not bool((tr.reward == 1.0).all()):
        return "reward"
    if not torch.equal(tr.done, ((e[None, :] ^ k) & 3).to(torch.uint8)):
        return "done"
    return None


@pytest.mark.parametrize("n,K", [(1, 3), (1000, 7), (70000, 33)])
def test_probe_values_ragged(n, K):
    from paper_2207_07736_amd import Trajectory
    from paper_2207_07736_amd.probe import probe_store
    tr = Trajectory(K, n, stats=False)
    for t in (tr.obs, tr.reward):
        t.fill_(float("nan"))
    tr.action.fill_(7)
    tr.done.fill_(7)
    probe_store(n, K, tr.obs, tr.action, tr.reward, tr.done)
    torch.cuda.synchronize()
    assert _expected_ok(tr, n, K) is None


def test_probe_headline_size():
    from paper_2207_07736_amd import Trajectory
    from paper_2207_07736_amd.probe import probe_store
    w = workloads.WORKLOADS[workloads.HEADLINE]
    n, K = w["n"], w["T"]
    tr = Trajectory(K, n, stats=False)
    tr.done.fill_(9)
    s = torch.cuda.Stream()
    probe_store(n, K, tr.obs, tr.action, tr.reward, tr.done, stream=s)
    torch.cuda.synchronize()
    assert _expected_ok(tr, n, K) is None
    del tr


def test_stream_probe_values():
    """rlsim_probe_stream computes s <- fma(a, s, b) on every word.  Small
    integers over 16 keep a * s + b exact in double, so the fp32 result must be
    that value rounded once."""
    import numpy as np
    from paper_2207_07736_amd.probe import probe_stream
    rng = np.random.Generator(np.random.PCG64(3))
    n = 4 * 70001
    s, a, b = (rng.integers(-1000, 1001, size=n).astype(np.float32) / np.float32(16) for _ in range(3))
    want = (a.astype(np.float64) * s + b).astype(np.float32)
    ts, ta, tb = (torch.from_numpy(x).cuda() for x in (s, a, b))
    probe_stream(ts, ta, tb)
    torch.cuda.synchronize()
    assert np.array_equal(ts.cpu().numpy().view(np.uint32), want.view(np.uint32))
    assert np.array_equal(ta.cpu().numpy(), a) and np.array_equal(tb.cpu().numpy(), b)


@pytest.mark.parametrize("per", [1, 4, 275])
def test_fill_probe_values(per):
    """rlsim_probe_fill writes float4 i as (v, v + 1, v + 2, v + 3), v = i mod
    2^20, at every index of a buffer whose size is no multiple of a
    workgroup's chunk, and nothing past it."""
    import numpy as np
    from paper_2207_07736_amd.probe import probe_fill
    n4 = 3 * 256 * 275 + 1234
    buf = torch.full((4 * n4 + 64,), -7.0, dtype=torch.float32, device="cuda")
    probe_fill(buf[:4 * n4], per)
    torch.cuda.synchronize()
    got = buf.cpu().numpy()
    v = (np.arange(n4, dtype=np.int64) & 0xFFFFF).astype(np.float32)
    want = np.stack([v, v + 1, v + 2, v + 3], axis=1).reshape(-1)
    assert np.array_equal(got[:4 * n4], want)
    assert np.all(got[4 * n4:] == -7.0)


def _hash32(x: int) -> int:
    m = 0xFFFFFFFF
    x ^= x >> 16
    x = (x * 0x7FEB352D) & m
    x ^= x >> 15
    x = (x * 0x846CA68B) & m
    x ^= x >> 16
    return x


def _replay_tree_want(blocks: int, iters: int):
    """Closed form of the replay kind: per wave, 8 x (the count of action-1
    steps since each environment's last done bit), from the bit recipe of
    include/rlsim_probe.h."""
    import numpy as np
    want = np.zeros((blocks, 4, 64))
    for g in range(blocks * 4):
        cnt = [0, 0]
        for w in range(iters):
            k = (g * iters + w) & 0xFFFFFFFF
            u = [_hash32((4 * k) & 0xFFFFFFFF), _hash32((4 * k + 1) & 0xFFFFFFFF)]
            h = _hash32((4 * k + 2) & 0xFFFFFFFF)
            d = [(1 << (h & 31)) | ((1 << ((h >> 8) & 31)) if (h >> 5) % 3 == 0 else 0),
                 (1 << ((h >> 13) & 31)) | ((1 << ((h >> 21) & 31)) if (h >> 18) % 3 == 0 else 0)]
            for t in range(32):
                for e in range(2):
                    if (u[e] >> t) & 1:
                        cnt[e] += 1
                    if (d[e] >> t) & 1:
                        cnt[e] = 0
        want[g // 4, g % 4, :] = 8 * (cnt[0] + cnt[1])
    return want


@pytest.mark.parametrize("kind", ["fma", "select_fma", "exp", "rcp", "mfma", "mixed", "mul", "fma_shared",
                                  "replay_tree", "replay_flat"])
def test_issue_probe_values(kind):
    """rlsim_probe_issue runs the instruction chains it claims: every thread's
    sum of chain results equals the closed form of its kind (exact integers for
    the FMA, select, MFMA and replay chains and the rcp cycle; the fixed point
    of x = 2^-x for exp, to the hardware exp2's accuracy), and each
    workgroup's clock record puts its shader clock between 0.3 and 3.5 GHz."""
    import math

    import numpy as np
    from paper_2207_07736_amd.probe import probe_issue, wall_clock_khz
    blocks, iters = 3, 101
    out = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda")
    clocks = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    probe_issue(kind, blocks, iters, out, clocks=clocks)
    torch.cuda.synchronize()
    c = clocks.cpu().numpy().reshape(blocks, 2)
    assert np.all(c > 0)
    ghz = c[:, 0] / c[:, 1] * wall_clock_khz() * 1e-6
    assert np.all((ghz > 0.3) & (ghz < 3.5)), ghz
    got = out.cpu().numpy().reshape(blocks, 4, 64)
    lane = np.arange(64)
    fma = np.sum([lane + j + iters for j in range(8)], axis=0).astype(np.float64)
    if kind in ("fma", "fma_shared"):
        want = np.broadcast_to(fma, got.shape)
    elif kind == "mul":
        want = np.broadcast_to(np.sum([lane + j for j in range(8)], axis=0).astype(np.float64), got.shape)
    elif kind == "select_fma":
        odd_steps = np.where(lane % 2 == 0, iters // 2, (iters + 1) // 2)
        want = np.broadcast_to(np.sum([j + odd_steps for j in range(8)], axis=0), got.shape)
    elif kind == "rcp":
        want = np.full(got.shape, sum(2.0**-j for j in range(8)))          # odd iteration count: reciprocals
    elif kind == "mfma":
        want = np.full(got.shape, 8.0 * iters)
    elif kind == "replay_tree":
        want = _replay_tree_want(blocks, iters)
        assert np.any(want != want.flat[0])                             # the bits differ between waves
    elif kind == "replay_flat":
        want = np.full(got.shape, 8.0 * 32 * iters)
    elif kind == "mixed":
        b = np.arange(blocks)[:, None, None]
        w = np.arange(4)[None, :, None]
        fma16 = np.sum([lane + j + 16 * iters for j in range(8)], axis=0)
        want = np.where((b + w) % 2 == 1, fma16[None, None, :], 8.0 * iters)
    else:
        root = 0.5
        for _ in range(200):
            root = 2.0 ** -root
        assert abs(root - 0.6411857445) < 1e-9
        assert np.all(np.abs(got - 8 * root) < 8 * 2e-6), got.min()
        return
    assert np.array_equal(got.astype(np.float64), want), (kind, got[0, 0, :4], np.asarray(want)[0, 0, :4])
    assert not math.isnan(float(got.sum()))


def test_issue_probe_rejects_bad_arguments():
    from paper_2207_07736_amd.probe import probe_issue
    out = torch.zeros(256, dtype=torch.float32, device="cuda")
    for kind, blocks, iters in (("fma", 0, 1), ("fma", 1, 0), ("mixed", 1, (1 << 19) + 1), ("fma", 1, (1 << 22) + 1),
                                ("replay_tree", 1, (1 << 16) + 1)):
        with pytest.raises(ValueError):
            probe_issue(kind, blocks, iters, out)
    with pytest.raises(ValueError):
        probe_issue("fma", 2, 1, out)                                        # out too small
