"""Proof that no cart-pole episode of the default configuration ends before
its eighth step (CPU only).

The reset draws are keyed by the 8-step block of the step an episode begins
at, so two episodes of one environment share an initial state only if one of
them lasts fewer than 8 steps.  This test shows that none does, for every
initial state in the reset box [-0.05, 0.05]^4 and every one of the 2^7 action
sequences: the fp32 operation sequence of seven steps is evaluated in interval
arithmetic that encloses fp32 rounding (tests/interval_fp32.py), over a
subdivision of the box refined where an enclosure is too wide, and after every
step the enclosure must lie within both thresholds.  The enclosure itself is
checked against the oracle at sampled points."""
import math

import numpy as np

import oracle
import workloads
from interval_fp32 import Iv, fma

F32 = np.float32
C = workloads.CARTPOLE


def _consts():
    mc, mp, hl = F32(C["masscart"]), F32(C["masspole"]), F32(C["half_length"])
    total = F32(mc + mp)
    pole_ml = F32(mp * hl)
    inv_total = F32(F32(1.0) / total)
    return dict(g=F32(C["gravity"]), hl=hl, fm=F32(C["force_mag"]), tau=F32(C["tau"]), pole_ml=pole_ml,
                inv_total=inv_total, m_over_M=F32(mp * inv_total), ml_over_M=F32(pole_ml * inv_total),
                c43=F32(F32(4.0) / F32(3.0)))


K = _consts()
S3, S5, S7, S9 = (F32(v) for v in (-1.0 / 6.0, 1.0 / 120.0, -1.0 / 5040.0, 1.0 / 362880.0))
C2, C4, C6, C8 = (F32(v) for v in (-0.5, 1.0 / 24.0, -1.0 / 720.0, 1.0 / 40320.0))


def _sincos(th):
    z = th.square()
    q = fma(S9, z, S7)
    q = fma(q, z, S5)
    q = fma(q, z, S3)
    s = fma(th * z, q, th)
    q = fma(C8, z, C6)
    q = fma(q, z, C4)
    q = fma(q, z, C2)
    c = fma(z, q, F32(1.0))
    return s, c


def _step(st, force):
    """The cart-pole step's fp32 operation sequence on intervals; the angle
    must lie within pi/4, where sin/cos are the series alone."""
    x, xd, th, thd = st
    assert np.all(th.abs_max() <= math.pi / 4)
    sn, cs = _sincos(th)
    ml_thd2 = thd.square() * K["pole_ml"]
    temp = fma(ml_thd2, sn, force) * K["inv_total"]
    num = fma(-cs, temp, sn * K["g"])
    den = fma(Iv(-np.float64(K["m_over_M"])), cs.square(), K["c43"]) * K["hl"]
    thacc = num / den
    xacc = fma(-(thacc * K["ml_over_M"]), cs, temp)
    tau = K["tau"]
    return [fma(tau, xd, x), fma(tau, xacc, xd), fma(tau, thd, th), fma(tau, thacc, thd)]


def _survives(lo, hi, steps=7):
    """For boxes [lo, hi] (B x 4), whether every action sequence of `steps`
    steps keeps the state inside both thresholds after each step."""
    thr_x, thr_th = np.float64(F32(C["x_threshold"])), np.float64(F32(C["theta_threshold_rad"]))
    B = lo.shape[0]
    owner = np.arange(B)
    st = [Iv(lo[:, c], hi[:, c]) for c in range(4)]
    ok = np.ones(B, dtype=bool)
    for _ in range(steps):
        nxt = []
        for a in (0, 1):
            force = K["fm"] if a else -K["fm"]
            nxt.append(_step(st, force))
        st = [Iv(np.concatenate([nxt[0][c].lo, nxt[1][c].lo]), np.concatenate([nxt[0][c].hi, nxt[1][c].hi]))
              for c in range(4)]
        owner = np.concatenate([owner, owner])
        inside = (st[0].abs_max() <= thr_x) & (st[2].abs_max() <= thr_th)
        np.logical_and.at(ok, owner, inside)
    return ok


def test_no_episode_shorter_than_eight_steps_over_the_whole_reset_box():
    lo0 = np.float64(F32(C["reset_low"]))
    hi0 = np.float64(F32(C["reset_high"]))
    n0 = 4
    edges = np.linspace(lo0, hi0, n0 + 1)
    grid = np.stack(np.meshgrid(*[np.arange(n0)] * 4, indexing="ij"), axis=-1).reshape(-1, 4)
    lo, hi = edges[grid], edges[grid + 1]
    proven, rounds = 0.0, 0
    while len(lo):
        rounds += 1
        assert rounds <= 12 and len(lo) <= 200000, (rounds, len(lo))
        ok = _survives(lo, hi)
        proven += float(np.prod(hi[ok] - lo[ok], axis=1).sum())
        lo, hi = lo[~ok], hi[~ok]
        if len(lo):                                  # bisect the failing boxes along their widest side
            d = np.argmax(hi - lo, axis=1)
            mid = 0.5 * (lo[np.arange(len(lo)), d] + hi[np.arange(len(lo)), d])
            lo2, hi2 = lo.copy(), hi.copy()
            hi[np.arange(len(lo)), d] = mid
            lo2[np.arange(len(lo)), d] = mid
            lo, hi = np.concatenate([lo, lo2]), np.concatenate([hi, hi2])
    assert abs(proven - (hi0 - lo0) ** 4) <= 1e-12 * (hi0 - lo0) ** 4
    # the same machinery cannot prove the false claim for eight steps: the
    # corner that falls fastest does end an episode at step 8
    corner = np.array([[0.04, 0.04, 0.04, 0.04]]), np.array([[hi0, hi0, hi0, hi0]])
    assert not _survives(*corner, steps=8).any()


def test_the_bound_is_tight_and_the_enclosure_holds():
    """Eight steps can end an episode (so the bound cannot be raised), and the
    oracle's fp32 steps at sampled points stay inside the enclosures."""
    P = oracle.make_params(**C)
    s = np.array([0.0, 0.05, 0.05, 0.05], dtype=np.float32)
    for _ in range(7):
        s = oracle.cartpole_step(P, s, 0)
        assert not oracle.terminated(P, s)
    assert oracle.terminated(P, oracle.cartpole_step(P, s, 0))
    rng = np.random.Generator(np.random.PCG64(17))
    lo = np.array([-0.05, -0.05, 0.0, 0.01])
    hi = np.array([-0.04, -0.02, 0.02, 0.05])
    for _ in range(200):
        acts = rng.integers(0, 2, size=7)
        p = rng.uniform(lo, hi).astype(np.float32)
        st = [Iv(lo[c], hi[c]) for c in range(4)]
        for a in acts:
            st = _step(st, K["fm"] if a else -K["fm"])
            p = oracle.cartpole_step(P, p, int(a))
            for c in range(4):
                assert st[c].contains(p[c]).all(), (c, p, st[c].lo, st[c].hi)
