"""Seeded synthetic workloads shared by the tests, the smoke check and the bench.

This module holds inputs only -- simulator constants, workload shapes and MLP
weights drawn from a seed -- and none of the method's arithmetic.  Both the GPU
library (through its Python binding) and the CPU oracle receive exactly these
values; neither imports the other.

The paper runs cart-pole (Background, "Cartpole Simulator") with N parallel
simulators and K fused steps (Simulator Kernel Fusion) and scales the state by
a factor S (Simulator Complexity).  It publishes no dataset, trained weights or
constants, so all inputs here are synthetic; the five workloads below give the
shapes, and the simulator's own Philox streams generate every state and action
on the device from the seed.
"""
from __future__ import annotations

import math

import numpy as np

# Cart-pole constants (classic cart-pole benchmark values; the paper cites the
# simulator but prints none).  Threshold angle = 12 degrees rounded to fp32.
CARTPOLE = dict(
    gravity=9.8,
    masscart=1.0,
    masspole=0.1,
    half_length=0.5,
    force_mag=10.0,
    tau=0.02,
    x_threshold=2.4,
    theta_threshold_rad=float(np.float32(12.0 * 2.0 * math.pi / 360.0)),
    max_episode_steps=500,
    reset_low=-0.05,
    reset_high=0.05,
    pad_a_low=0.9,
    pad_a_high=0.99,
    pad_b_low=-1.0,
    pad_b_high=1.0,
    no_termination=0,
    compute_factor=1,
)


def cartpole(**overrides) -> dict:
    """The cart-pole constants with some fields replaced."""
    d = dict(CARTPOLE)
    for k, v in overrides.items():
        if k not in d:
            raise KeyError(k)
        d[k] = v
    return d


# The five workloads, keyed by name.  n: environments, T: steps per run, K:
# fused steps per launch (several values = a sweep), D: padding words per
# environment.
SMALL = "cartpole-1k-100-K1"              # correctness size, launch-bound
K_SWEEP = "cartpole-64k-1000-Ksweep"      # fused steps per launch 1 .. 1,000
HEADLINE = "cartpole-4M-200-K200"         # 4,194,304 envs x 200 steps in one launch
STATE_SWEEP = "cartpole-256k-500-Dsweep"  # padding words D = 4 .. 4,096
MLP = "cartpole-1M-256-K16-mlp"           # the fused MLP policy, fp32 and bf16
WORKLOADS = {
    SMALL: dict(name=SMALL, n=1024, T=100, K=[1], D=[0], seed=0, policy=None),
    K_SWEEP: dict(name=K_SWEEP, n=65536, T=1000, K=[1, 10, 100, 1000], D=[0], seed=0, policy=None),
    HEADLINE: dict(name=HEADLINE, n=4194304, T=200, K=[200], D=[0], seed=0, policy=None),
    STATE_SWEEP: dict(name=STATE_SWEEP, n=262144, T=500, K=[1, 500], D=[4, 64, 512, 4096], seed=0, policy=None),
    MLP: dict(name=MLP, n=1048576, T=256, K=[16], D=[0], seed=0, policy=("f32", "bf16")),
}

# Compute-factor sweep (the paper's "Simulator Complexity", factor C): C Euler
# iterations per step at a fixed state size, fused against unfused.
C_SWEEP = dict(name="cartpole-64k-100-Csweep", n=65536, T=100, K=[1, 100], C=[1, 4, 16, 64, 256, 1024], seed=0)

# The second simulator (the paper's Future Work: heavier, multi-body
# simulators): a cart carrying a chain of N uniform rods with the cart-pole's
# constants per link, N = 1 .. 4, fused (K = 200) against unfused (K = 1).
CHAIN_SWEEP = dict(name="chain-1M-200-Nsweep", n=1048576, T=200, K=[1, 200], N=[1, 2, 3, 4], seed=0)

# Parity seeds: 0, 1, and one whose high 32 bits are nonzero.
PARITY_SEEDS = (0, 1, (1 << 40) + 7)

# Per env-step bytes of the trajectory: obs 4 x f32, action u8, reward f32, done u8.
TRAJ_BYTES_PER_ENV_STEP = 4 * 4 + 1 + 4 + 1


def chain_traj_bytes_per_env_step(n_links: int) -> int:
    """Trajectory bytes per env-step of the chain: obs (2 N + 2) x f32, action
    u8, reward f32, done u8."""
    return 4 * (2 * n_links + 2) + 1 + 4 + 1


def mlp_weights(seed: int, hidden: int = 64):
    """4 -> hidden -> hidden -> 2 policy weights and the hidden -> 1 value head,
    ~ N(0, 1/fan_in), row-major [out][in], zero biases, fp32.  Drawn with numpy's
    PCG64 generator from ``seed`` (the value head last)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shapes = [(hidden, 4), (hidden, hidden), (2, hidden), (1, hidden)]
    ws = [(rng.standard_normal(s) / math.sqrt(s[1])).astype(np.float32) for s in shapes]
    bs = [np.zeros(s[0], dtype=np.float32) for s in shapes]
    return dict(w1=ws[0], b1=bs[0], w2=ws[1], b2=bs[1], w3=ws[2], b3=bs[2], wv=ws[3], bv=bs[3])
