"""Pins of the oracle's MLP policy (CPU only).

The policy is h1 = tanh(W1 obs + b1), h2 = tanh(W2 h1 + b2), logits = W3 h2 +
b3, p0 = softmax(logits)[0], action = (u < p0 ? 0 : 1).  Pins:

* zero weights give p0 = 1/2 exactly, so the action is (u >= 1/2);
* sparse, asymmetric weights reduce the network to a scalar composition with
  a closed form (a transposed or misplaced weight changes the value);
* bf16 rounding agrees with torch's float -> bfloat16 conversion;
* the empirical action frequency matches the mean p0.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads

P = oracle.make_params(**workloads.CARTPOLE)


def _zeros():
    z = lambda *s: np.zeros(s, dtype=np.float32)  # noqa: E731
    return dict(w1=z(64, 4), b1=z(64), w2=z(64, 64), b2=z(64), w3=z(2, 64), b3=z(2))


def test_zero_weights_half():
    pol = oracle.Policy(**_zeros())
    for obs in ([0, 0, 0, 0], [1.0, -2.0, 0.1, 3.0]):
        assert pol.p0(np.array(obs, dtype=np.float32)) == 0.5
    # the loop then takes action 1 exactly when u >= 1/2
    sim = oracle.Sim(32, 0, P)
    sim.reset(3)
    tr = sim.step(40, policy=pol)
    for e in range(32):
        for t in range(40):
            u = oracle.policy_u(3, e, t)
            assert tr["action"][t, e] == (0 if u < 0.5 else 1)
            assert tr["p0"][t, e] == 0.5


@pytest.mark.parametrize("bf16", [False, True])
def test_sparse_weights_closed_form(bf16):
    w = _zeros()
    # h1[5] = tanh(0.75 * theta + 0.125); h2[9] = tanh(1.5 * h1[5] - 0.25)
    # logits = (2 h2[9] + 0.5, -h2[9]): every value below is exact in bf16
    w["w1"][5, 2] = 0.75
    w["b1"][5] = 0.125
    w["w2"][9, 5] = 1.5
    w["b2"][9] = -0.25
    w["w3"][0, 9] = 2.0
    w["w3"][1, 9] = -1.0
    w["b3"][0] = 0.5
    pol = oracle.Policy(**w, bf16=bf16)
    rb = oracle.round_bf16 if bf16 else (lambda v: v)
    for th in (-0.2, -0.03125, 0.0, 0.0625, 0.2):
        obs = np.array([0.3, -0.7, th, 1.1], dtype=np.float32)
        h1 = rb(math.tanh(0.75 * rb(float(obs[2])) + 0.125))
        h2 = rb(math.tanh(1.5 * h1 - 0.25))
        l0, l1 = 2.0 * h2 + 0.5, -h2
        want = math.exp(l0) / (math.exp(l0) + math.exp(l1))
        assert abs(pol.p0(obs) - want) < 1e-14, th


def test_bf16_rounding_matches_torch():
    rng = np.random.Generator(np.random.PCG64(5))
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-38).astype(np.float32),     # subnormal range
        np.array([1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8), 3.0e38, 1e-45, 0.0], dtype=np.float32),  # ties / extremes
    ])
    want = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in vals])
    assert np.array_equal(got, want)


def test_action_frequency_matches_p0():
    wts = workloads.mlp_weights(7)
    pol = oracle.Policy(**wts)
    sim = oracle.Sim(512, 0, P)
    sim.reset(11)
    tr = sim.step(64, policy=pol)
    p0 = tr["p0"]
    frac0 = (tr["action"] == 0).mean()
    n = p0.size
    sd = math.sqrt((p0 * (1 - p0)).sum()) / n
    assert abs(frac0 - p0.mean()) < 5 * sd + 1e-12
    assert 0.0 < p0.min() and p0.max() < 1.0 and p0.std() > 0.01
