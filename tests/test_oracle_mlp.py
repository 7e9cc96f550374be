"""Pins of the oracle's MLP policy (CPU only).

The policy is h1 = tanh(W1 obs + b1), h2 = tanh(W2 h1 + b2), logits = W3 h2 +
b3, p0 = softmax(logits)[0], action = (u < p0 ? 0 : 1).  Pins:

* zero weights give p0 = 1/2 exactly, so the action is (u >= 1/2);
* sparse, asymmetric weights reduce the network to a scalar composition with
  a closed form (a transposed or misplaced weight changes the value);
* bf16 rounding agrees with torch's float -> bfloat16 conversion;
* the empirical action frequency matches the mean p0.

The learner outputs (the value head v = Wv h2 + bv on the shared trunk, and
log pi(a|obs) = log softmax(logits)[a] of the action taken) are pinned by:

* zero weights: log pi = log 1/2 for both actions and v = bv;
* the sparse closed form above, extended by a value weight;
* extreme logits, where a direct log(e^l0 / (e^l0 + e^l1)) overflows;
* the identities e^logp0 + e^logp1 = 1 and logp0 - logp1 = l0 - l1;
* a value head that copies the first logit row reproduces logit 0 exactly;
* an independent float64 torch evaluation (torch.tanh, log_softmax) of every
  recorded step of a trajectory, for fp32 and bf16-rounded weights.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads

P = oracle.make_params(**workloads.CARTPOLE)


def _zeros(value=False):
    z = lambda *s: np.zeros(s, dtype=np.float32)  # noqa: E731
    w = dict(w1=z(64, 4), b1=z(64), w2=z(64, 64), b2=z(64), w3=z(2, 64), b3=z(2))
    if value:
        w.update(wv=z(1, 64), bv=z(1))
    return w


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


@pytest.mark.parametrize("bf16", [False, True])
def test_sparse_weights_closed_form_value_and_logp(bf16):
    w = _zeros(value=True)
    w["w1"][5, 2] = 0.75
    w["b1"][5] = 0.125
    w["w2"][9, 5] = 1.5
    w["b2"][9] = -0.25
    w["w3"][0, 9] = 2.0
    w["w3"][1, 9] = -1.0
    w["b3"][0] = 0.5
    w["wv"][0, 9] = -3.0        # v = -3 h2[9] + 0.25
    w["bv"][0] = 0.25
    pol = oracle.Policy(**w, bf16=bf16)
    rb = oracle.round_bf16 if bf16 else (lambda v: v)
    for th in (-0.2, -0.03125, 0.0, 0.0625, 0.2):
        obs = np.array([0.3, -0.7, th, 1.1], dtype=np.float32)
        h2 = rb(math.tanh(1.5 * rb(math.tanh(0.75 * rb(float(obs[2])) + 0.125)) - 0.25))
        l0, l1 = 2.0 * h2 + 0.5, -h2
        logit, p0, v = pol.eval(obs)
        assert abs(logit[0] - l0) < 1e-15 and abs(logit[1] - l1) < 1e-15
        assert abs(v - (-3.0 * h2 + 0.25)) < 1e-15
        p = math.exp(l0) / (math.exp(l0) + math.exp(l1))
        assert abs(pol.log_prob(obs, 0) - math.log(p)) < 1e-14
        assert abs(pol.log_prob(obs, 1) - math.log(1.0 - p)) < 1e-14


def test_zero_weights_logp_and_value():
    w = _zeros(value=True)
    w["bv"][0] = 0.375
    pol = oracle.Policy(**w)
    obs = np.array([1.0, -2.0, 0.1, 3.0], dtype=np.float32)
    _, p0, v = pol.eval(obs)
    assert p0 == 0.5 and v == 0.375
    assert pol.log_prob(obs, 0) == pol.log_prob(obs, 1) == -math.log(2.0)
    # no value head: value reads 0 and the trajectory has no value plane
    w.pop("wv"), w.pop("bv")
    assert oracle.Policy(**w).eval(obs)[2] == 0.0
    sim = oracle.Sim(8, 0, P)
    sim.reset(0)
    assert "value" not in sim.step(2, policy=oracle.Policy(**w))


@pytest.mark.parametrize("l0,l1", [(1000.0, 0.0), (-800.0, 800.0), (0.0, -745.5), (3.0, 3.0), (1e-3, -1e-3)])
def test_log_prob_extreme_logits(l0, l1):
    lp0 = oracle.log_prob([l0, l1], 0)
    lp1 = oracle.log_prob([l0, l1], 1)
    # log pi(a) = -softplus(l_other - l_a), softplus(z) = max(z, 0) + log1p(e^-|z|)
    sp = lambda z: max(z, 0.0) + math.log1p(math.exp(-abs(z)))  # noqa: E731
    assert math.isfinite(lp0) and math.isfinite(lp1)
    assert abs(lp0 + sp(l1 - l0)) <= 1e-15 * max(1.0, abs(lp0))
    assert abs(lp1 + sp(l0 - l1)) <= 1e-15 * max(1.0, abs(lp1))


def test_logp_identities_and_value_copy_of_logit_row():
    wts = workloads.mlp_weights(21)
    rng = np.random.Generator(np.random.PCG64(4))
    for bf16 in (False, True):
        w = dict(wts, wv=wts["w3"][:1].copy(), bv=np.array([0.7], dtype=np.float32))
        w["b3"] = np.array([0.7, -0.2], dtype=np.float32)
        pol = oracle.Policy(**w, bf16=bf16)
        for _ in range(50):
            obs = rng.uniform(-0.3, 0.3, 4).astype(np.float32)
            logit, p0, v = pol.eval(obs)
            assert v == logit[0]                      # same row, same order of sums
            lp0, lp1 = oracle.log_prob(logit, 0), oracle.log_prob(logit, 1)
            assert abs(math.exp(lp0) + math.exp(lp1) - 1.0) < 1e-15
            assert abs((lp0 - lp1) - (logit[0] - logit[1])) < 1e-14
            assert abs(math.exp(lp0) - p0) < 1e-15


@pytest.mark.parametrize("bf16", [False, True])
def test_trajectory_outputs_match_torch_float64(bf16):
    """Every recorded step: the oracle's logp and value equal a float64 torch
    evaluation (a separate implementation) on the recorded obs and action.  In
    bf16 mode the two sum in different orders, so a hidden unit within an ulp of
    a bf16 rounding tie may round the other way: a few steps may differ by such
    a flip (|w| 2^-8 at most), the rest agree to 1e-13."""
    import torch.nn.functional as F
    wts = workloads.mlp_weights(8)
    rng = np.random.Generator(np.random.PCG64(9))
    for k in ("b1", "b2", "b3", "bv"):
        wts[k] = (rng.standard_normal(wts[k].shape) * 0.2).astype(np.float32)
    pol = oracle.Policy(**wts, bf16=bf16)
    sim = oracle.Sim(64, 0, P)
    sim.reset(2)
    tr = sim.step(48, policy=pol)

    def r(x):
        t = torch.as_tensor(np.asarray(x), dtype=torch.float64)
        return t.to(torch.bfloat16).to(torch.float64) if bf16 else t

    W = {k: r(wts[k]) for k in ("w1", "w2", "w3", "wv")}
    B = {k: torch.as_tensor(wts[k], dtype=torch.float64) for k in ("b1", "b2", "b3", "bv")}
    obs = r(tr["obs"].transpose(0, 2, 1).reshape(-1, 4))                 # [K*n, 4]
    h1 = r(torch.tanh(obs @ W["w1"].T + B["b1"]))
    h2 = r(torch.tanh(h1 @ W["w2"].T + B["b2"]))
    logits = h2 @ W["w3"].T + B["b3"]
    value = (h2 @ W["wv"].T + B["bv"])[:, 0]
    act = torch.as_tensor(tr["action"].reshape(-1).astype(np.int64))
    logp = F.log_softmax(logits, dim=1).gather(1, act[:, None])[:, 0]
    for got, want in ((tr["logp"], logp), (tr["value"], value), (tr["p0"], torch.softmax(logits, 1)[:, 0])):
        d = np.abs(got.reshape(-1) - want.numpy())
        if bf16:
            assert (d > 1e-13).mean() < 0.01 and d.max() < 1e-2
        else:
            assert d.max() < 1e-13


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
