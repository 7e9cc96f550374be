"""Pins of the policy tolerance, the oracle's orc_mlp_bounds (CPU only).

The enclosure must hold every value that a device evaluation under its error
model can return, and not be vacuous:
* with a zero error model (no accumulation error, exact functions) it
  collapses onto the oracle's own evaluation;
* a policy with zero output weights has logits equal to their biases, and with
  zero biases too p0 = 1/2 exactly: the enclosure is then exactly 1/2 +- the
  p0 error and log 1/2 +- the log pi error;
* an emulation of device arithmetic written here independently of the oracle
  (numpy float32 dot products summed in a random order, torch's bf16
  rounding, tanh, p0 and log pi perturbed by up to 95% of the model's function
  errors, every dot product moved by 45% of its accumulation allowance on top
  of its own fp32 rounding, at random or all in the direction that moves the
  logit difference most) lands inside it: with the function errors zero, at
  the model's own size, and inflated 1000-fold, where bf16 rounding flips of
  hidden units are frequent;
* the same emulation with perturbations four times past the model lands
  outside it for a large share of observations.
"""
import numpy as np
import pytest
import torch

import oracle
import policy_bounds
import workloads

F32 = np.float32


def _round_bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=F32)).to(torch.bfloat16).to(torch.float32).numpy()


def _setup(seed=3, n=600):
    rng = np.random.Generator(np.random.PCG64(seed))
    w = workloads.mlp_weights(seed)
    for k in ("b1", "b2", "b3", "bv"):
        w[k] = (rng.standard_normal(w[k].shape) * 0.3).astype(F32)
    # cart-pole-like observations, some far from the reset box
    obs = (rng.standard_normal((n, 4)) * np.array([1.0, 1.5, 0.15, 1.5])).astype(F32)
    return w, obs


def _emulate(w, obs, bf16, scale, over, adversarial, rng, acc_over=0.45):
    """p0, log pi(0), log pi(1), value of a device-like evaluation of each obs."""
    n = obs.shape[0]
    W = {k: (_round_bf16(w[k]) if bf16 else w[k].astype(F32)) for k in ("w1", "w2", "w3", "wv")}
    B = {k: w[k].astype(F32) for k in ("b1", "b2", "b3", "bv")}
    x = _round_bf16(obs) if bf16 else obs.astype(F32)

    def dot(Wm, b, h, sign=None):
        nout, nin = Wm.shape
        terms = np.concatenate([np.broadcast_to(b[None, :, None], (n, nout, 1)), h[:, None, :] * Wm[None, :, :]],
                               axis=2)                       # fp32 products, rounded once (exact for bf16)
        acc = np.zeros((n, nout), dtype=F32)
        for j in rng.permutation(nin + 1):
            acc = (acc + terms[:, :, j]).astype(F32)
        # plus a share of the accumulation allowance: the fp32 sum's own rounding
        # (at most (n + 1) u S) and this (0.9 (n + 1) u S) and the final
        # rounding stay inside 2 (n + 1) u S
        mag = np.abs(terms.astype(np.float64)).sum(axis=2)
        if sign is None:
            sign = rng.uniform(-1, 1, acc.shape)
        return (acc + sign * acc_over * policy_bounds.ACC * (nin + 1) * mag).astype(F32)

    e_tanh = policy_bounds.E_TANH * scale
    dw3 = W["w3"][1].astype(np.float64) - W["w3"][0]

    def act(z, sign):
        t = (np.tanh(z.astype(np.float64)) + sign * over * e_tanh).astype(F32)
        return _round_bf16(t) if bf16 else t

    if adversarial:
        # push every hidden unit the way that raises the logit difference d
        z1 = dot(W["w1"], B["b1"], x, np.zeros((n, 64)))
        z2p = dot(W["w2"], B["b2"], act(z1, 0.0), np.zeros((n, 64)))
        g1 = ((1.0 - np.tanh(z2p.astype(np.float64)) ** 2) * dw3[None, :]) @ W["w2"].astype(np.float64)
        s1, s2 = np.sign(g1), np.sign(dw3)[None, :]
        z1 = dot(W["w1"], B["b1"], x, s1)
        sl, sv = np.array([[-1.0, 1.0]]), np.ones((n, 1))
    else:
        z1 = dot(W["w1"], B["b1"], x)
        s1, s2, sl, sv = rng.uniform(-1, 1, z1.shape), rng.uniform(-1, 1, (n, 64)), None, None
    h2 = act(dot(W["w2"], B["b2"], act(z1, s1), s2), s2)
    logit = dot(W["w3"], B["b3"], h2, sl)
    value = dot(W["wv"], B["bv"], h2, sv)[:, 0]
    d = (logit[:, 1] - logit[:, 0]).astype(F32).astype(np.float64)
    sp = np.sign(d) if adversarial else rng.uniform(-1, 1, n)
    p0 = (1.0 / (1.0 + np.exp(d)) + sp * over * policy_bounds.E_P0 * scale).astype(F32)

    def logpi(z):
        r = -(np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z))))
        return (r + rng.uniform(-1, 1, n) * over * policy_bounds.E_LOGPI * scale * (1.0 + np.abs(r))).astype(F32)

    return dict(p0=p0, logp0=logpi(d), logp1=logpi(-d), value=value)


def _inside_fraction(pol, obs, em, errs):
    hits = {k: 0 for k in em}
    for i in range(obs.shape[0]):
        b = pol.bounds(obs[i], errs)
        for k in em:
            lo, hi = b[k]
            hits[k] += int(lo <= float(em[k][i]) <= hi)
    return {k: v / obs.shape[0] for k, v in hits.items()}


@pytest.mark.parametrize("bf16", [False, True])
def test_zero_error_model_collapses_onto_the_oracle(bf16):
    w, obs = _setup(n=50)
    pol = oracle.Policy(**w, bf16=bf16)
    zero = oracle.Errs(0.0, 0.0, 0.0, 0.0)
    for o in obs:
        logit, p0, v = pol.eval(o)
        b = pol.bounds(o, zero)
        want = dict(p0=p0, logp0=oracle.log_prob(logit, 0), logp1=oracle.log_prob(logit, 1), value=v)
        for k, x in want.items():
            lo, hi = b[k]
            assert abs(lo - x) <= 1e-12 and abs(hi - x) <= 1e-12, (k, lo, hi, x)


@pytest.mark.parametrize("bf16", [False, True])
def test_constant_logits_closed_form(bf16):
    """W3 = 0 and b3 = 0 make d = 0 whatever the trunk does, so a device's p0 is
    1/2 up to the p0 error alone and its log pi log 1/2 up to the log pi error;
    Wv = 0 and bv = 0 make the value exactly 0."""
    w, obs = _setup(n=20)
    for k in ("w3", "b3", "wv", "bv"):
        w[k] = np.zeros_like(w[k])
    pol = oracle.Policy(**w, bf16=bf16)
    errs = policy_bounds.errs()
    lg = np.log(0.5)
    for o in obs:
        b = pol.bounds(o, errs)
        assert b["p0"] == (0.5 - errs.p0, 0.5 + errs.p0)
        for k in ("logp0", "logp1"):
            assert np.allclose(b[k], (lg - errs.logpi * (1 - lg), lg + errs.logpi * (1 - lg)), rtol=0, atol=1e-15)
        assert b["value"] == (0.0, 0.0)


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("scale,over,adversarial", [(0.0, 0.0, False), (1.0, 0.95, False), (1000.0, 0.95, False),
                                                    (1000.0, 0.95, True), (1.0, 0.95, True)])
def test_emulated_device_evaluations_lie_inside(bf16, scale, over, adversarial):
    w, obs = _setup()
    pol = oracle.Policy(**w, bf16=bf16)
    rng = np.random.Generator(np.random.PCG64(11))
    em = _emulate(w, obs, bf16, scale, over, adversarial, rng)
    frac = _inside_fraction(pol, obs, em, policy_bounds.errs(scale))
    assert all(v == 1.0 for v in frac.values()), frac
    # the oracle's own values lie inside too
    for o in obs[:50]:
        logit, p0, v = pol.eval(o)
        b = pol.bounds(o, policy_bounds.errs(scale))
        assert b["p0"][0] <= p0 <= b["p0"][1] and b["value"][0] <= v <= b["value"][1]


@pytest.mark.parametrize("bf16", [False, True])
def test_perturbations_past_the_model_escape(bf16):
    w, obs = _setup()
    pol = oracle.Policy(**w, bf16=bf16)
    rng = np.random.Generator(np.random.PCG64(12))
    em = _emulate(w, obs, bf16, 1000.0, 4.0, True, rng)
    frac = _inside_fraction(pol, obs, em, policy_bounds.errs(1000.0))
    assert frac["p0"] <= 0.75 and frac["logp0"] <= 0.8 and frac["logp1"] <= 0.8, frac


def test_bf16_enclosure_covers_rounding_flips():
    """At the model's real size most bf16 enclosures are as narrow as fp32's;
    the few wide ones are observations with a hidden unit near a bf16 rounding
    boundary, where the flip moves p0 by far more than fp32 arithmetic does."""
    w, obs = _setup(n=400)
    widths = {}
    for bf16 in (False, True):
        pol = oracle.Policy(**w, bf16=bf16)
        widths[bf16] = np.array([np.subtract(*pol.bounds(o, policy_bounds.errs())["p0"][::-1]) for o in obs])
    assert np.median(widths[True]) < 2 * np.median(widths[False])
    assert widths[True].max() > 4 * widths[False].max()
