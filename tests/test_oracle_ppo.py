"""Pins of the PPO-update oracle (oracle/ppo.py) against things other than itself:
torch autograd for the MLP backward, central finite differences of the whole objective,
scipy's normal log-density and entropy, hand-computed clipped-surrogate cases,
torch.optim.Adam and torch's global-norm clipping, and the bf16 error bound for the
quantised gradient."""
import math

import numpy as np
import pytest
import scipy.stats
import torch

from oracle import ppo
from oracle.mlp import bf16_round


def _params(rng, n_in, hidden, n_out, log_std=True, scale=1.0):
    p = {"W1": rng.standard_normal((hidden, n_in)) / math.sqrt(n_in) * scale,
         "W2": rng.standard_normal((hidden, hidden)) / math.sqrt(hidden) * scale,
         "W3": rng.standard_normal((n_out, hidden)) / math.sqrt(hidden) * scale,
         "b1": rng.uniform(-0.1, 0.1, hidden), "b2": rng.uniform(-0.1, 0.1, hidden),
         "b3": rng.uniform(-0.1, 0.1, n_out)}
    if log_std:
        p["log_std"] = rng.uniform(-0.8, -0.2, 8)
    return p


def _batch(rng, B, pol, ratio_targets=None):
    """obs, act, logp_old, adv, ret; logp_old set so the ratios hit ratio_targets (using
    scipy's log-density of the unquantised policy mean, independent of the oracle)."""
    obs = rng.uniform(-1.5, 1.5, (23, B))
    mu, _ = ppo.mlp_forward_cache(obs, pol, quantize=False)
    sig = np.exp(pol["log_std"])[:, None]
    act = mu + sig * rng.standard_normal((8, B))
    logp = scipy.stats.norm.logpdf(act, loc=mu, scale=sig).sum(axis=0)
    if ratio_targets is None:
        ratio_targets = rng.uniform(0.5, 1.5, B)
    logp_old = logp - np.log(ratio_targets)
    adv = rng.standard_normal(B)
    ret = rng.standard_normal(B)
    return obs, act, logp_old, adv, ret


def test_mlp_backward_matches_torch_autograd():
    rng = np.random.default_rng(0)
    p = _params(rng, 23, 16, 8, log_std=False)
    x = rng.uniform(-1, 1, (23, 9))
    gy = rng.standard_normal((8, 9))
    y, cache = ppo.mlp_forward_cache(x, p, quantize=False)
    got = ppo.mlp_backward(p, cache, gy, quantize=False)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    X = torch.tensor(x.T)
    h1 = torch.tanh(torch.nn.functional.linear(X, t["W1"], t["b1"]))
    h2 = torch.tanh(torch.nn.functional.linear(h1, t["W2"], t["b2"]))
    Y = torch.nn.functional.linear(h2, t["W3"], t["b3"])
    assert np.allclose(Y.detach().numpy().T, y, rtol=1e-13, atol=1e-13)
    (Y * torch.tensor(gy.T)).sum().backward()
    for k in p:
        assert np.allclose(got[k], t[k].grad.numpy(), rtol=1e-11, atol=1e-13), k


@pytest.mark.parametrize("normalize", [True, False])
def test_ppo_gradient_central_differences(normalize):
    """Analytic gradient of the whole objective (policy and value parameters, log_std)
    against central differences, with ratios on both sides of both clip bounds."""
    rng = np.random.default_rng(1)
    hidden, B = 8, 16
    pol = _params(rng, 23, hidden, 8)
    val = _params(rng, 23, hidden, 1, log_std=False)
    ratios = np.array([0.5, 0.7, 0.9, 1.0, 1.1, 1.3, 1.5, 0.6] * 2)
    obs, act, logp_old, adv, ret = _batch(rng, B, pol, ratios)
    hp = dict(normalize_adv=normalize, ent_coef=0.01, vf_coef=0.5)
    out = ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, pol, val, hp, quantize=False)
    r = out["ratio"]
    assert np.all(np.abs(r - 0.8) > 1e-3) and np.all(np.abs(r - 1.2) > 1e-3)
    assert 0 < out["clip_frac"] < 1

    def loss_at(which, theta):
        shapes = (23, hidden, 8, True) if which == "pol" else (23, hidden, 1, False)
        p = ppo.unpack(theta, *shapes)
        args = (p, val) if which == "pol" else (pol, p)
        return ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, *args, hp, quantize=False)["loss"]

    for which, net, g in (("pol", pol, out["grad_pol"]), ("val", val, out["grad_val"])):
        theta = ppo.pack(net)
        idx = np.unique(np.concatenate([rng.choice(theta.size, 60, replace=False),
                                        np.arange(theta.size - (16 if which == "pol" else 1), theta.size)]))
        h = 1e-6
        for i in idx:
            tp, tm = theta.copy(), theta.copy()
            tp[i] += h
            tm[i] -= h
            fd = (loss_at(which, tp) - loss_at(which, tm)) / (2 * h)
            assert abs(fd - g[i]) <= 1e-6 * max(1e-3, abs(g[i])) + 1e-9, (which, i, fd, g[i])


def test_clipped_surrogate_hand_cases():
    """One sample, no normalisation, eps = 0.2: the four sign / side cases of
    min(rho A, clip(rho) A) and whether the gradient flows."""
    rng = np.random.default_rng(2)
    pol = _params(rng, 23, 8, 8)
    val = _params(rng, 23, 8, 1, log_std=False)
    cases = [(+2.0, 1.5, -2.4, False), (-2.0, 0.5, 1.6, False), (+2.0, 0.5, -1.0, True),
             (-2.0, 1.5, 3.0, True), (+2.0, 1.1, -2.2, True)]
    for A, rho, want_loss, flows in cases:
        obs, act, logp_old, _, ret = _batch(rng, 1, pol, np.array([rho]))
        out = ppo.ppo_loss_grad(obs, act, logp_old, np.array([A]), ret, pol, val,
                                dict(normalize_adv=False), quantize=False)
        assert abs(out["ratio"][0] - rho) < 1e-12
        assert abs(out["pg_loss"] - want_loss) < 1e-12
        g_mu_part = out["grad_pol"][:-8]
        g_ls = out["grad_pol"][-8:]
        n_w1 = 8 * 23
        assert (np.abs(g_mu_part[:n_w1]).max() > 0) == flows
        assert (np.abs(g_ls).max() > 0) == flows
        assert out["clip_frac"] == (0.0 if flows else 1.0)


def test_ratio_one_is_the_policy_gradient():
    """At rho = 1 every sample is unclipped and dL/dmu = -(1/B) A^ (a - mu) / sigma^2;
    with normalised advantages pg_loss = -mean(A^) = 0."""
    rng = np.random.default_rng(3)
    pol = _params(rng, 23, 8, 8)
    val = _params(rng, 23, 8, 1, log_std=False)
    B = 20
    obs, act, logp_old, adv, ret = _batch(rng, B, pol, np.ones(B))
    out = ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, pol, val, quantize=False)
    assert abs(out["pg_loss"]) < 1e-12 and out["clip_frac"] == 0.0
    ah = out["adv_hat"]
    assert abs(ah.mean()) < 1e-12 and abs(ah.std() - 1.0) < 1e-6
    # b3's gradient is the sum over samples of dL/dmu
    sig2 = np.exp(2 * pol["log_std"])[:, None]
    g_mu = -(ah[None, :] / B) * (act - out["mu"]) / sig2
    b3 = out["grad_pol"][-16:-8]
    assert np.allclose(b3, g_mu.sum(axis=1), rtol=1e-12, atol=1e-15)


def test_logp_entropy_value_loss_closed_forms():
    rng = np.random.default_rng(4)
    mu = rng.standard_normal((8, 5))
    ls = rng.uniform(-1, 0.5, 8)
    act = mu + rng.standard_normal((8, 5))
    want = scipy.stats.norm.logpdf(act, loc=mu, scale=np.exp(ls)[:, None]).sum(axis=0)
    assert np.allclose(ppo.gaussian_logp(act, mu, ls), want, rtol=1e-13)
    assert abs(ppo.gaussian_entropy(ls) - scipy.stats.norm(scale=np.exp(ls)).entropy().sum()) < 1e-12
    # value loss and gradient: zero when V = R; b3 gradient = c_v mean(V - R)
    pol = _params(rng, 23, 8, 8)
    val = _params(rng, 23, 8, 1, log_std=False)
    obs, act, logp_old, adv, _ = _batch(rng, 6, pol)
    v, _ = ppo.mlp_forward_cache(obs, val, quantize=False)
    out = ppo.ppo_loss_grad(obs, act, logp_old, adv, v[0], pol, val, quantize=False)
    assert out["v_loss"] == 0.0 and np.all(out["grad_val"] == 0.0)
    ret = v[0] - 0.25
    out = ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, pol, val, dict(vf_coef=0.5), quantize=False)
    assert abs(out["v_loss"] - 0.5 * 0.5 * 0.0625) < 1e-14
    assert abs(out["grad_val"][-1] - 0.5 * 0.25) < 1e-14


def test_quantised_gradient_within_bf16_bound():
    """With bf16 weights and the full 256-wide hidden layers, the quantised gradient
    differs from the exact one only by the bf16 rounding of the layer inputs and of the
    back-propagated values: a few units of 2^-8 of each tensor's scale."""
    rng = np.random.default_rng(5)
    pol = _params(rng, 23, 256, 8)
    val = _params(rng, 23, 256, 1, log_std=False)
    for p in (pol, val):
        for k in ("W1", "W2", "W3"):
            p[k] = bf16_round(p[k])
    obs, act, logp_old, adv, ret = _batch(rng, 64, pol, np.full(64, 1.0))
    q = ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, pol, val, quantize=True)
    e = ppo.ppo_loss_grad(obs, act, logp_old, adv, ret, pol, val, quantize=False)
    for net, shapes in (("grad_pol", (23, 256, 8, True)), ("grad_val", (23, 256, 1, False))):
        gq, ge = ppo.unpack(q[net], *shapes), ppo.unpack(e[net], *shapes)
        for k in gq:
            scale = np.abs(ge[k]).max()
            err = np.abs(gq[k] - ge[k]).max()
            assert err <= 16 * 2.0 ** -8 * scale, (net, k, err / scale)
            assert np.linalg.norm(gq[k] - ge[k]) <= 4 * 2.0 ** -8 * np.linalg.norm(ge[k]), (net, k)


def test_adam_matches_torch_and_first_step():
    rng = np.random.default_rng(6)
    hp = dict(lr=3e-4, beta1=0.9, beta2=0.999, adam_eps=1e-8)
    theta = rng.standard_normal(50)
    m = np.zeros(50)
    v = np.zeros(50)
    t_param = torch.tensor(theta.copy(), requires_grad=True)
    opt = torch.optim.Adam([t_param], lr=3e-4, betas=(0.9, 0.999), eps=1e-8)
    for t in range(1, 5):
        g = rng.standard_normal(50) * 10.0 ** rng.uniform(-4, 1, 50)
        if t == 1:
            want1 = theta - 3e-4 * g / (np.abs(g) + 1e-8)
        theta, m, v = ppo.adam_step(theta, g, m, v, t, hp)
        if t == 1:
            assert np.allclose(theta, want1, rtol=1e-14, atol=1e-16)
        t_param.grad = torch.tensor(g)
        opt.step()
        assert np.allclose(theta, t_param.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_clip_scale_matches_torch():
    rng = np.random.default_rng(7)
    gs = [rng.standard_normal(30), rng.standard_normal(7) * 3]
    for max_norm in (0.5, 100.0):
        ts = [torch.tensor(g.copy(), requires_grad=True) for g in gs]
        for t, g in zip(ts, gs):
            t.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_(ts, max_norm)
        s = ppo.clip_scale(gs, max_norm)
        for t, g in zip(ts, gs):
            assert np.allclose(t.grad.numpy(), s * g, rtol=1e-12)
    assert ppo.clip_scale(gs, 0.0) == 1.0
