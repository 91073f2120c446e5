"""Pins for the oracle's bf16 rounding, MLP forward, Gaussian log-prob and GAE (CPU only)."""
import math

import numpy as np
import pytest
import torch
from scipy.stats import norm

import workloads as W
from oracle import gae as ogae
from oracle import mlp as omlp


def test_bf16_round_matches_torch():
    r = np.random.Generator(np.random.PCG64(2))
    bits = r.integers(0, 2**32, size=2_000_000, dtype=np.uint64).astype(np.uint32)
    # add ties (lower 16 bits exactly 0x8000), near-ties, subnormals, extremes
    ties = (r.integers(0, 2**16, size=20000, dtype=np.uint32) << 16) | np.uint32(0x8000)
    extra = np.array([0, 0x80000000, 0x00000001, 0x00008000, 0x00018000, 0x7F7FFFFF, 0x7F7F8000,
                      0x7F800000, 0xFF800000, 0x3F808000, 0x3F818000, 0x3F807FFF], np.uint32)
    bits = np.concatenate([bits, ties, ties ^ np.uint32(1), extra])
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    mine = omlp.bf16_round(x.astype(np.float64))
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mine, ref)
    assert np.isnan(omlp.bf16_round(np.array([np.nan]))[0])
    assert omlp.bf16_round(np.array([np.inf]))[0] == np.inf


def _net(n_out, W1=None, W2=None, W3=None, b=(0.0, 0.0, 0.0), n_in=23, hidden=256):
    def bits(a):
        return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    net = {"W1": bits(np.zeros((hidden, n_in)) if W1 is None else W1),
           "W2": bits(np.zeros((hidden, hidden)) if W2 is None else W2),
           "W3": bits(np.zeros((n_out, hidden)) if W3 is None else W3),
           "b1": np.full(hidden, b[0], np.float32), "b2": np.full(hidden, b[1], np.float32),
           "b3": np.full(n_out, b[2], np.float32)}
    return net


def test_mlp_zero_weights_give_bias_chain():
    net = _net(8, b=(0.3, -0.2, 0.05))
    y, h1, h2 = omlp.mlp_forward(np.random.default_rng(0).normal(size=(23, 5)), net, hidden_out=True)
    assert np.allclose(h1, math.tanh(float(np.float32(0.3))))
    assert np.allclose(h2, math.tanh(float(np.float32(-0.2))))
    assert np.allclose(y, float(np.float32(0.05)))


def test_mlp_orientation_and_quantisation_points():
    """Single-entry weights route input j -> hidden i -> hidden k -> output o; the input
    1 + 2^-8 (a bf16 tie) rounds to 1.0 before layer 1, and each hidden value is rounded
    to bf16 before the next layer."""
    W1 = np.zeros((256, 23)); W1[5, 17] = 1.0
    W2 = np.zeros((256, 256)); W2[200, 5] = 1.0
    W3 = np.zeros((8, 256)); W3[3, 200] = 2.0
    net = _net(8, W1, W2, W3)
    obs = np.zeros((23, 1)); obs[17, 0] = 1.0 + 2.0 ** -8
    y, h1, h2 = omlp.mlp_forward(obs, net, hidden_out=True)
    assert h1[5, 0] == math.tanh(1.0) and np.count_nonzero(h1) == 1
    t1 = float(torch.tensor(math.tanh(1.0), dtype=torch.float64).to(torch.bfloat16).double())
    assert h2[200, 0] == math.tanh(t1) and np.count_nonzero(h2) == 1
    t2 = float(torch.tensor(math.tanh(t1), dtype=torch.float64).to(torch.bfloat16).double())
    assert y[3, 0] == 2.0 * t2 and np.count_nonzero(y) == 1


def test_mlp_odd_symmetry_and_seeded_net_ranges():
    net = W.mlp_weights(8, W.POLICY_SEED)
    for k in ("b1", "b2", "b3"):
        net[k] = np.zeros_like(net[k])
    x = np.random.default_rng(1).normal(size=(23, 64))
    assert np.array_equal(omlp.mlp_forward(-x, net), -omlp.mlp_forward(x, net))
    net = W.mlp_weights(8, W.POLICY_SEED)
    w2 = omlp.bf16_bits_to_f64(net["W2"])
    assert abs(w2.std() - 1 / 16) < 2e-3 and abs(w2.mean()) < 2e-3
    assert np.all(np.abs(net["b1"]) <= 0.1)


def test_gaussian_logp_matches_scipy():
    r = np.random.default_rng(3)
    eps = r.normal(size=(8, 100))
    log_std = np.full(8, -0.5, np.float32)
    mu = r.normal(size=(8, 100))
    sigma = np.exp(float(np.float32(-0.5)))
    a = mu + sigma * eps
    ref = norm.logpdf(a, loc=mu, scale=sigma).sum(axis=0)
    assert np.allclose(omlp.gaussian_logp(eps, log_std), ref, atol=1e-12)


# ---- GAE ----------------------------------------------------------------------------

def _traj(T=64, n=50, p_done=0.05, seed=4):
    r = np.random.default_rng(seed)
    return (r.normal(size=(T, n)), r.normal(size=(T, n)), (r.random((T, n)) < p_done).astype(float),
            r.normal(size=n))


def test_gae_lambda0_is_td_error():
    rew, val, done, last = _traj()
    adv, ret = ogae.gae(rew, val, done, last, 0.99, 0.0)
    nxt = np.concatenate([val[1:], last[None]])
    assert np.allclose(adv, rew + 0.99 * (1 - done) * nxt - val, atol=1e-12)
    assert np.allclose(ret, adv + val)


def test_gae_lambda1_no_dones_is_discounted_return():
    rew, val, _, last = _traj()
    T = rew.shape[0]
    g = 0.97
    adv, _ = ogae.gae(rew, val, np.zeros_like(rew), last, g, 1.0)
    for t in (0, 10, T - 1):
        ret = sum(g ** k * rew[t + k] for k in range(T - t)) + g ** (T - t) * last
        assert np.allclose(adv[t], ret - val[t], atol=1e-10)


def test_gae_gamma0_and_done_cut():
    rew, val, done, last = _traj(p_done=0.3)
    adv, _ = ogae.gae(rew, val, done, last, 0.0, 0.95)
    assert np.allclose(adv, rew - val)
    adv, _ = ogae.gae(rew, val, done, last, 0.99, 0.95)
    m = done.astype(bool)
    assert np.allclose(adv[m], (rew - val)[m])


def test_gae_equals_truncated_sum_definition():
    """A_t = sum_l (gamma lambda)^l delta_{t+l}, summed until the first episode end."""
    rew, val, done, last = _traj(T=40, n=30, p_done=0.1)
    g, lam = 0.99, 0.95
    adv, _ = ogae.gae(rew, val, done, last, g, lam)
    T, n = rew.shape
    nxt = np.concatenate([val[1:], last[None]])
    delta = rew + g * (1 - done) * nxt - val
    for i in range(n):
        for t in range(T):
            s, f = 0.0, 1.0
            for l in range(t, T):
                s += f * delta[l, i]
                if done[l, i]:
                    break
                f *= g * lam
            assert adv[t, i] == pytest.approx(s, abs=1e-10)


def test_mlp_candidates_reduce_to_forward_without_ambiguity():
    net = W.mlp_weights(8, W.POLICY_SEED)
    x = np.random.default_rng(7).normal(size=(23, 300))
    y, cands = omlp.mlp_candidates(x, net, 0.0)
    assert np.array_equal(y, omlp.mlp_forward(x, net)) and cands == {}
    y, cands = omlp.mlp_candidates(x, net, 1e-6)
    assert 0 < len(cands) < 300
    for c, ys in cands.items():
        assert ys.shape[0] == 8 and ys.shape[1] >= 2
        # the plain forward is one of the valid outputs (up to fp64 summation order)
        assert np.min(np.max(np.abs(ys - y[:, c:c + 1]), axis=0)) < 1e-12
    assert np.all(omlp.nearest_valid_error(y, x, net, 1e-6) < 1e-12)


def test_mlp_candidates_contain_both_roundings_of_a_tie():
    """Hidden-1 value exactly at a bf16 midpoint (bias makes tanh land there): both
    roundings must appear among the valid outputs."""
    import math
    W1 = np.zeros((256, 23)); W1[5, 0] = 1.0
    W2 = np.zeros((256, 256)); W2[9, 5] = 1.0
    W3 = np.zeros((8, 256)); W3[2, 9] = 1.0
    net = _net(8, W1, W2, W3)
    mid = 0.5 + 2.0 ** -9                       # midpoint between bf16 0.5 and 0.50390625
    net["b1"][:] = 0.0
    obs = np.zeros((23, 1))
    obs[0, 0] = 0.0
    net["b1"][5] = np.float32(math.atanh(mid))  # tanh(b1) ~ mid (within fp32 of b1)
    h = math.tanh(float(net["b1"][5]))
    assert abs(h - mid) < 1e-7
    y, cands = omlp.mlp_candidates(obs, net, 1e-6)
    assert 0 in cands
    outs = sorted(set(np.round(cands[0][2], 12)))
    want = sorted({round(math.tanh(0.5), 12), round(math.tanh(0.50390625), 12)})
    got_h2 = [float(torch.tensor(v, dtype=torch.float64).to(torch.bfloat16).double()) for v in want]
    assert len(outs) == 2 and np.allclose(outs, got_h2)
