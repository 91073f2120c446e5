"""PPO update of the policy and value MLPs on one minibatch (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper trains its PPO agent (Sec. III-A1, the on-policy learner) with the
clipped surrogate objective of Schulman et al. (2017), which it cites, and gives no
hyperparameters.  This module writes out that objective, its gradient through the two
MLPs, global-norm gradient clipping and Adam (Kingma and Ba, Algorithm 1), in float64.

Objective on a minibatch of B samples (columns b), with sigma_j = exp(log_std_j):
  logp_b   = sum_j [ -((a_jb - mu_jb) / sigma_j)^2 / 2 - log sigma_j - log(2 pi) / 2 ]
  rho_b    = exp(logp_b - logp_old_b)
  A^_b     = (A_b - mean A) / (std A + 1e-8)   (population std; or A_b if not normalised)
  L_clip   = -(1/B) sum_b min(rho_b A^_b, clip(rho_b, 1 - eps, 1 + eps) A^_b)
  L_value  = (c_v / 2) (1/B) sum_b (V_b - R_b)^2
  L_ent    = -c_e H,   H = sum_j (log sigma_j + (1 + log 2 pi) / 2)
  L        = L_clip + L_value + L_ent
The gradient of min(.) flows through the unclipped term where that term is the smaller
(ties included), and is zero where the clipped, constant term is the smaller.

Quantisation points (quantize=True), those of a bf16 MFMA implementation: the forward
as in mlp.mlp_forward (inputs of every layer rounded to bf16); in the backward, the output
gradient gy, dz2 and dz1 are rounded to bf16 before they enter a product (dW3 = q(gy)
q(h2)^T, dh2 = W3^T q(gy), dW2 = q(dz2) q(h1)^T, dh1 = W2^T q(dz2), dW1 = q(dz1) q(o)^T);
the bias gradients sum the unrounded values, and the tanh derivatives use the unrounded
activations.  Products are exact (float64).  With quantize=False every q is the identity.

Parameter packing (the same as the device buffers): W1 [H][n_in] | W2 [H][H] | W3 [n_out][H]
| b1 [H] | b2 [H] | b3 [n_out] | log_std [n_out] (policy only), row-major, float.
"""
from __future__ import annotations

import math

import numpy as np

from .mlp import bf16_round

LOG_2PI = math.log(2.0 * math.pi)

DEFAULTS = dict(clip_eps=0.2, vf_coef=0.5, ent_coef=0.0, max_grad_norm=0.5, lr=3e-4,
                beta1=0.9, beta2=0.999, adam_eps=1e-8, normalize_adv=True)


def _q(x, on: bool):
    return bf16_round(x) if on else np.asarray(x, np.float64)


# ---- parameters -----------------------------------------------------------------------
def unpack(theta: np.ndarray, n_in: int, hidden: int, n_out: int, with_log_std: bool) -> dict:
    """Flat packed parameters -> {W1, W2, W3, b1, b2, b3[, log_std]} (float64 views)."""
    t = np.asarray(theta, np.float64)
    shapes = [("W1", (hidden, n_in)), ("W2", (hidden, hidden)), ("W3", (n_out, hidden)),
              ("b1", (hidden,)), ("b2", (hidden,)), ("b3", (n_out,))]
    if with_log_std:
        shapes.append(("log_std", (n_out,)))
    out, o = {}, 0
    for k, s in shapes:
        n = int(np.prod(s))
        out[k] = t[o:o + n].reshape(s)
        o += n
    if o != t.size:
        raise ValueError(f"packed size {t.size} != {o}")
    return out


def pack(p: dict) -> np.ndarray:
    keys = ["W1", "W2", "W3", "b1", "b2", "b3"] + (["log_std"] if "log_std" in p else [])
    return np.concatenate([np.asarray(p[k], np.float64).ravel() for k in keys])


# ---- MLP forward with cache, backward -------------------------------------------------
def mlp_forward_cache(x: np.ndarray, p: dict, quantize: bool):
    """y = W3 q(h2) + b3, h2 = tanh(W2 q(h1) + b2), h1 = tanh(W1 q(x) + b1); x [n_in, B]."""
    u0 = _q(x, quantize)
    h1 = np.tanh(p["W1"] @ u0 + p["b1"][:, None])
    u1 = _q(h1, quantize)
    h2 = np.tanh(p["W2"] @ u1 + p["b2"][:, None])
    u2 = _q(h2, quantize)
    y = p["W3"] @ u2 + p["b3"][:, None]
    return y, dict(u0=u0, h1=h1, u1=u1, h2=h2, u2=u2)


def mlp_backward(p: dict, c: dict, gy: np.ndarray, quantize: bool) -> dict:
    """Gradients of sum_b <gy_b, y_b> w.r.t. the MLP parameters (chain rule, layer by
    layer from the output; d tanh(z) / dz = 1 - tanh(z)^2)."""
    gq = _q(gy, quantize)
    g = {"W3": gq @ c["u2"].T, "b3": gy.sum(axis=1)}
    dz2 = (p["W3"].T @ gq) * (1.0 - c["h2"] ** 2)
    dz2q = _q(dz2, quantize)
    g["W2"] = dz2q @ c["u1"].T
    g["b2"] = dz2.sum(axis=1)
    dz1 = (p["W2"].T @ dz2q) * (1.0 - c["h1"] ** 2)
    dz1q = _q(dz1, quantize)
    g["W1"] = dz1q @ c["u0"].T
    g["b1"] = dz1.sum(axis=1)
    return g


# ---- the PPO objective --------------------------------------------------------------
def normalized_advantages(adv: np.ndarray, on: bool) -> np.ndarray:
    a = np.asarray(adv, np.float64)
    if not on:
        return a
    return (a - a.mean()) / (a.std() + 1e-8)


def gaussian_logp(act: np.ndarray, mu: np.ndarray, log_std: np.ndarray) -> np.ndarray:
    """sum_j log N(a_j; mu_j, sigma_j^2) for columns of act, mu [8, B]."""
    z = (act - mu) * np.exp(-log_std)[:, None]
    return np.sum(-0.5 * z * z - log_std[:, None] - 0.5 * LOG_2PI, axis=0)


def gaussian_entropy(log_std: np.ndarray) -> float:
    return float(np.sum(log_std + 0.5 * (1.0 + LOG_2PI)))


def ppo_loss_grad(obs, act, logp_old, adv, ret, pol: dict, val: dict, hp: dict | None = None,
                  quantize: bool = True) -> dict:
    """Loss terms, statistics and gradients of one minibatch.

    obs [23, B], act [8, B], logp_old, adv, ret [B]; pol / val parameter dicts (float64
    values; pass bf16-valued weights to model the device).  Returns a dict with
    loss, pg_loss, v_loss, entropy, approx_kl (mean of logp_old - logp), clip_frac
    (fraction of samples whose gradient the clip removes), grad_pol / grad_val (packed),
    and the intermediate mu, value, logp, ratio, adv_hat."""
    hp = {**DEFAULTS, **(hp or {})}
    obs = np.asarray(obs, np.float64)
    act = np.asarray(act, np.float64)
    logp_old = np.asarray(logp_old, np.float64)
    ret = np.asarray(ret, np.float64)
    B = obs.shape[1]
    eps = hp["clip_eps"]
    ls = np.asarray(pol["log_std"], np.float64)

    mu, cp = mlp_forward_cache(obs, pol, quantize)
    v, cv = mlp_forward_cache(obs, val, quantize)
    v = v[0]
    ah = normalized_advantages(adv, hp["normalize_adv"])
    logp = gaussian_logp(act, mu, ls)
    ratio = np.exp(logp - logp_old)
    unclipped = ratio * ah
    clipped = np.clip(ratio, 1.0 - eps, 1.0 + eps) * ah
    active = unclipped <= clipped                 # gradient flows through the ratio
    pg_loss = -np.mean(np.minimum(unclipped, clipped))
    v_loss = 0.5 * hp["vf_coef"] * np.mean((v - ret) ** 2)
    ent = gaussian_entropy(ls)
    loss = pg_loss + v_loss - hp["ent_coef"] * ent

    # dL/dlogp_b = -(1/B) A^_b rho_b [active]; dlogp/dmu_j = (a_j - mu_j) / sigma_j^2,
    # dlogp/dlog_std_j = ((a_j - mu_j) / sigma_j)^2 - 1
    c = -(ah * ratio * active) / B
    inv_var = np.exp(-2.0 * ls)[:, None]
    d = act - mu
    g_mu = c[None, :] * d * inv_var
    g_ls = np.sum(c[None, :] * (d * d * inv_var - 1.0), axis=1) - hp["ent_coef"]
    g_v = (hp["vf_coef"] / B) * (v - ret)

    gp = mlp_backward(pol, cp, g_mu, quantize)
    gp["log_std"] = g_ls
    gv = mlp_backward(val, cv, g_v[None, :], quantize)
    return dict(loss=loss, pg_loss=pg_loss, v_loss=v_loss, entropy=ent,
                approx_kl=float(np.mean(logp_old - logp)), clip_frac=float(np.mean(~active)),
                grad_pol=pack(gp), grad_val=pack(gv), mu=mu, value=v, logp=logp, ratio=ratio,
                adv_hat=ah)


# ---- gradient clipping and Adam -------------------------------------------------------
def clip_scale(grads, max_norm: float) -> float:
    """Factor min(1, max_norm / (||g|| + 1e-6)) of global-norm clipping over all grads."""
    if max_norm <= 0:
        return 1.0
    norm = math.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in grads))
    return min(1.0, max_norm / (norm + 1e-6))


def adam_step(theta, grad, m, v, t: int, hp: dict | None = None, scale: float = 1.0):
    """One Adam step (t >= 1 counts steps including this one) on gradient scale * grad:
    m <- b1 m + (1 - b1) g, v <- b2 v + (1 - b2) g^2,
    theta <- theta - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
    Returns new (theta, m, v)."""
    hp = {**DEFAULTS, **(hp or {})}
    g = scale * np.asarray(grad, np.float64)
    b1, b2 = hp["beta1"], hp["beta2"]
    m = b1 * np.asarray(m, np.float64) + (1.0 - b1) * g
    v = b2 * np.asarray(v, np.float64) + (1.0 - b2) * g * g
    mh = m / (1.0 - b1 ** t)
    vh = v / (1.0 - b2 ** t)
    theta = np.asarray(theta, np.float64) - hp["lr"] * mh / (np.sqrt(vh) + hp["adam_eps"])
    return theta, m, v
