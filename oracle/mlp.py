"""Policy / value MLP forward and Gaussian log-probability (oracle side).

The paper trains Flax policy and value networks with PPO (Sec. II-A, IV) without giving
their sizes; the workloads here use 23 -> 256 -> 256 -> n_out with tanh hidden layers and
a linear output (the Gaussian mean for the policy, V for the value net).

Quantisation points of the bf16 path: the input of every layer is rounded to bf16
(round to nearest, ties to even), the weights are bf16, the biases fp32; the oracle
accumulates the products exactly in float64 and applies tanh in float64.
"""
from __future__ import annotations

import math

import numpy as np


def bf16_round(x) -> np.ndarray:
    """Round real values (float64) to the nearest bf16 value, ties to even.

    bf16 has 8 significant bits and fp32's exponent range: for |x| >= 2^-126 the quantum
    is 2^(e-7) with 2^e <= |x| < 2^(e+1); below that (subnormal) it is 2^-133.
    Values beyond the largest finite bf16 round to infinity; NaN and inf pass through."""
    x = np.asarray(x, np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x) & (x != 0.0)
    xf = x[fin]
    _, e = np.frexp(np.abs(xf))              # |x| = f 2^e, f in [0.5, 1) -> 2^(e-1) <= |x|
    e = np.maximum(e - 1, -126)
    quantum = np.ldexp(1.0, e - 7)
    r = np.rint(xf / quantum) * quantum      # np.rint rounds half to even
    max_bf16 = (2.0 - 2.0 ** -7) * 2.0 ** 127
    r = np.where(np.abs(r) > max_bf16, np.copysign(np.inf, r), r)
    out[fin] = r
    return out


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Value of bf16 bit patterns (uint16), exactly."""
    b = np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def mlp_forward(obs: np.ndarray, net: dict, hidden_out: bool = False):
    """MLP forward for observations obs [n_in, n] (column per env).

    h1 = tanh(W1 q(o) + b1), h2 = tanh(W2 q(h1) + b2), y = W3 q(h2) + b3, q = bf16 round.
    Returns y [n_out, n] (and (h1, h2) when hidden_out)."""
    W = [bf16_bits_to_f64(net[f"W{i}"]) for i in (1, 2, 3)]
    b = [np.asarray(net[f"b{i}"], np.float32).astype(np.float64) for i in (1, 2, 3)]
    h1 = np.tanh(W[0] @ bf16_round(obs) + b[0][:, None])
    h2 = np.tanh(W[1] @ bf16_round(h1) + b[1][:, None])
    y = W[2] @ bf16_round(h2) + b[2][:, None]
    return (y, h1, h2) if hidden_out else y


def gaussian_logp(eps: np.ndarray, log_std: np.ndarray) -> np.ndarray:
    """log N(a; mu, sigma) summed over action dims for a = mu + sigma eps:
    sum_j [-eps_j^2 / 2 - log sigma_j - log(2 pi) / 2]; eps [8, n] -> [n]."""
    ls = np.asarray(log_std, np.float32).astype(np.float64)[:, None]
    return np.sum(-0.5 * eps * eps - ls - 0.5 * math.log(2.0 * math.pi), axis=0)
