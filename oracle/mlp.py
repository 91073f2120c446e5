"""Policy / value MLP forward and Gaussian log-probability (oracle side).

The paper trains Flax policy and value networks with PPO (Sec. III-A, V) without giving
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


def mlp_candidates(obs: np.ndarray, net: dict, delta: float, max_amb: int = 10):
    """Every output the bf16 MLP may validly produce when hidden values are computed with
    an absolute error up to `delta` before their bf16 rounding.

    The hidden activations are rounded to bf16 before the next layer.  Where the exact
    value lies within `delta` of the midpoint between two bf16 neighbours, either
    rounding is a correct result of an implementation whose pre-rounding error is below
    `delta` (fp32 accumulation, fp32 tanh), and the two choices lead to different
    outputs.  This function branches on those values, layer by layer: for hidden layer 1
    both roundings of each ambiguous value; for each such choice, hidden layer 2 exactly,
    again branching on its ambiguous values.  Values whose two candidate roundings are
    less than 8 delta apart (tiny activations, whose bf16 spacing is below the error
    bound) are not branched on: any choice moves them by at most ~9 delta, which the
    caller's tolerance absorbs.  The observation itself is an exact input.

    Returns (y, cands): y [n_out, n] the plain forward (every rounding to nearest), and
    cands {column: array [n_out, k]} with all k valid outputs of each column that has an
    ambiguous value (at most 2^max_amb per layer; more raises)."""
    W = [bf16_bits_to_f64(net[f"W{i}"]) for i in (1, 2, 3)]
    b = [np.asarray(net[f"b{i}"], np.float32).astype(np.float64) for i in (1, 2, 3)]

    def split(h):
        q, lo, hi = bf16_round(h), bf16_round(h - delta), bf16_round(h + delta)
        return q, lo, hi, np.abs(hi - lo) > 8.0 * delta

    x0 = bf16_round(obs)
    h1q, lo1, hi1, amb1 = split(np.tanh(W[0] @ x0 + b[0][:, None]))
    z2 = W[1] @ h1q + b[1][:, None]                    # pre-activation of layer 2
    h2q, lo2, hi2, amb2 = split(np.tanh(z2))
    y = W[2] @ h2q + b[2][:, None]
    cands = {}
    for c in np.nonzero(amb1.any(axis=0) | amb2.any(axis=0))[0]:
        idx1 = np.nonzero(amb1[:, c])[0]
        if idx1.size > max_amb:
            raise ValueError(f"column {c}: {idx1.size} ambiguous hidden-1 values")
        outs = []
        for mask in range(1 << idx1.size):
            pick = np.array([(mask >> bit) & 1 for bit in range(idx1.size)], bool)
            v = np.where(pick, hi1[idx1, c], lo1[idx1, c])
            z = z2[:, c] + W[1][:, idx1] @ (v - h1q[idx1, c])     # rank-k update of W2 h1
            q, lo, hi, amb = split(np.tanh(z))
            idx2 = np.nonzero(amb)[0]
            if idx2.size > max_amb:
                raise ValueError(f"column {c}: {idx2.size} ambiguous hidden-2 values")
            base = W[2] @ q + b[2]
            for mask2 in range(1 << idx2.size):
                pick2 = np.array([(mask2 >> bit) & 1 for bit in range(idx2.size)], bool)
                v2 = np.where(pick2, hi[idx2], lo[idx2])
                outs.append(base + W[2][:, idx2] @ (v2 - q[idx2]))
        cands[int(c)] = np.stack(outs, axis=1)
    return y, cands


def nearest_valid_error(y_got: np.ndarray, obs: np.ndarray, net: dict, delta: float) -> np.ndarray:
    """Per column, the max-abs distance of y_got [n_out, n] to the nearest valid output
    of mlp_candidates (to the plain forward where no value is ambiguous)."""
    y, cands = mlp_candidates(obs, net, delta)
    err = np.max(np.abs(y_got - y), axis=0)
    for c, ys in cands.items():
        err[c] = min(err[c], np.min(np.max(np.abs(y_got[:, c:c + 1] - ys), axis=0)))
    return err
