"""Generalised advantage estimation (oracle side).

The PPO learner the paper uses (Sec. III-A1) consumes advantages of the fresh on-policy
trajectories; GAE (Schulman et al., 2016) computes them by a backward recursion over
the rollout:
    delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t,   V_T = V(o_T) (bootstrap value)
    A_t     = delta_t + gamma lambda (1 - d_t) A_{t+1},   A_T = 0
    R_t     = A_t + V_t
An episode end (d_t = 1) cuts both the bootstrap and the recursion; the fixed episode
length is treated as terminal.
"""
from __future__ import annotations

import numpy as np


def gae(reward, value, done, last_value, gamma: float, lam: float):
    """reward, value, done [T, n]; last_value [n] -> (adv, ret) [T, n], float64."""
    r = np.asarray(reward, np.float64)
    v = np.asarray(value, np.float64)
    d = np.asarray(done, np.float64)
    T = r.shape[0]
    adv = np.zeros_like(r)
    next_v = np.asarray(last_value, np.float64)
    next_a = np.zeros(r.shape[1:])
    for t in range(T - 1, -1, -1):
        nd = 1.0 - d[t]
        delta = r[t] + gamma * nd * next_v - v[t]
        next_a = delta + gamma * lam * nd * next_a
        adv[t] = next_a
        next_v = v[t]
    return adv, adv + v
