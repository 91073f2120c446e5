"""Seeded synthetic inputs shared by the CPU oracle, the tests and the benchmark.

This module holds data only: vehicle constants, the thruster allocation table, the
five workload presets and seeded policy/value weights.  It contains none of the
method's arithmetic (no dynamics, no random-draw maps, no network evaluation), so the
oracle and the HIP path can both take their inputs from here without sharing code.

Vehicle numbers: the 6-DOF vehicle used by the benchmark workloads (mass, inertia,
added mass, linear and quadratic damping, weight, buoyancy, centre of buoyancy 0.02 m
above the centre of gravity, 8 thrusters of at most 40 N).  The paper names its vehicle
(a BlueROV2 Heavy) and says thrust commands reach the thrusters through an allocation
matrix (Sec. V-B, real-world experiments) but gives neither the geometry nor the
matrix, so the thruster geometry below is this project's constant.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "VEHICLE", "THRUSTER_POS", "THRUSTER_DIR", "ALLOC", "EPISODE_LEN",
    "FLAG_DR", "FLAG_CURRENT", "FLAG_LISSAJOUS", "FLAG_STAGGER", "FLAG_TRAJ_STATE",
    "MODE_EXTERNAL", "MODE_RANDOM", "MODE_POLICY_MEAN", "MODE_POLICY_SAMPLE",
    "CONFIGS", "config", "mlp_weights", "vehicle_variant", "random_states",
    "PPO", "ppo_draws", "ppo_minibatch_idx", "PAPER_TASK", "PAPER_TASK_BOX", "SHAC",
]

# --- vehicle (fp32 values; every consumer promotes them exactly) -------------------
# The body frame has its origin at the centre of gravity, so r_g = 0 by construction.
VEHICLE = {
    "m": np.float32(11.5),
    "inertia": np.array([0.16, 0.16, 0.16], np.float32),
    "added_mass": np.array([5.5, 12.7, 14.6, 0.12, 0.12, 0.12], np.float32),
    "lin_damp": np.array([4.0, 6.2, 5.2, 0.07, 0.07, 0.07], np.float32),
    "quad_damp": np.array([18.2, 21.7, 37.0, 1.5, 1.5, 1.5], np.float32),
    "W": np.float32(112.8),
    "B": np.float32(114.8),
    # body frame is forward-right-down, so "0.02 m above the CoG" is -z
    "r_b": np.array([0.0, 0.0, -0.02], np.float32),
    "f_max": np.float32(40.0),
}

# --- thruster geometry (project constant, FRD body frame, metres) ------------------
# Four horizontal thrusters at 45 degrees in the x-y plane, four vertical thrusters.
_C45 = 0.70710678118654752
THRUSTER_POS = np.array([
    [0.156, 0.111, 0.0], [0.156, -0.111, 0.0], [-0.156, 0.111, 0.0], [-0.156, -0.111, 0.0],
    [0.120, 0.218, 0.0], [0.120, -0.218, 0.0], [-0.120, 0.218, 0.0], [-0.120, -0.218, 0.0],
], np.float64)
THRUSTER_DIR = np.array([
    [_C45, -_C45, 0.0], [_C45, _C45, 0.0], [_C45, _C45, 0.0], [_C45, -_C45, 0.0],
    [0.0, 0.0, 1.0], [0.0, 0.0, 1.0], [0.0, 0.0, 1.0], [0.0, 0.0, 1.0],
], np.float64)

# 6x8 allocation table, row-major, rows = (X, Y, Z, K, M, N), column i = [d_i ; r_i x d_i].
# Written out as literals (the geometry above is the documentation; a test re-derives it).
_Y = 0.18879751  # 0.267 * cos(45 deg)
ALLOC = np.array([
    [_C45, _C45, _C45, _C45, 0.0, 0.0, 0.0, 0.0],
    [-_C45, _C45, _C45, -_C45, 0.0, 0.0, 0.0, 0.0],
    [0.0, 0.0, 0.0, 0.0, 1.0, 1.0, 1.0, 1.0],
    [0.0, 0.0, 0.0, 0.0, 0.218, -0.218, 0.218, -0.218],
    [0.0, 0.0, 0.0, 0.0, -0.120, -0.120, 0.120, 0.120],
    [-_Y, _Y, -_Y, _Y, 0.0, 0.0, 0.0, 0.0],
], np.float32)

EPISODE_LEN = 500

# --- flags and action modes (same values as the C header) -------------------------
FLAG_DR = 1           # per-env mass / added-mass / damping scales at reset
FLAG_CURRENT = 2      # per-env constant ocean current at reset
FLAG_LISSAJOUS = 4    # per-env Lissajous position reference plus yaw ramp
FLAG_STAGGER = 8      # initial episode step of env i is i mod episode length
FLAG_TRAJ_STATE = 16  # record the state trajectory in rollouts

MODE_EXTERNAL = 0
MODE_RANDOM = 1
MODE_POLICY_MEAN = 2
MODE_POLICY_SAMPLE = 3

# --- the five workloads ------------------------------------------------------------
# c1 small parity case; c2 randomised open loop; c3 closed loop with the policy;
# c4 the headline: 16384 envs, 4 RK4 substeps per 0.04 s control step, Lissajous
# references; c5 PPO rollout of 65536 envs x 64 steps plus GAE.
CONFIGS = {
    "c1": dict(name="c1", n_envs=64, T=200, substeps=1, dt_control=0.02, seed=1,
               flags=0, mode=MODE_RANDOM, policy=False, value=False),
    "c2": dict(name="c2", n_envs=4096, T=1000, substeps=1, dt_control=0.02, seed=2,
               flags=FLAG_DR | FLAG_CURRENT, mode=MODE_RANDOM, policy=False, value=False),
    "c3": dict(name="c3", n_envs=4096, T=1000, substeps=1, dt_control=0.02, seed=3,
               flags=FLAG_DR | FLAG_CURRENT, mode=MODE_POLICY_MEAN, policy=True, value=False),
    "c4": dict(name="c4", n_envs=16384, T=2000, substeps=4, dt_control=0.04, seed=4,
               flags=FLAG_DR | FLAG_CURRENT | FLAG_LISSAJOUS, mode=MODE_POLICY_MEAN,
               policy=True, value=False),
    "c5": dict(name="c5", n_envs=65536, T=64, substeps=1, dt_control=0.02, seed=5,
               flags=FLAG_DR | FLAG_CURRENT | FLAG_STAGGER, mode=MODE_POLICY_SAMPLE,
               policy=True, value=True, gamma=0.99, lam=0.95),
}
# c6: the paper's own training task (12-D observation, 6-D wrench, five-term reward, gravity
# randomisation) at the paper's training scale: 4096 envs, one 512-step episode.
CONFIGS["c6"] = dict(name="c6", n_envs=4096, T=512, substeps=2, dt_control=0.05, seed=6, flags=0,
                     mode=MODE_POLICY_MEAN, policy=True, value=False, episode_len=512)

for _c in CONFIGS.values():
    _c.setdefault("episode_len", EPISODE_LEN)
    _c.setdefault("env_offset", 0)

POLICY_SEED = 7
VALUE_SEED = 8
LOG_STD = -0.5
OBS_DIM, ACT_DIM, HIDDEN = 23, 8, 256


def config(name: str, **overrides) -> dict:
    """A copy of a preset with fields overridden (e.g. a smaller n_envs or T)."""
    c = dict(CONFIGS[name])
    c.update(overrides)
    return c


def vehicle_variant(**overrides) -> dict:
    """A copy of VEHICLE with selected fields replaced (fp32), for closed-form cases."""
    v = {k: (np.array(x, np.float32) if np.ndim(x) else np.float32(x)) for k, x in VEHICLE.items()}
    for k, x in overrides.items():
        v[k] = np.array(x, np.float32) if np.ndim(x) else np.float32(x)
    return v


def mlp_weights(n_out: int, seed: int, n_in: int = OBS_DIM, hidden: int = HIDDEN) -> dict:
    """Seeded MLP parameters n_in -> hidden -> hidden -> n_out.

    Weights: N(0, 1/fan_in) from NumPy PCG64, rounded fp64 -> fp32 -> bf16 (round to
    nearest even, by torch's conversion).  Returned as uint16 bf16 bit patterns in
    PyTorch Linear layout W[out][in], row-major.  Biases: U[-0.1, 0.1] in fp32.
    log_std: -0.5 for every action dimension.
    """
    import torch

    rng = np.random.Generator(np.random.PCG64(seed))
    shapes = [(hidden, n_in), (hidden, hidden), (n_out, hidden)]
    out = {}
    for i, (o, k) in enumerate(shapes, start=1):
        w = rng.standard_normal((o, k)) / math.sqrt(k)
        wb = torch.from_numpy(w.astype(np.float32)).to(torch.bfloat16)
        out[f"W{i}"] = wb.view(torch.int16).numpy().view(np.uint16).copy()
    for i, o in enumerate([hidden, hidden, n_out], start=1):
        out[f"b{i}"] = rng.uniform(-0.1, 0.1, size=o).astype(np.float32)
    out["log_std"] = np.full(ACT_DIM, LOG_STD, np.float32)
    out["n_in"], out["hidden"], out["n_out"] = n_in, hidden, n_out
    return out


def random_states(n: int, seed: int, pos_scale=2.0, vel_scale=1.0, rate_scale=1.0) -> np.ndarray:
    """Seeded fp32 states [13][n] (p, unit q, v, w) for one-step parity cases."""
    rng = np.random.Generator(np.random.PCG64(seed))
    p = rng.uniform(-pos_scale, pos_scale, (3, n))
    q = rng.standard_normal((4, n))
    q /= np.linalg.norm(q, axis=0, keepdims=True)
    v = rng.uniform(-vel_scale, vel_scale, (3, n))
    w = rng.uniform(-rate_scale, rate_scale, (3, n))
    return np.concatenate([p, q, v, w]).astype(np.float32)


# --- PPO update workload -----------------------------------------------------------
# One update epoch over a c5-sized rollout buffer (65536 envs x 64 steps = 4194304 samples)
# in 16 minibatches of 262144; hyperparameters of common PPO practice (the paper gives none).
PPO = dict(M=65536 * 64, B=262144, epochs=4, clip_eps=0.2, vf_coef=0.5, ent_coef=0.0,
           max_grad_norm=0.5, lr=3e-4, beta1=0.9, beta2=0.999, adam_eps=1e-8, normalize_adv=True)


def ppo_draws(M: int, seed: int) -> dict:
    """Seeded raw draws for a synthetic rollout buffer of M samples: observations with the
    ranges of the environment's rows (body-frame position error, rotation columns,
    velocities, previous action), standard-normal action noise, advantages, returns, and
    target probability ratios in [0.6, 1.4] kept 0.03 away from 0.8 and 1.2 (so that a
    clipping decision never sits at a boundary).  The caller forms actions and old
    log-probabilities from these with its own policy evaluation."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lo = np.array([-3.0] * 3 + [-1.0] * 6 + [-1.0] * 3 + [-1.5] * 3 + [-1.0] * 8)
    obs = rng.uniform(lo[:, None], -lo[:, None], (23, M)).astype(np.float32)
    eps = rng.standard_normal((8, M))
    adv = (2.0 * rng.standard_normal(M) + 0.3).astype(np.float32)
    ret = rng.standard_normal(M).astype(np.float32)
    ratio = rng.uniform(0.6, 1.4, M)
    near = (np.abs(ratio - 0.8) < 0.03) | (np.abs(ratio - 1.2) < 0.03)
    ratio[near] = 1.0 + 0.5 * (ratio[near] - 1.0)
    return dict(obs=obs, eps=eps, adv=adv, ret=ret, ratio=ratio)


def ppo_minibatch_idx(M: int, B: int, seed: int) -> np.ndarray:
    """B sample indices: a seeded permutation of the buffer's 16-sample blocks (16
    consecutive envs of one step), cut to B entries (int32)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    blocks = rng.permutation(M // 16)
    idx = (blocks[:, None] * 16 + np.arange(16)[None, :]).ravel()
    return idx[:B].astype(np.int32)


# --- the paper task's constants (Sec. IV-B / IV-C; the values the paper leaves open are this
# project's choice: wrench limits within the thrusters' envelope, reward weights) -----------
PAPER_TASK = dict(kind=1, f_max=60.0, tau_max=10.0, w_pos=1.0, d_pos=(1.0, 1.0, 1.5), w_att=0.5,
                  w_act=0.01, w_vel=0.05, w_mavg=0.1, beta=0.8, gamma_lo=0.95, gamma_span=0.1,
                  euler_max=float(np.float32(math.pi / 3.0)), fluid=0, density=1000.0, viscosity=1.0e-3)
# The same task with the hydrodynamics of the paper's MJX simulation (Sec. IV-B): the
# inertia-box fluid model in water (density 1000 kg/m^3, viscosity 1.0e-3 Pa s).
PAPER_TASK_BOX = dict(PAPER_TASK, fluid=1)
PAPER_POLICY_SEED = 9
PAPER_VALUE_SEED = 10

# --- SHAC on the paper task ----------------------------------------------------------
# Short-horizon actor-critic windows (the differentiable-simulation learner of the paper):
# h = 32 control steps per window (16 windows per 512-step episode), discount 0.99, the
# actor gradient clipped to norm 1; the paper's best SHAC scale is 512 environments and its
# main experiments use 4096.
SHAC = dict(h=32, gamma=0.99, max_grad_norm=1.0, n_envs=4096, n_envs_small=512)
