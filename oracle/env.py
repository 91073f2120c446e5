"""Batched environment: reset / domain randomisation, references, observation, reward,
auto-reset, batch statistics and rollouts (oracle side, float64).

Paper passages: many independent environments in one batch, each with its own random
initial conditions and randomisation parameters (Sec. IV-A); the error-based
observation in the body frame with body velocities (Sec. IV-B), here in its 23-value
form with two columns of the error rotation matrix (the rotation-matrix attitude error
converged fastest, Sec. V-A) and the previous action; the reward shape of Sec. IV-B
(Eqs. 2-5: position error, attitude error, action effort), here -|dp| - 0.5 theta - 0.01 |u|^2;
a random reference per episode (Sec. V-A); fixed-length episodes with automatic reset.

Step order for env i at control step t (the paper gives none; this is the reading):
  1. action a (caller's, Philox uniform, or policy mean / sample); u = clip(a, -1, 1);
     thrust f = f_max u; body wrench tau = T f (6x8 allocation table)
  2. S RK4 substeps of dt / S with tau held
  3. ep_step += 1; reference at t_ep = ep_step * dt
  4. observation o = [R^T (p_ref - p), R_err[:,0], R_err[:,1], v, omega, u], R_err = R^T R_ref
  5. reward r = -|R^T (p_ref - p)| - 0.5 theta_err - 0.01 |u|^2, theta_err the angle of R_err
  6. done = (ep_step == H); a done env starts its next episode (episode += 1, fresh
     reset draws, ep_step = 0, previous action 0) and its observation is the reset one
  7. batch statistics: sum over envs of r, done and |dp| (before any reset)
"""
from __future__ import annotations

import math

import numpy as np

from . import dynamics as dyn
from . import mlp as mlpmod
from . import rng

# Flag bits and action modes (values fixed by the C interface).
FLAG_DR, FLAG_CURRENT, FLAG_LISSAJOUS, FLAG_STAGGER, FLAG_TRAJ_STATE = 1, 2, 4, 8, 16
MODE_EXTERNAL, MODE_RANDOM, MODE_POLICY_MEAN, MODE_POLICY_SAMPLE = 0, 1, 2, 3

F32_2PI = float(np.float32(2.0 * math.pi))
F32_PI = float(np.float32(math.pi))

# Reset draw map: word index -> (lo, span) of an fp32 affine draw lo + span*u.
# Ranges: mass / added mass / damping scales U[0.8, 1.2]; current U[-0.3, 0.3] m/s per
# axis; positions U[-2, 2] m (the paper's reference range, Sec. V-A); Lissajous
# amplitude U[0.5, 2] m, frequency U[0.02, 0.1] Hz, phase U[0, 2 pi); yaw rate
# U[-0.1, 0.1] rad/s; initial reference yaw U[-pi, pi).
R_SCALE = (0.8, 0.4)
R_CURRENT = (-0.3, 0.6)
R_POS = (-2.0, 4.0)
R_AMP = (0.5, 1.5)
R_FREQ = (0.02, 0.08)
R_PHASE = (0.0, F32_2PI)
R_YAWRATE = (-0.1, 0.2)
R_YAW0 = (-F32_PI, F32_2PI)
W_SCALE, W_CURRENT, W_P0, W_Q0, W_PGOAL, W_QGOAL = 0, 3, 6, 9, 12, 15
W_AMP, W_FREQ, W_PHASE, W_YAWRATE, W_YAW0 = 18, 21, 24, 27, 28
N_RESET_BLOCKS = 8          # 32 words per reset, always all drawn


def _f64(x):
    return np.asarray(x, np.float32).astype(np.float64)


def quat_mul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Hamilton product a (x) b of quaternions [4, n] written with the matrix L(a) b."""
    w, x, y, z = a
    L = np.array([[w, -x, -y, -z],
                  [x, w, -z, y],
                  [y, z, w, -x],
                  [z, -y, x, w]])              # [4, 4, n]
    return np.einsum("ijn,jn->in", L, b)


def rotation_angle(Rm: np.ndarray) -> np.ndarray:
    """Geodesic angle in [0, pi] of rotation matrices [n, 3, 3]:
    atan2(|axial(R - R^T)| / 2, (tr R - 1) / 2)."""
    ax = np.stack([Rm[:, 2, 1] - Rm[:, 1, 2], Rm[:, 0, 2] - Rm[:, 2, 0], Rm[:, 1, 0] - Rm[:, 0, 1]])
    s = 0.5 * np.linalg.norm(ax, axis=0)
    c = 0.5 * (np.trace(Rm, axis1=1, axis2=2) - 1.0)
    return np.arctan2(s, c)


class Env:
    """N environments in float64.  State arrays are [k, n] (component, env)."""

    def __init__(self, cfg: dict, vehicle: dict, alloc: np.ndarray):
        self.cfg = dict(cfg)
        self.n = int(cfg["n_envs"])
        self.ids = np.arange(self.n, dtype=np.int64) + int(cfg.get("env_offset", 0))
        self.seed = int(cfg["seed"])
        self.flags = int(cfg["flags"])
        self.H = int(cfg["episode_len"])
        self.S = int(cfg["substeps"])
        self.dt = float(np.float32(cfg["dt_control"]))   # the control period is an fp32 input
        self.veh_data = vehicle
        self.alloc = _f64(alloc)                   # [6, 8]
        self.f_max = float(_f64(vehicle["f_max"]))
        n = self.n
        self.x = np.zeros((13, n))
        self.scales = np.ones((3, n))
        self.c_w = np.zeros((3, n))
        self.p_goal = np.zeros((3, n))
        self.q_goal = np.zeros((4, n))
        self.amp = np.zeros((3, n))
        self.freq = np.zeros((3, n))
        self.phase = np.zeros((3, n))
        self.yaw_rate = np.zeros(n)
        self.yaw0 = np.zeros(n)
        self.ep_step = np.zeros(n, np.int64)
        self.episode = np.zeros(n, np.int64)
        self.u_prev = np.zeros((8, n))
        self.obs = np.zeros((23, n))
        self.global_step = 0
        self.veh = dyn.Vehicle(vehicle, n)

    # ---- reset --------------------------------------------------------------------
    def _draw(self, idx: np.ndarray):
        """Reset draws (tag 0, counter word 1 = episode) for envs idx."""
        if idx.size == 0:
            return
        w = rng.words(self.seed, self.ids[idx], self.episode[idx], rng.TAG_RESET, N_RESET_BLOCKS)
        u = rng.uniform01(w)                       # [32, k]
        aff = lambda r, j: _f64(rng.affine_f32(r[0], r[1], u[j]))  # noqa: E731
        if self.flags & FLAG_DR:
            self.scales[:, idx] = np.stack([aff(R_SCALE, W_SCALE + i) for i in range(3)])
        else:
            self.scales[:, idx] = 1.0
        if self.flags & FLAG_CURRENT:
            self.c_w[:, idx] = np.stack([aff(R_CURRENT, W_CURRENT + i) for i in range(3)])
        else:
            self.c_w[:, idx] = 0.0
        p0 = np.stack([aff(R_POS, W_P0 + i) for i in range(3)])
        q0 = rng.shoemake(u[W_Q0], u[W_Q0 + 1], u[W_Q0 + 2])
        self.p_goal[:, idx] = np.stack([aff(R_POS, W_PGOAL + i) for i in range(3)])
        self.q_goal[:, idx] = rng.shoemake(u[W_QGOAL], u[W_QGOAL + 1], u[W_QGOAL + 2])
        self.amp[:, idx] = np.stack([aff(R_AMP, W_AMP + i) for i in range(3)])
        self.freq[:, idx] = np.stack([aff(R_FREQ, W_FREQ + i) for i in range(3)])
        self.phase[:, idx] = np.stack([aff(R_PHASE, W_PHASE + i) for i in range(3)])
        self.yaw_rate[idx] = aff(R_YAWRATE, W_YAWRATE)
        self.yaw0[idx] = aff(R_YAW0, W_YAW0)
        self.x[:, idx] = np.concatenate([p0, q0, np.zeros((6, idx.size))])
        self.u_prev[:, idx] = 0.0
        self.veh = dyn.Vehicle(self.veh_data, self.n, *self.scales)

    def reset(self):
        """Reset every env: episode 0 (ep_step = global id mod H with STAGGER, else 0),
        draws, observation; global step back to 0."""
        self.episode[:] = 0
        self.ep_step[:] = (self.ids % self.H) if (self.flags & FLAG_STAGGER) else 0
        self.global_step = 0
        self._draw(np.arange(self.n))
        self.obs = self.observe()[0]
        return self.obs

    # ---- reference, observation, reward --------------------------------------------
    def reference(self, ep_step=None):
        """(p_ref [3, n], q_ref [4, n]) at t = ep_step * dt.  Lissajous: p_goal +
        A sin(2 pi f t + phi) and a level yaw-only attitude psi0 + psi_dot t; otherwise
        the episode's goal pose."""
        if not (self.flags & FLAG_LISSAJOUS):
            return self.p_goal.copy(), self.q_goal.copy()
        t = (self.ep_step if ep_step is None else ep_step) * self.dt
        p_ref = self.p_goal + self.amp * np.sin(2.0 * math.pi * self.freq * t + self.phase)
        psi = self.yaw0 + self.yaw_rate * t
        z = np.zeros_like(psi)
        q_ref = np.stack([np.cos(0.5 * psi), z, z, np.sin(0.5 * psi)])
        return p_ref, q_ref

    def observe(self, x=None, u_prev=None):
        """Observation [23, n] plus (|dp|, theta_err) of state x against the reference."""
        x = self.x if x is None else x
        u_prev = self.u_prev if u_prev is None else u_prev
        p_ref, q_ref = self.reference()
        R = dyn.rotation(x[3:7])                                   # [n, 3, 3]
        R_ref = dyn.rotation(q_ref)
        dp_b = np.einsum("nji,jn->in", R, p_ref - x[0:3])          # R^T (p_ref - p)
        R_err = np.transpose(R, (0, 2, 1)) @ R_ref
        obs = np.concatenate([dp_b, R_err[:, :, 0].T, R_err[:, :, 1].T, x[7:10], x[10:13], u_prev])
        return obs, np.linalg.norm(dp_b, axis=0), rotation_angle(R_err)

    # ---- one control step ------------------------------------------------------------
    def step(self, actions: np.ndarray):
        """Advance every env by one control step with actions [8, n] (before clipping).
        Returns (reward [n], done bool [n], stats (3,), obs after any reset [23, n])."""
        u = np.clip(actions, -1.0, 1.0)
        tau = self.alloc @ (self.f_max * u)                          # [6, n]
        self.x = dyn.integrate(self.x, tau, self.veh, self.c_w, self.dt, self.S)
        self.ep_step += 1
        self.u_prev = u
        obs, dp, theta = self.observe()
        reward = -dp - 0.5 * theta - 0.01 * np.sum(u * u, axis=0)
        done = self.ep_step == self.H
        stats = np.array([reward.sum(), float(done.sum()), dp.sum()])
        idx = np.nonzero(done)[0]
        if idx.size:
            self.episode[idx] += 1
            self.ep_step[idx] = 0
            self._draw(idx)
            obs[:, idx] = self.observe()[0][:, idx]
        self.obs = obs
        self.global_step += 1
        return reward, done, stats, obs

    def actions_for(self, mode, policy=None, external=None):
        """Action for the current step: (a [8, n], eps [8, n] or None)."""
        if mode == MODE_EXTERNAL:
            return np.asarray(external, np.float64), None
        if mode == MODE_RANDOM:
            return rng.random_actions(self.seed, self.ids, self.global_step), None
        mu = mlpmod.mlp_forward(self.obs, policy)
        if mode == MODE_POLICY_MEAN:
            return mu, None
        eps = rng.gaussian8(self.seed, self.ids, self.global_step)
        sigma = np.exp(_f64(policy["log_std"]))[:, None]
        return mu + sigma * eps, eps

    def rollout(self, T: int, mode: int, policy=None, value=None, external=None,
                record_state: bool = False):
        """T control steps.  external: actions [T, 8, n] for MODE_EXTERNAL.  Returns a dict
        of per-step records: obs [23, T, n] (the observation each action was chosen on),
        act [8, T, n], logp/value/reward/done [T, n], last_value [n], stats [3, T],
        traj_state [13, T+1, n] (if record_state)."""
        n = self.n
        rec = {k: np.zeros((T, n)) for k in ("logp", "value", "reward", "done")}
        rec["obs"] = np.zeros((23, T, n))
        rec["act"] = np.zeros((8, T, n))
        rec["stats"] = np.zeros((3, T))
        if record_state:
            rec["traj_state"] = np.zeros((13, T + 1, n))
            rec["traj_state"][:, 0] = self.x
        for t in range(T):
            a, eps = self.actions_for(mode, policy, None if external is None else external[t])
            rec["obs"][:, t] = self.obs
            rec["act"][:, t] = a
            if eps is not None:
                rec["logp"][t] = mlpmod.gaussian_logp(eps, policy["log_std"])
            if value is not None:
                rec["value"][t] = mlpmod.mlp_forward(self.obs, value)[0]
            r, d, s, _ = self.step(a)
            rec["reward"][t], rec["done"][t], rec["stats"][:, t] = r, d, s
            if record_state:
                rec["traj_state"][:, t + 1] = self.x
        if value is not None:
            rec["last_value"] = mlpmod.mlp_forward(self.obs, value)[0]
        return rec

    # ---- state exchange with fp32 buffers (for one-step and teacher-forced checks) ---
    def params_f32(self) -> np.ndarray:
        """Per-env parameters [24, n] in the C interface's order: s_m, s_a, s_d, c_w(3),
        p_goal(3), q_goal(4), A(3), f(3), phi(3), psi_dot, psi0."""
        return np.concatenate([self.scales, self.c_w, self.p_goal, self.q_goal, self.amp,
                               self.freq, self.phase, self.yaw_rate[None], self.yaw0[None]]
                              ).astype(np.float32)

    def load(self, state, params, ep_step, episode, u_prev):
        """Overwrite the env with fp32 buffers (exact promotion to float64)."""
        state = _f64(state)
        params = _f64(params)
        self.x = state.copy()
        self.scales = params[0:3].copy()
        self.c_w = params[3:6].copy()
        self.p_goal = params[6:9].copy()
        self.q_goal = params[9:13].copy()
        self.amp = params[13:16].copy()
        self.freq = params[16:19].copy()
        self.phase = params[19:22].copy()
        self.yaw_rate = params[22].copy()
        self.yaw0 = params[23].copy()
        self.ep_step = np.asarray(ep_step, np.int64).copy()
        self.episode = np.asarray(episode, np.int64).copy()
        self.u_prev = _f64(u_prev).copy()
        self.veh = dyn.Vehicle(self.veh_data, self.n, *self.scales)
        self.obs = self.observe()[0]
