"""The paper's own training task (oracle side, float64): 12-D error observation with an
axis-angle attitude error, 6-D normalised body-wrench action, five-term reward with an
action moving average, gravity randomisation, goal poses within +-2 m and +-60 degrees.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages: observation = body-frame position error, axis-angle attitude error between
reference and measured orientation, body linear and angular velocity (Sec. IV-B, observation
space; 12 values, not normalised); action = forces and torques in surge, sway, heave, roll,
pitch, yaw, each in [-1, 1] and scaled by F_max / tau_max (Sec. IV-B, action space, Eq. 1);
reward = r_pos + r_att + r_act + r_vel + r_act-mavg (Sec. IV-B, Eqs. 2-7); gravity randomised
per environment to stand for buoyancy variation with the centres of gravity and buoyancy
aligned (Sec. IV-C); 512-step episodes with references within [-2, 2] m and [-60, 60] degrees
(Sec. V-A).

Readings where the paper is silent (the same on both sides):
  * dynamics: the Fossen model of the other workloads (dynamics.py) with the buoyancy centre
    at the centre of gravity (r_b = 0), no current, no mass / damping randomisation; the
    gravity factor gamma scales the weight: W = gamma W0, gamma ~ U[0.95, 1.05]; or, with
    task["fluid"] == 1, the inertia-box fluid model of the paper's MJX setup (fluid.py: no
    added mass, viscous + quadratic drag on the equivalent box, task density and viscosity)
  * wrench tau = [F_max u_0:3, tau_max u_3:6], u = clip(a, -1, 1)
  * reset: p0 = 0, q0 = identity, v = omega = 0; goal position U[-2, 2]^3; goal attitude from
    Z-Y-X Euler angles (roll, pitch, yaw) each U[-60, 60] degrees, q = q_z(yaw) q_y(pitch) q_x(roll)
  * attitude error: q_err = q^* (x) q_ref (body frame), taken with a non-negative scalar part;
    axis-angle vector = angle * axis, angle = 2 atan2(|vec|, w)
  * w_act weighs the normalised torque commands u_3:6; the action average is an exponential
    moving average of past clipped actions, abar <- beta abar + (1 - beta) u after each step's
    reward, zero at an episode start
  * the constants (F_max, tau_max, weights, D, beta, gravity and angle ranges) come in a task
    dict (workloads.PAPER_TASK); every value is an fp32 number promoted exactly
  * step order as in env.py; done at ep_step == H; a done env is reset and observed afresh
"""
from __future__ import annotations

import math

import numpy as np

from . import dynamics as dyn
from . import fluid as fl
from . import mlp as mlpmod
from . import rng
from .env import _f64

MODE_EXTERNAL, MODE_RANDOM, MODE_POLICY_MEAN, MODE_POLICY_SAMPLE = 0, 1, 2, 3
FLAG_STAGGER = 8

R_POS = (-2.0, 4.0)
W_GFAC, W_PGOAL, W_EULER = 0, 12, 15                 # Philox reset words (block layout of env.py)
N_RESET_BLOCKS = 8


def quat_mul(a, b):
    """Hamilton product of quaternion columns (w, x, y, z)."""
    aw, ax, ay, az = a
    bw, bx, by, bz = b
    return np.stack([aw * bw - ax * bx - ay * by - az * bz,
                     aw * bx + ax * bw + ay * bz - az * by,
                     aw * by - ax * bz + ay * bw + az * bx,
                     aw * bz + ax * by - ay * bx + az * bw])


def euler_zyx_quat(roll, pitch, yaw):
    """q = q_z(yaw) (x) q_y(pitch) (x) q_x(roll), body -> world."""
    z = np.zeros_like(roll)
    qx = np.stack([np.cos(roll / 2), np.sin(roll / 2), z, z])
    qy = np.stack([np.cos(pitch / 2), z, np.sin(pitch / 2), z])
    qz = np.stack([np.cos(yaw / 2), z, z, np.sin(yaw / 2)])
    return quat_mul(qz, quat_mul(qy, qx))


def axis_angle_error(q, q_ref):
    """Rotation vector of q^* (x) q_ref (body frame), shortest rotation: [3, n]."""
    qc = q * np.array([1.0, -1.0, -1.0, -1.0])[:, None]
    e = quat_mul(qc, q_ref)
    e = e * np.where(e[0] < 0.0, -1.0, 1.0)[None, :]
    n = np.linalg.norm(e[1:4], axis=0)
    ang = 2.0 * np.arctan2(n, e[0])
    k = np.where(n > 0.0, ang / np.where(n > 0.0, n, 1.0), 2.0)
    return k[None, :] * e[1:4]


class Task:
    """The task constants as fp32 values promoted exactly: the gravity factor is drawn as
    lo + span u and the Euler angles as -e + (2e) u with fp32 (lo, span)."""

    def __init__(self, t: dict):
        f = lambda x: float(np.float32(x))  # noqa: E731
        self.f_max, self.tau_max = f(t["f_max"]), f(t["tau_max"])
        self.w_pos, self.w_att, self.w_act = f(t["w_pos"]), f(t["w_att"]), f(t["w_act"])
        self.w_vel, self.w_mavg, self.beta = f(t["w_vel"]), f(t["w_mavg"]), f(t["beta"])
        self.d_pos = np.asarray(t["d_pos"], np.float32).astype(np.float64)
        self.r_gfac = (t["gamma_lo"], t["gamma_span"])
        e = np.float32(t["euler_max"])
        self.r_euler = (-float(e), float(np.float32(2.0) * e))
        self.fluid = int(t.get("fluid", 0))                 # 0 Fossen, 1 inertia box (fluid.py)
        self.rho = f(t.get("density", fl.RHO_WATER))
        self.mu = f(t.get("viscosity", fl.MU_WATER))


def paper_reward(k: Task, dp, dth, om, u, abar):
    """The five reward terms of Sec. IV-B (Eqs. 2-7) summed, per env: position error weighted by
    D, attitude error (rotation vector), torque commands u_3:6, body rates and the deviation of
    the clipped action u from its moving average abar (taken before this step's update):
        r = -w_pos |D dp|^2 - w_att |dth|^2 - w_act |u_3:6|^2 - w_vel |om|^2 - w_mavg |u - abar|^2."""
    return (-k.w_pos * np.sum((k.d_pos[:, None] * dp) ** 2, axis=0) - k.w_att * np.sum(dth * dth, axis=0)
            - k.w_act * np.sum(u[3:6] ** 2, axis=0) - k.w_vel * np.sum(om * om, axis=0)
            - k.w_mavg * np.sum((u - abar) ** 2, axis=0))


class PaperEnv:
    def __init__(self, cfg: dict, vehicle: dict, task: dict):
        self.tk = Task(task)
        self.n = n = int(cfg["n_envs"])
        self.ids = np.arange(n, dtype=np.int64) + int(cfg.get("env_offset", 0))
        self.seed = int(cfg["seed"])
        self.flags = int(cfg.get("flags", 0))
        self.H = int(cfg["episode_len"])
        self.S = int(cfg["substeps"])
        self.dt = float(np.float32(cfg["dt_control"]))
        veh = dict(vehicle)
        veh["r_b"] = np.zeros(3, np.float32)
        self.veh_data = veh
        self.x = np.zeros((13, n))
        self.gfac = np.ones(n)
        self.p_goal = np.zeros((3, n))
        self.q_goal = np.zeros((4, n))
        self.abar = np.zeros((6, n))
        self.ep_step = np.zeros(n, np.int64)
        self.episode = np.zeros(n, np.int64)
        self.global_step = 0
        self.c_w = np.zeros((3, n))
        self.veh = self._vehicle()

    def _vehicle(self):
        if self.tk.fluid == 1:
            v = fl.InertiaBoxVehicle(self.veh_data, self.n, self.tk.rho, self.tk.mu)
        else:
            v = dyn.Vehicle(self.veh_data, self.n)
        v.W = _f64(self.veh_data["W"]) * self.gfac          # per-env weight [n]
        return v

    def _draw(self, idx):
        if idx.size == 0:
            return
        w = rng.words(self.seed, self.ids[idx], self.episode[idx], 0, N_RESET_BLOCKS)
        u = rng.uniform01(w)
        aff = lambda r, j: _f64(rng.affine_f32(r[0], r[1], u[j]))  # noqa: E731
        self.gfac[idx] = aff(self.tk.r_gfac, W_GFAC)
        self.p_goal[:, idx] = np.stack([aff(R_POS, W_PGOAL + i) for i in range(3)])
        e = [aff(self.tk.r_euler, W_EULER + i) for i in range(3)]
        self.q_goal[:, idx] = euler_zyx_quat(e[0], e[1], e[2])
        self.x[:, idx] = 0.0
        self.x[3, idx] = 1.0
        self.abar[:, idx] = 0.0
        self.veh = self._vehicle()

    def reset(self):
        self.episode[:] = 0
        self.ep_step[:] = (self.ids % self.H) if (self.flags & FLAG_STAGGER) else 0
        self.global_step = 0
        self._draw(np.arange(self.n))
        self.obs = self.observe()
        return self.obs

    def observe(self, x=None):
        """[dp_b (3), axis-angle error (3), v (3), omega (3)] -> [12, n]."""
        x = self.x if x is None else x
        R = dyn.rotation(x[3:7])
        dp_b = np.einsum("nji,jn->in", R, self.p_goal - x[0:3])
        dth = axis_angle_error(x[3:7], self.q_goal)
        return np.concatenate([dp_b, dth, x[7:10], x[10:13]])

    def step(self, actions):
        """actions [6, n] before clipping -> (reward [n], done [n], stats (3,), obs [12, n]);
        stats = sums of reward, done and |dp_b|."""
        k = self.tk
        u = np.clip(np.asarray(actions, np.float64), -1.0, 1.0)
        tau = np.concatenate([k.f_max * u[0:3], k.tau_max * u[3:6]])
        self.x = dyn.integrate(self.x, tau, self.veh, self.c_w, self.dt, self.S)
        self.ep_step += 1
        obs = self.observe()
        reward = paper_reward(k, obs[0:3], obs[3:6], obs[9:12], u, self.abar)
        self.abar = k.beta * self.abar + (1.0 - k.beta) * u
        done = self.ep_step == self.H
        stats = np.array([reward.sum(), float(done.sum()), np.linalg.norm(obs[0:3], axis=0).sum()])
        idx = np.nonzero(done)[0]
        if idx.size:
            self.episode[idx] += 1
            self.ep_step[idx] = 0
            self._draw(idx)
            obs[:, idx] = self.observe()[:, idx]
        self.obs = obs
        self.global_step += 1
        return reward, done, stats, obs

    def actions_for(self, mode, policy=None, external=None):
        """(a [6, n], eps [6, n] or None).  Random: action j from Philox words of the same
        counter as env.py's random actions: action c <- word 2c, action 3 + c <- word 2c + 1
        (c = 0, 1, 2).  Sample: noise of actions c and 3 + c is the Box-Muller pair of words
        (2c, 2c + 1) of the noise counter."""
        if mode == MODE_EXTERNAL:
            return np.asarray(external, np.float64), None
        if mode == MODE_RANDOM:
            a8 = rng.random_actions(self.seed, self.ids, self.global_step)
            return np.concatenate([a8[0:6:2], a8[1:6:2]]), None
        mu = mlpmod.mlp_forward(self.obs, policy)
        if mode == MODE_POLICY_MEAN:
            return mu, None
        e8 = rng.gaussian8(self.seed, self.ids, self.global_step)
        eps = np.concatenate([e8[0:6:2], e8[1:6:2]])
        sigma = np.exp(_f64(policy["log_std"]))[:6, None]
        return mu + sigma * eps, eps

    def rollout(self, T, mode, policy=None, external=None, record_state=False):
        n = self.n
        rec = {"obs": np.zeros((12, T, n)), "act": np.zeros((6, T, n)), "logp": np.zeros((T, n)),
               "reward": np.zeros((T, n)), "done": np.zeros((T, n)), "stats": np.zeros((3, T))}
        if record_state:
            rec["traj_state"] = np.zeros((13, T + 1, n))
            rec["traj_state"][:, 0] = self.x
        for t in range(T):
            a, eps = self.actions_for(mode, policy, None if external is None else external[t])
            rec["obs"][:, t] = self.obs
            rec["act"][:, t] = a
            if eps is not None:
                ls = _f64(policy["log_std"])[:6, None]
                rec["logp"][t] = np.sum(-0.5 * eps * eps - ls - 0.5 * math.log(2 * math.pi), axis=0)
            r, d, s, _ = self.step(a)
            rec["reward"][t], rec["done"][t], rec["stats"][:, t] = r, d, s
            if record_state:
                rec["traj_state"][:, t + 1] = self.x
        return rec

    def load(self, state, gfac, p_goal, q_goal, ep_step, episode, abar):
        """Overwrite the env with fp32 buffers (exact promotion)."""
        self.x = _f64(state).copy()
        self.gfac = _f64(gfac).copy()
        self.p_goal = _f64(p_goal).copy()
        self.q_goal = _f64(q_goal).copy()
        self.ep_step = np.asarray(ep_step, np.int64).copy()
        self.episode = np.asarray(episode, np.int64).copy()
        self.abar = _f64(abar).copy()
        self.veh = self._vehicle()
        self.obs = self.observe()
