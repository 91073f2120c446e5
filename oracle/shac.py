"""SHAC actor objective over a short window of the paper task, and its gradient (oracle
side, float64).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages: the differentiable-simulation learner SHAC (Sec. III-A3, Xu et al.'s
Short-Horizon Actor-Critic, which the paper cites) backpropagates through the dynamics
over short sub-trajectories and closes each of them with the critic's estimate of the
remaining return; the paper trains it on its own task (Sec. IV-B, IV-C, V-A), whose
step is written out in paper_task.py.

Actor objective of one window (SHAC's actor loss): N environments, h control steps from
states s_0, discount gamma,
    L = -(1 / (N h)) sum_i [ sum_{t < h} gamma^t r_t^i + gamma^h V(o(s_h^i)) ]
    a_t = mu(o_t) + sigma eps_t   (reparameterised Gaussian policy, sigma = exp(log_std);
                                   eps_t from the Philox noise stream of the rollouts)
    u_t = clip(a_t, -1, 1),  s_{t+1} = RK4 step of the paper task under wrench(u_t),
    r_t = five-term reward of (o(s_{t+1}), u_t, abar_t),  abar_{t+1} = beta abar_t + (1 - beta) u_t
With external actions (mode EXTERNAL) a_t is an input and no policy is evaluated.

The gradient is reverse-mode differentiation of exactly this forward: torch autograd on
float64 CPU tensors (a library primitive), with the two rounding operators below as the
only hand-written derivative rules.  The physics is written out in the textbook matrix
forms of dynamics.py (6x6 mass, Coriolis and damping matrices, a linear solve), batched
over environments in torch.

Readings (the paper is silent; the device path takes the same):
  * a window never crosses an episode end: its last step may end the episode, and then the
    terminal value is taken on the state before the reset (the time limit truncates the
    return, it does not end it)
  * clip: the derivative of clip(a, -1, 1) is 1 for -1 <= a <= 1 (ends included), else 0
  * |x| in the quadratic damping: derivative sign(x), 0 at x = 0
  * bf16 quantisation points, those of a bf16 MFMA implementation: in the forward, the
    input of every layer is rounded to bf16 (mlp.mlp_forward), passed straight through in
    the backward; in the backward, the cotangent of every layer's pre-activation is rounded
    to bf16 before it reaches that layer's weights, bias and input (dW3 = q(gy) q(h2)^T,
    db3 = sum q(gy), dh2 = W3^T q(gy), dz2 = dh2 (1 - h2^2) with the unrounded h2,
    dW2 = q(dz2) q(h1)^T, db2 = sum q(dz2), dh1 = W2^T q(dz2), dz1 = dh1 (1 - h1^2),
    dW1 = q(dz1) q(o)^T, db1 = sum q(dz1), do = W1^T q(dz1)).  With quantize=False both
    operators are the identity.
  * the terminal value is differentiated the same way; the value net's own parameters are
    not trained by this objective (SHAC fits the critic separately)

Teacher forcing (window(..., forced=...)): a closed-loop window's trajectory is not unique
under bf16 rounding (a hidden value within rounding error of a bf16 midpoint may round either
way), so two correct implementations drift apart over a long window.  Given a trajectory
(the states after each step and the actions taken), the forward replaces each state and
action by the given value while keeping its derivative, x <- x + (x_given - x) held constant
in the backward.  The result is the same objective's gradient linearised along the given
trajectory; with the oracle's own trajectory it is the plain gradient.
"""
from __future__ import annotations

import numpy as np
import torch

from . import rng
from .mlp import bf16_bits_to_f64, bf16_round

MODE_EXTERNAL, MODE_POLICY_MEAN, MODE_POLICY_SAMPLE = 0, 2, 3
DT = torch.float64


def _t(x) -> torch.Tensor:
    return torch.as_tensor(np.asarray(x, np.float64), dtype=DT)


def _f32(x) -> float:
    return float(np.float32(x))


# ---- the two rounding operators -------------------------------------------------------
class _RoundForward(torch.autograd.Function):
    """Forward: round to the nearest bf16 value (ties to even); backward: identity."""

    @staticmethod
    def forward(ctx, x):
        return torch.from_numpy(bf16_round(x.detach().numpy()))

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundCotangent(torch.autograd.Function):
    """Forward: identity; backward: the incoming cotangent rounded to bf16."""

    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return torch.from_numpy(bf16_round(g.detach().numpy()))


def _ident(x):
    return x


# ---- networks ------------------------------------------------------------------------
def net_params(net: dict, n_out: int, requires_grad: bool = False) -> dict:
    """Parameter dict of a workloads MLP as float64 tensors (W from bf16 bits, b fp32):
    W1 [H][n_in], W2 [H][H], W3 [n_out][H], b1, b2, b3 and (policy) log_std [n_out]."""
    p = {k: _t(bf16_bits_to_f64(net[k])) for k in ("W1", "W2", "W3")}
    p.update({k: _t(np.asarray(net[k], np.float32)) for k in ("b1", "b2", "b3")})
    p["W3"], p["b3"] = p["W3"][:n_out], p["b3"][:n_out]
    if "log_std" in net:
        p["log_std"] = _t(np.asarray(net["log_std"], np.float32)[:n_out])
    for v in p.values():
        v.requires_grad_(requires_grad)
    return p


def mlp(x: torch.Tensor, p: dict, quantize: bool) -> torch.Tensor:
    """y = W3 q(h2) + b3, h2 = tanh(W2 q(h1) + b2), h1 = tanh(W1 q(x) + b1) for x [n_in, n],
    with the cotangent rounding on every pre-activation (module docstring)."""
    q = _RoundForward.apply if quantize else _ident
    gq = _RoundCotangent.apply if quantize else _ident
    h1 = torch.tanh(gq(p["W1"] @ q(x) + p["b1"][:, None]))
    h2 = torch.tanh(gq(p["W2"] @ q(h1) + p["b2"][:, None]))
    return gq(p["W3"] @ q(h2) + p["b3"][:, None])


# ---- physics (dynamics.py's forms, in torch, no current, buoyancy centre at the CoG) ------
def skew(a: torch.Tensor) -> torch.Tensor:
    """S(a) with S(a) b = a x b; a [n, 3] -> [n, 3, 3]."""
    z = torch.zeros_like(a[:, 0])
    return torch.stack([torch.stack([z, -a[:, 2], a[:, 1]], 1),
                        torch.stack([a[:, 2], z, -a[:, 0]], 1),
                        torch.stack([-a[:, 1], a[:, 0], z], 1)], 1)


def rotation(q: torch.Tensor) -> torch.Tensor:
    """R(q) = I + 2 eta S(eps) + 2 S(eps)^2; q [4, n] -> [n, 3, 3]."""
    s = skew(q[1:4].T)
    return torch.eye(3, dtype=DT)[None] + 2.0 * q[0][:, None, None] * s + 2.0 * s @ s


class Vehicle:
    """The paper task's vehicle: workloads constants promoted exactly, weight gamma W per
    environment (gfac [n]), centre of buoyancy at the centre of gravity."""

    def __init__(self, veh: dict, gfac):
        f = lambda x: _t(np.asarray(x, np.float32))  # noqa: E731
        gfac = _t(gfac)
        n = gfac.shape[0]
        m, inertia, ma = f(veh["m"]), f(veh["inertia"]), f(veh["added_mass"])
        self.m = m.expand(n)
        self.inertia = inertia[None, :].expand(n, 3)
        self.ma = ma[None, :].expand(n, 6)
        rb = torch.cat([m.expand(3), inertia])
        self.M = torch.diag_embed((rb + ma)[None, :].expand(n, 6))
        self.D_L = f(veh["lin_damp"])[None, :].expand(n, 6)
        self.D_Q = f(veh["quad_damp"])[None, :].expand(n, 6)
        self.W = f(veh["W"]) * gfac
        self.B = f(veh["B"])

    def lhs_terms(self, nu: torch.Tensor, R: torch.Tensor) -> torch.Tensor:
        """C_RB(nu) nu + C_A(nu) nu + D(nu) nu + g(q); nu [n, 6]."""
        n = nu.shape[0]
        v, w = nu[:, 0:3], nu[:, 3:6]
        zero = torch.zeros(n, 3, 3, dtype=DT)
        C_RB = torch.cat([torch.cat([self.m[:, None, None] * skew(w), zero], 2),
                          torch.cat([zero, -skew(self.inertia * w)], 2)], 1)
        a = self.ma * nu
        C_A = torch.cat([torch.cat([zero, -skew(a[:, 0:3])], 2),
                         torch.cat([-skew(a[:, 0:3]), -skew(a[:, 3:6])], 2)], 1)
        D = torch.diag_embed(self.D_L + self.D_Q * torch.abs(nu))
        k = R[:, 2, :]                                            # R^T e3
        g = torch.cat([(self.B - self.W)[:, None] * k, torch.zeros_like(k)], 1)
        return (C_RB @ nu[..., None])[..., 0] + (C_A @ nu[..., None])[..., 0] + (D @ nu[..., None])[..., 0] + g


def rhs(x: torch.Tensor, tau: torch.Tensor, veh: Vehicle) -> torch.Tensor:
    """dx/dt for states x [13, n] under body wrench tau [6, n]."""
    q, v, w = x[3:7], x[7:10], x[10:13]
    R = rotation(q)
    nu = torch.cat([v.T, w.T], 1)
    nu_dot = torch.linalg.solve(veh.M, (tau.T - veh.lhs_terms(nu, R))[..., None])[..., 0]
    p_dot = (R @ v.T[..., None])[..., 0].T
    T = 0.5 * torch.cat([-q[1:4].T[:, None, :], q[0][:, None, None] * torch.eye(3, dtype=DT)[None] + skew(q[1:4].T)], 1)
    q_dot = (T @ w.T[..., None])[..., 0].T
    return torch.cat([p_dot, q_dot, nu_dot.T], 0)


def rk4_substep(x, tau, veh, h):
    k1 = rhs(x, tau, veh)
    k2 = rhs(x + 0.5 * h * k1, tau, veh)
    k3 = rhs(x + 0.5 * h * k2, tau, veh)
    k4 = rhs(x + h * k3, tau, veh)
    y = x + (h / 6.0) * (k1 + 2.0 * k2 + 2.0 * k3 + k4)
    qn = y[3:7] / torch.linalg.norm(y[3:7], dim=0, keepdim=True)
    return torch.cat([y[0:3], qn, y[7:13]], 0)


def step_dynamics(x, tau, veh, dt: float, substeps: int):
    h = dt / substeps
    for _ in range(substeps):
        x = rk4_substep(x, tau, veh, h)
    return x


# ---- observation and reward of the paper task ------------------------------------------
def quat_mul(a, b):
    aw, ax, ay, az = a
    bw, bx, by, bz = b
    return torch.stack([aw * bw - ax * bx - ay * by - az * bz, aw * bx + ax * bw + ay * bz - az * by,
                        aw * by - ax * bz + ay * bw + az * bx, aw * bz + ax * by - ay * bx + az * bw])


def observe(x, p_goal, q_goal):
    """[R^T (p_goal - p), rotation vector of q^* (x) q_goal (non-negative scalar part), v, w]."""
    R = rotation(x[3:7])
    dp_b = (R.transpose(1, 2) @ (p_goal - x[0:3]).T[..., None])[..., 0].T
    qc = x[3:7] * _t([1.0, -1.0, -1.0, -1.0])[:, None]
    e = quat_mul(qc, q_goal)
    e = e * torch.where(e[0] < 0.0, -1.0, 1.0).to(DT)[None, :]
    n = torch.linalg.norm(e[1:4], dim=0)
    safe = torch.where(n > 0.0, n, torch.ones_like(n))
    k = torch.where(n > 0.0, 2.0 * torch.atan2(n, e[0]) / safe, 2.0 / e[0])
    return torch.cat([dp_b, k[None, :] * e[1:4], x[7:10], x[10:13]], 0)


def reward(task: dict, o, u, abar):
    f = _f32
    d = _t(np.asarray(task["d_pos"], np.float32))[:, None]
    return (-f(task["w_pos"]) * torch.sum((d * o[0:3]) ** 2, 0) - f(task["w_att"]) * torch.sum(o[3:6] ** 2, 0)
            - f(task["w_act"]) * torch.sum(u[3:6] ** 2, 0) - f(task["w_vel"]) * torch.sum(o[9:12] ** 2, 0)
            - f(task["w_mavg"]) * torch.sum((u - abar) ** 2, 0))


def clip_action(a):
    """clip(a, -1, 1) with derivative 1 on the closed interval (module docstring)."""
    inside = ((a >= -1.0) & (a <= 1.0)).to(DT)
    return a * inside + torch.clamp(a, -1.0, 1.0).detach() * (1.0 - inside)


def noise(seed: int, env_ids, step: int) -> np.ndarray:
    """eps [6, n] of the paper task's sampled actions at global step `step`: action c and
    3 + c take the Box-Muller pair of words (2c, 2c + 1) (c = 0, 1, 2)."""
    e8 = rng.gaussian8(seed, env_ids, step)
    return np.concatenate([e8[0:6:2], e8[1:6:2]])


# ---- one window ------------------------------------------------------------------------
def _force(v: torch.Tensor, given) -> torch.Tensor:
    """v with the value `given` and the derivative of v (module docstring, teacher forcing)."""
    return v + (_t(given) - v).detach()


def _force_state(x: torch.Tensor, given) -> torch.Tensor:
    """_force for states [13, n]: q and -q are the same attitude, and the derivative of the
    computed state is that of its own quaternion, so the given quaternion takes the sign
    nearest the computed one first."""
    g = np.array(given, np.float64)
    s = np.where(np.sum(g[3:7] * x[3:7].detach().numpy(), axis=0) < 0.0, -1.0, 1.0)
    g[3:7] *= s[None, :]
    return _force(x, g)


def window(start: dict, cfg: dict, vehicle: dict, task: dict, h: int, gamma: float, mode: int,
           policy: dict | None = None, value: dict | None = None, external=None, quantize: bool = True,
           grad_state0: bool = False, forced: dict | None = None) -> dict:
    """Forward of one window (torch graph kept for the backward).

    start: {x [13, n], abar [6, n], p_goal [3, n], q_goal [4, n], gfac [n], step (global step
    of the window's first action), env_ids [n]} as float64 numpy arrays (ints for the last
    two); policy / value: net_params dicts (12 inputs; 6 and 1 outputs); external [h][6][n];
    forced: None or {x [h][13][n] states after each step, a [h][6][n] actions} (teacher forcing).
    Returns tensors: loss, per-env J, rewards [h, n], actions a [h][6, n] (leaves in EXTERNAL
    mode), mu [h][6, n], the final state and abar, and V of the final observation."""
    x = _t(start["x"]).clone().requires_grad_(grad_state0)
    x0 = x
    abar = _t(start["abar"])
    pg, qg = _t(start["p_goal"]), _t(start["q_goal"])
    veh = Vehicle(vehicle, start["gfac"])
    dt, S = _f32(cfg["dt_control"]), int(cfg["substeps"])
    fm, tm = _f32(task["f_max"]), _f32(task["tau_max"])
    beta = _f32(task["beta"])
    n = x.shape[1]
    J = torch.zeros(n, dtype=DT)
    rewards, acts, mus = [], [], []
    o = observe(x, pg, qg)
    for t in range(h):
        if mode == MODE_EXTERNAL:
            a = _t(external[t]).clone().requires_grad_(True)
            mu = None
        else:
            mu = mlp(o, policy, quantize)
            if mu.requires_grad:
                mu.retain_grad()
            a = mu
            if mode == MODE_POLICY_SAMPLE:
                eps = _t(noise(int(cfg["seed"]), start["env_ids"], int(start["step"]) + t))
                a = mu + torch.exp(policy["log_std"])[:, None] * eps
            if forced is not None:
                a = _force(a, forced["a"][t])
        u = clip_action(a)
        tau = torch.cat([fm * u[0:3], tm * u[3:6]], 0)
        x = step_dynamics(x, tau, veh, dt, S)
        if forced is not None:
            x = _force_state(x, forced["x"][t])
        o = observe(x, pg, qg)
        r = reward(task, o, u, abar)
        abar = beta * abar + (1.0 - beta) * u
        J = J + gamma ** t * r
        rewards.append(r)
        acts.append(a)
        mus.append(mu)
    v_last = mlp(o, value, quantize)[0] if value is not None else torch.zeros(n, dtype=DT)
    J = J + gamma ** h * v_last
    loss = -J.sum() / (n * h)
    return dict(loss=loss, J=J, rewards=torch.stack(rewards), acts=acts, mus=mus, x=x, abar=abar,
                v_last=v_last, x0=x0)


def window_grad(start: dict, cfg: dict, vehicle: dict, task: dict, h: int, gamma: float, mode: int,
                policy_net: dict | None = None, value_net: dict | None = None, external=None,
                quantize: bool = True, forced: dict | None = None) -> dict:
    """Loss and gradients of one window as float64 numpy arrays: grad_policy {W1, W2, W3,
    b1, b2, b3, log_std} (12-input, 6-output shapes), grad_act [h][6][n] (dL/da_t before the
    clip: the external actions' gradient, or the policy outputs' total derivative dL/dmu_t
    plus nothing else in mean mode / the same quantity for the sampled action), grad_state0
    [13][n], and the forward's rewards [h][n], J [n], v_last [n], final state [13][n] and abar."""
    pol = net_params(policy_net, 6, requires_grad=True) if policy_net is not None else None
    val = net_params(value_net, 1) if value_net is not None else None
    w = window(start, cfg, vehicle, task, h, gamma, mode, pol, val, external, quantize, grad_state0=True,
               forced=forced)
    w["loss"].backward()
    out = dict(loss=float(w["loss"].detach()), rewards=w["rewards"].detach().numpy(), J=w["J"].detach().numpy(),
               v_last=w["v_last"].detach().numpy(), x=w["x"].detach().numpy(), abar=w["abar"].detach().numpy(),
               grad_state0=w["x0"].grad.numpy())
    if mode == MODE_EXTERNAL:
        out["grad_act"] = np.stack([a.grad.numpy() for a in w["acts"]])
    else:
        out["grad_act"] = np.stack([m.grad.numpy() for m in w["mus"]])
        out["acts"] = np.stack([a.detach().numpy() for a in w["acts"]])
        out["grad_policy"] = {k: (v.grad.numpy() if v.grad is not None else np.zeros(tuple(v.shape)))
                              for k, v in pol.items()}   # log_std is unused in mean mode
    return out


def start_from_paper_env(env) -> dict:
    """The window start of a paper_task.PaperEnv (its current state, goals and counters)."""
    return dict(x=env.x.copy(), abar=env.abar.copy(), p_goal=env.p_goal.copy(), q_goal=env.q_goal.copy(),
                gfac=env.gfac.copy(), step=env.global_step, env_ids=env.ids.copy())
