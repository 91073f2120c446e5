"""Pins of the SHAC oracle (oracle/shac.py).

Forward: the torch physics against the numpy Fossen oracle (dynamics.py), and whole windows
against the paper-task oracle (paper_task.PaperEnv) under external and sampled policy
actions.  Gradient: central finite differences of the float64 forward (per environment,
since each environment's return depends only on its own actions and state) for the
open-loop chain through reward, observation, RK4, Fossen and the terminal value, and
directional differences along random parameter directions for the closed loop through the
policy; the quantised MLP backward against the PPO oracle's hand-written backward."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import dynamics as dyn
from oracle import paper_task as P
from oracle import ppo as oppo
from oracle import shac as S
from oracle.mlp import bf16_round

CFG = dict(n_envs=16, seed=6, flags=0, episode_len=512, substeps=2, dt_control=0.05)


def _env(n=16, seed=6):
    e = P.PaperEnv({**CFG, "n_envs": n, "seed": seed}, W.VEHICLE, W.PAPER_TASK)
    e.reset()
    return e


def _moving_start(n=16, seed=3):
    """A window start away from rest (so that |v| and |omega| kinks are not at 0)."""
    e = _env(n)
    r = np.random.default_rng(seed)
    x = W.random_states(n, seed=seed).astype(np.float64)
    e.load(x, e.gfac.astype(np.float32), e.p_goal.astype(np.float32), e.q_goal.astype(np.float32),
           e.ep_step, e.episode, r.uniform(-0.5, 0.5, (6, n)).astype(np.float32))
    return e, S.start_from_paper_env(e)


def _nets():
    pol = W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12)
    val = W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12)
    return pol, val


def test_torch_physics_matches_numpy_fossen_oracle():
    n = 64
    r = np.random.default_rng(1)
    x = W.random_states(n, seed=11).astype(np.float64)
    tau = r.uniform(-30, 30, (6, n))
    gfac = r.uniform(0.95, 1.05, n)
    veh = dict(W.VEHICLE)
    veh["r_b"] = np.zeros(3, np.float32)
    ov = dyn.Vehicle(veh, n)
    ov.W = float(np.float32(veh["W"])) * gfac
    want = dyn.rhs(x, tau, ov, np.zeros((3, n)))
    got = S.rhs(torch.from_numpy(x), torch.from_numpy(tau), S.Vehicle(veh, gfac)).numpy()
    assert np.max(np.abs(got - want)) <= 1e-12 * np.max(np.abs(want))
    want = dyn.integrate(x, tau, ov, np.zeros((3, n)), 0.05, 2)
    got = S.step_dynamics(torch.from_numpy(x), torch.from_numpy(tau), S.Vehicle(veh, gfac), 0.05, 2).numpy()
    assert np.max(np.abs(got - want)) <= 1e-13


def test_window_forward_matches_paper_env_external():
    n, h = 24, 7
    e = _env(n)
    start = S.start_from_paper_env(e)
    ext = np.random.default_rng(2).uniform(-1.3, 1.3, (h, 6, n))
    w = S.window(start, {**CFG, "n_envs": n}, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_EXTERNAL, external=ext)
    rec = e.rollout(h, P.MODE_EXTERNAL, external=ext)
    assert np.max(np.abs(w["rewards"].detach().numpy() - rec["reward"])) <= 1e-11 * np.max(np.abs(rec["reward"]))
    assert np.max(np.abs(w["x"].detach().numpy() - e.x)) <= 1e-12
    assert np.max(np.abs(w["abar"].detach().numpy() - e.abar)) <= 1e-15
    disc = sum(0.99 ** t * rec["reward"][t] for t in range(h))
    assert np.allclose(w["J"].detach().numpy(), disc, rtol=1e-12, atol=0)
    assert abs(float(w["loss"].detach()) + disc.sum() / (n * h)) <= 1e-12 * abs(disc.sum() / (n * h))


def test_window_forward_matches_paper_env_policy_sample():
    n, h = 32, 6
    pol, val = _nets()
    e = _env(n)
    start = S.start_from_paper_env(e)
    w = S.window(start, {**CFG, "n_envs": n}, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE,
                 policy=S.net_params(pol, 6), value=S.net_params(val, 1))
    rec = e.rollout(h, P.MODE_POLICY_SAMPLE, policy=pol)
    assert np.max(np.abs(torch.stack(w["acts"]).detach().numpy() - np.transpose(rec["act"], (1, 0, 2)))) <= 1e-12
    assert np.max(np.abs(w["rewards"].detach().numpy() - rec["reward"])) <= 1e-11 * np.max(np.abs(rec["reward"]))
    from oracle.mlp import mlp_forward
    assert np.allclose(w["v_last"].detach().numpy(), mlp_forward(e.obs, val)[0], rtol=0, atol=1e-13)


def _per_env_fd(fun, base, delta):
    """Central differences of the per-env vector fun(x) [n] w.r.t. every row of base [..., n]
    (all envs perturbed together: each env's value depends only on its own column)."""
    g = np.zeros_like(base)
    it = np.ndindex(*base.shape[:-1])
    for idx in it:
        xp, xm = base.copy(), base.copy()
        xp[idx] += delta
        xm[idx] -= delta
        g[idx] = (fun(xp) - fun(xm)) / (2.0 * delta)
    return g


def test_open_loop_gradient_matches_finite_differences():
    """dL/da_t and dL/ds_0 through reward, observation, RK4 + Fossen and the terminal value
    (value net without rounding, so the objective is smooth), against central differences;
    actions beyond the clip have an exactly zero gradient."""
    n, h, gamma = 12, 5, 0.97
    _, val = _nets()
    e, start = _moving_start(n)
    cfg = {**CFG, "n_envs": n}
    ext = np.random.default_rng(4).uniform(-0.9, 0.9, (h, 6, n))
    ext[2, 1, 3], ext[4, 5, 0] = 1.25, -1.4           # outside the clip
    g = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_EXTERNAL, value_net=val,
                      external=ext, quantize=False)

    def J_of_actions(a):
        w = S.window(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_EXTERNAL,
                     value=S.net_params(val, 1), external=a, quantize=False)
        return w["J"].detach().numpy()

    fd = -_per_env_fd(J_of_actions, ext, 1e-6) / (n * h)
    assert np.max(np.abs(g["grad_act"] - fd)) <= 1e-6 * np.max(np.abs(g["grad_act"]))
    assert g["grad_act"][2, 1, 3] == 0.0 and g["grad_act"][4, 5, 0] == 0.0
    assert np.min(np.abs(g["grad_act"][0])) > 0.0

    def J_of_state(x0):
        s = dict(start, x=x0)
        w = S.window(s, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_EXTERNAL,
                     value=S.net_params(val, 1), external=ext, quantize=False)
        return w["J"].detach().numpy()

    fd = -_per_env_fd(J_of_state, start["x"], 1e-6) / (n * h)
    assert np.max(np.abs(g["grad_state0"] - fd)) <= 1e-6 * np.max(np.abs(g["grad_state0"]))


def test_closed_loop_policy_gradient_matches_directional_differences():
    """Gradient w.r.t. every policy parameter (log_std included) through the closed loop,
    without rounding: <grad, d> against (L(theta + delta d) - L(theta - delta d)) / 2 delta
    for random directions d."""
    n, h, gamma = 8, 4, 0.99
    pol, val = _nets()
    e, start = _moving_start(n, seed=5)
    cfg = {**CFG, "n_envs": n}
    g = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_POLICY_SAMPLE, pol, val, quantize=False)
    base = S.net_params(pol, 6)
    vp = S.net_params(val, 1)
    r = np.random.default_rng(7)
    for _ in range(3):
        d = {k: r.standard_normal(v.shape) for k, v in base.items()}
        dd = sum(float(np.sum(g["grad_policy"][k] * d[k])) for k in d)

        def L(s):
            p = {k: base[k] + s * torch.from_numpy(d[k]) for k in base}
            return float(S.window(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_POLICY_SAMPLE, p, vp,
                                  quantize=False)["loss"].detach())

        delta = 1e-6
        fd = (L(delta) - L(-delta)) / (2 * delta)
        assert abs(dd - fd) <= 1e-6 * abs(dd), (dd, fd)


def test_quantized_mlp_backward_matches_ppo_oracle():
    """The rounding operators put the bf16 points where the PPO oracle's hand-written
    backward has them: identical weight gradients; bias gradients are the sums of the
    rounded cotangents (equal to the PPO oracle's unrounded sums without rounding)."""
    pol, _ = _nets()
    r = np.random.default_rng(3)
    x = r.uniform(-2, 2, (12, 40))
    gy = r.standard_normal((6, 40)) * 1e-2
    for quantize in (True, False):
        p = S.net_params(pol, 6, requires_grad=True)
        y = S.mlp(torch.from_numpy(x), p, quantize)
        (y * torch.from_numpy(gy)).sum().backward()
        pn = {k: v.detach().numpy() for k, v in p.items()}
        y_ref, cache = oppo.mlp_forward_cache(x, pn, quantize)
        assert np.max(np.abs(y.detach().numpy() - y_ref)) <= 1e-13
        want = oppo.mlp_backward(pn, cache, gy, quantize)
        for k in ("W1", "W2", "W3"):
            assert np.max(np.abs(p[k].grad.numpy() - want[k])) <= 1e-13 * np.max(np.abs(want[k])), k
        if quantize:
            assert np.array_equal(p["b3"].grad.numpy(), bf16_round(gy).sum(axis=1))
            for k in ("b1", "b2"):
                bound = 2.0 ** -8 * np.abs(want[k]).max() * 40
                assert np.max(np.abs(p[k].grad.numpy() - want[k])) <= bound
                assert not np.array_equal(p[k].grad.numpy(), want[k])
        else:
            for k in ("b1", "b2", "b3"):
                assert np.max(np.abs(p[k].grad.numpy() - want[k])) <= 1e-13 * np.max(np.abs(want[k])), k


def test_terminal_value_and_discount_enter_linearly():
    """L = -(sum_t gamma^t r_t + gamma^h V) / (N h): with the value net removed the loss
    changes by exactly gamma^h sum V / (N h)."""
    n, h, gamma = 10, 3, 0.9
    pol, val = _nets()
    e = _env(n)
    start = S.start_from_paper_env(e)
    cfg = {**CFG, "n_envs": n}
    a = S.window(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_POLICY_MEAN, S.net_params(pol, 6),
                 S.net_params(val, 1))
    b = S.window(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_POLICY_MEAN, S.net_params(pol, 6), None)
    dv = gamma ** h * float(a["v_last"].detach().sum()) / (n * h)
    assert abs((float(b["loss"].detach()) - float(a["loss"].detach())) - dv) <= 1e-14


def test_teacher_forcing_along_own_trajectory_is_the_plain_gradient():
    """Forcing the window onto its own trajectory changes nothing (the replacement keeps the
    value and the derivative); forcing it onto a perturbed trajectory moves the rewards to that
    trajectory's and the gradient by a comparably small amount."""
    pol, val = _nets()
    _, start = _moving_start(12, seed=21)
    cfg = dict(CFG, n_envs=12)
    h = 7
    w = S.window(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE, S.net_params(pol, 6),
                 S.net_params(val, 1), quantize=True)
    acts = [a.detach().numpy() for a in w["acts"]]
    # the states after each step under those actions (the forward's own step, replayed)
    xs, x = [], torch.as_tensor(start["x"])
    veh = S.Vehicle(W.VEHICLE, start["gfac"])
    f32 = lambda v: float(np.float32(v))  # noqa: E731
    for t in range(h):
        u = S.clip_action(torch.as_tensor(acts[t]))
        tau = torch.cat([f32(W.PAPER_TASK["f_max"]) * u[0:3], f32(W.PAPER_TASK["tau_max"]) * u[3:6]], 0)
        x = S.step_dynamics(x, tau, veh, f32(cfg["dt_control"]), cfg["substeps"])
        xs.append(x.numpy().copy())
    assert np.array_equal(xs[-1], w["x"].detach().numpy())
    plain = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE, pol, val)
    forced = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE, pol, val,
                           forced=dict(x=np.stack(xs), a=np.stack(acts)))
    for k in plain["grad_policy"]:
        assert np.allclose(forced["grad_policy"][k], plain["grad_policy"][k], rtol=1e-10, atol=1e-14), k
    assert np.allclose(forced["rewards"], plain["rewards"], rtol=1e-12, atol=1e-14)
    # the same trajectory with some quaternions given as -q (the same attitudes)
    flip = np.stack(xs).copy()
    flip[1::2, 3:7, ::3] *= -1.0
    forced2 = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE, pol, val,
                            forced=dict(x=flip, a=np.stack(acts)))
    for k in plain["grad_policy"]:
        assert np.allclose(forced2["grad_policy"][k], plain["grad_policy"][k], rtol=1e-10, atol=1e-14), k
    assert np.allclose(forced2["grad_act"], plain["grad_act"], rtol=1e-10, atol=1e-14)
    # a perturbed trajectory: the rewards follow it, the gradient moves a little
    r = np.random.default_rng(5)
    xp = np.stack(xs) + 1e-4 * r.standard_normal(np.stack(xs).shape)
    pert = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_SAMPLE, pol, val,
                         forced=dict(x=xp, a=np.stack(acts)))
    assert not np.allclose(pert["rewards"], plain["rewards"], rtol=1e-9, atol=0)
    for k in plain["grad_policy"]:
        g0 = plain["grad_policy"][k]
        assert np.max(np.abs(pert["grad_policy"][k] - g0)) <= 1e-2 * np.max(np.abs(g0)), k
