"""Pins of the paper-task oracle (oracle/paper_task.py): scipy's rotation routines for the
Euler-angle goal and the axis-angle error, closed forms of the reward terms, the action
moving average and the restoring force under the gravity factor, the initial accelerations
under a pure wrench, and episode bookkeeping."""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import workloads as W
from oracle import dynamics as dyn
from oracle import paper_task as P


def _env(n=16, **kw):
    cfg = dict(n_envs=n, seed=6, flags=0, episode_len=512, substeps=2, dt_control=0.05)
    cfg.update(kw)
    e = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK)
    e.reset()
    return e


def test_euler_goal_and_axis_angle_match_scipy():
    rng = np.random.default_rng(0)
    r, p, y = (rng.uniform(-1.0, 1.0, 50) for _ in range(3))
    q = P.euler_zyx_quat(r, p, y)
    want = Rotation.from_euler("ZYX", np.stack([y, p, r], axis=1)).as_quat()     # (x, y, z, w)
    want = np.stack([want[:, 3], want[:, 0], want[:, 1], want[:, 2]])
    s = np.sign(np.sum(q * want, axis=0))
    assert np.allclose(q, want * s, atol=1e-14)
    q1 = rng.standard_normal((4, 50))
    q1 /= np.linalg.norm(q1, axis=0)
    q2 = rng.standard_normal((4, 50))
    q2 /= np.linalg.norm(q2, axis=0)
    got = P.axis_angle_error(q1, q2)
    R1 = Rotation.from_quat(np.stack([q1[1], q1[2], q1[3], q1[0]], axis=1))
    R2 = Rotation.from_quat(np.stack([q2[1], q2[2], q2[3], q2[0]], axis=1))
    want = (R1.inv() * R2).as_rotvec().T                                          # R^T R_ref
    assert np.allclose(got, want, atol=1e-12)
    assert np.allclose(P.axis_angle_error(q1, q1), 0.0, atol=1e-12)


def test_reset_draw_ranges_and_initial_state():
    e = _env(2000)
    assert np.all(e.x[0:3] == 0) and np.all(e.x[3] == 1) and np.all(e.x[7:] == 0)
    assert np.all((e.gfac >= 0.95) & (e.gfac <= 1.05))
    assert np.all(np.abs(e.p_goal) <= 2.0)
    eul = Rotation.from_quat(np.stack([e.q_goal[1], e.q_goal[2], e.q_goal[3], e.q_goal[0]], axis=1)).as_euler("ZYX")
    assert np.all(np.abs(eul) <= math.pi / 3 + 1e-6)
    assert np.all(e.abar == 0)
    # the observation at reset: body error = goal position (identity attitude), rotation vector of q_goal
    assert np.allclose(e.obs[0:3], e.p_goal)
    assert np.allclose(e.obs[3:6], P.axis_angle_error(e.x[3:7], e.q_goal))


def test_restoring_force_and_wrench_initial_accelerations():
    """At rest and level the body acceleration is M^-1 (tau - g): heave (gamma W - B)/(m + A33)
    with no wrench; F_max/(m + A11) in surge and tau_max/(I + A44) in roll with gamma W = B."""
    e = _env(3)
    v = W.VEHICLE
    e.gfac[:] = [0.95, float(v["B"]) / float(v["W"]), 1.05]
    e.veh = e._vehicle()
    x = e.x.copy()
    d = dyn.rhs(x, np.zeros((6, 3)), e.veh, e.c_w)
    m33 = float(v["m"]) + float(v["added_mass"][2])
    want = (e.gfac * float(v["W"]) - float(v["B"])) / m33
    assert np.allclose(d[9], want, rtol=1e-12, atol=1e-15)
    assert abs(d[9, 1]) < 1e-12
    tau = np.zeros((6, 3))
    tau[0], tau[3] = e.tk.f_max, e.tk.tau_max
    d = dyn.rhs(x, tau, e.veh, e.c_w)
    assert abs(d[7, 1] - e.tk.f_max / (float(v["m"]) + float(v["added_mass"][0]))) < 1e-12
    assert abs(d[10, 1] - e.tk.tau_max / (float(v["inertia"][0]) + float(v["added_mass"][3]))) < 1e-12


def test_reward_terms_closed_forms():
    """One step from a hand-set state: each term against its formula, and the moving average."""
    e = _env(4)
    e.gfac[:] = float(W.VEHICLE["B"]) / float(W.VEHICLE["W"])
    e.veh = e._vehicle()
    e.p_goal[:] = 0.0
    e.q_goal[:] = 0.0
    e.q_goal[0] = 1.0
    # env 0 at rest at the goal, zero action: reward 0 and stays there
    a = np.zeros((6, 4))
    a[:, 1] = [0.5, 0.0, 0.0, 0.0, 0.0, 0.0]            # env 1: a surge command
    a[:, 2] = [0.0, 0.0, 0.0, 0.0, 0.0, 2.0]            # env 2: a yaw torque beyond the limit
    e.x[2, 3] = 0.3                                      # env 3: 0.3 m below the goal
    r, d, s, obs = e.step(a)
    assert abs(r[0]) < 1e-30 and np.all(np.abs(obs[:, 0]) < 1e-15)   # gamma W = B up to rounding
    u1 = np.clip(a[:, 1], -1, 1)
    want1 = (-e.tk.w_pos * np.sum((e.tk.d_pos * obs[0:3, 1]) ** 2) - e.tk.w_att * np.sum(obs[3:6, 1] ** 2)
             - e.tk.w_vel * np.sum(obs[9:12, 1] ** 2) - e.tk.w_mavg * np.sum(u1 ** 2))
    assert abs(r[1] - want1) < 1e-12
    assert abs(r[2] - (-e.tk.w_act * 1.0 - e.tk.w_mavg * 1.0 - e.tk.w_att * np.sum(obs[3:6, 2] ** 2)
                       - e.tk.w_vel * np.sum(obs[9:12, 2] ** 2) - e.tk.w_pos * np.sum((e.tk.d_pos * obs[0:3, 2]) ** 2))) < 1e-12
    assert np.allclose(e.abar[:, 2], (1 - e.tk.beta) * np.clip(a[:, 2], -1, 1))
    # env 3's position term dominates and uses D_z = 1.5
    assert r[3] == pytest.approx(-e.tk.w_pos * (1.5 * obs[2, 3]) ** 2 - e.tk.w_att * np.sum(obs[3:6, 3] ** 2)
                                 - e.tk.w_vel * np.sum(obs[9:12, 3] ** 2) - e.tk.w_pos * np.sum(obs[0:2, 3] ** 2), rel=1e-12)
    assert obs[2, 3] == pytest.approx(-0.3, abs=1e-3)
    # constant action for k steps: abar = u (1 - beta^k)
    for k in range(2, 6):
        e.step(a)
        assert np.allclose(e.abar[:, 1], np.clip(a[:, 1], -1, 1) * (1 - e.tk.beta ** k), rtol=1e-12)


def test_episode_end_and_reset():
    e = _env(8, episode_len=3)
    for t in range(3):
        r, d, s, obs = e.step(np.zeros((6, 8)))
    assert np.all(d) and np.all(e.episode == 1) and np.all(e.ep_step == 0)
    assert np.all(e.x[0:3] == 0) and np.all(e.abar == 0)
    assert np.allclose(obs, e.observe())


def test_random_and_sampled_action_maps():
    """Random actions: action c <- word 2c, action 3 + c <- word 2c + 1 of env.py's random
    counter; sampled: the same pairing of the Box-Muller outputs."""
    from oracle import rng
    e = _env(5)
    a, _ = e.actions_for(P.MODE_RANDOM)
    a8 = rng.random_actions(e.seed, e.ids, 0)
    for c in range(3):
        assert np.array_equal(a[c], a8[2 * c]) and np.array_equal(a[3 + c], a8[2 * c + 1])
    net = W.mlp_weights(6, 7, n_in=12)
    mu, eps = e.actions_for(P.MODE_POLICY_SAMPLE, net)
    e8 = rng.gaussian8(e.seed, e.ids, 0)
    for c in range(3):
        assert np.array_equal(eps[c], e8[2 * c]) and np.array_equal(eps[3 + c], e8[2 * c + 1])


def test_reward_hand_valued_case():
    """The five reward terms on numbers worked out by hand (weights chosen as exact binary
    fractions): w_pos 1, D = diag(1, 1, 1.5), w_att 0.5, w_act 0.25, w_vel 0.125, w_mavg 0.5.
    dp = (1, -2, 2):     |D dp|^2 = 1 + 4 + 9 = 14                  -> 14
    dth = (0.5, 0, 0):   0.5 * 0.25                                 -> 0.125
    u = (0.5, 0, 0, 1, 0, -0.5): torques 1 + 0.25, times 0.25       -> 0.3125
    om = (0, 1, -1):     0.125 * 2                                  -> 0.25
    abar = (0.25, 0, 0, 0.5, 0, 0): |u - abar|^2 = 0.0625 + 0.25 + 0.25, times 0.5 -> 0.28125
    reward = -(14 + 0.125 + 0.3125 + 0.25 + 0.28125) = -14.96875; with beta = 0.75 the moving
    average becomes 0.75 abar + 0.25 u = (0.3125, 0, 0, 0.625, 0, -0.125)."""
    task = dict(W.PAPER_TASK, w_pos=1.0, d_pos=(1.0, 1.0, 1.5), w_att=0.5, w_act=0.25, w_vel=0.125, w_mavg=0.5,
                beta=0.75)
    k = P.Task(task)
    col = lambda *v: np.array(v, np.float64)[:, None]  # noqa: E731
    dp, dth, om = col(1, -2, 2), col(0.5, 0, 0), col(0, 1, -1)
    u, abar = col(0.5, 0, 0, 1, 0, -0.5), col(0.25, 0, 0, 0.5, 0, 0)
    z3, z6 = col(0, 0, 0), col(0, 0, 0, 0, 0, 0)
    assert P.paper_reward(k, dp, dth, om, u, abar)[0] == -14.96875
    # each term alone
    assert P.paper_reward(k, dp, z3, z3, z6, z6)[0] == -14.0
    assert P.paper_reward(k, z3, dth, z3, z6, z6)[0] == -0.125
    assert P.paper_reward(k, z3, z3, om, z6, z6)[0] == -0.25
    assert P.paper_reward(k, z3, z3, z3, u, u)[0] == -0.3125        # no deviation from the average
    assert P.paper_reward(k, z3, z3, z3, z6, abar - u)[0] == -0.28125 - 0.0   # only the average term
    # the same numbers through one environment step: the step's reward is built from the
    # post-step observation, the clipped action and the average before the update
    e = _env(1)
    e.tk = k
    e.abar = abar.copy()
    e.step(u)
    assert np.array_equal(e.abar, col(0.3125, 0, 0, 0.625, 0, -0.125))
