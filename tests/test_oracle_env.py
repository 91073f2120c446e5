"""Pins for the oracle's environment: observation / reward special cases, reset and
auto-reset bookkeeping, randomisation ranges, sharding invariance (CPU only)."""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import workloads as W
from oracle import dynamics as dyn
from oracle import env as oenv
from oracle import rng


def _env(name="c2", **kw):
    e = oenv.Env(W.config(name, **kw), W.VEHICLE, W.ALLOC)
    e.reset()
    return e


def _set_pose(e, p, q, p_ref, q_ref):
    e.x[0:3] = np.asarray(p, float).reshape(3, -1)
    e.x[3:7] = np.asarray(q, float).reshape(4, -1)
    e.p_goal[:] = np.asarray(p_ref, float).reshape(3, -1)
    e.q_goal[:] = np.asarray(q_ref, float).reshape(4, -1)


def test_obs_zero_error_at_reference():
    e = _env("c2", n_envs=16)
    e.x[0:3] = e.p_goal
    e.x[3:7] = e.q_goal
    e.u_prev[:] = 0.0
    obs, dp, th = e.observe()
    assert np.allclose(obs[0:3], 0, atol=1e-14)
    assert np.allclose(obs[3:6], [[1], [0], [0]], atol=1e-14)
    assert np.allclose(obs[6:9], [[0], [1], [0]], atol=1e-14)
    assert np.allclose(th, 0, atol=1e-7)
    assert np.allclose(dp, 0, atol=1e-14)


def test_obs_hand_example_yaw90():
    """Vehicle at (1, 0, 0) yawed +90 deg, reference at the origin, level: the position
    error points along body +y, R_err = R^T, angle pi/2; reward with u = 0.5 on all 8
    thrusters is -1 - pi/4 - 0.01 * 8 * 0.25."""
    e = _env("c1", n_envs=1)
    c = math.cos(math.pi / 4)
    _set_pose(e, (1, 0, 0), (c, 0, 0, c), (0, 0, 0), (1, 0, 0, 0))
    e.x[7:13] = 0.0
    obs, dp, th = e.observe(u_prev=np.full((8, 1), 0.5))
    assert np.allclose(obs[0:3, 0], [0, 1, 0], atol=1e-15)
    assert np.allclose(obs[3:6, 0], [0, -1, 0], atol=1e-15)
    assert np.allclose(obs[6:9, 0], [1, 0, 0], atol=1e-15)
    assert np.allclose(obs[15:23, 0], 0.5)
    assert th[0] == pytest.approx(math.pi / 2, abs=1e-15)
    # through step(): zero thrust keeps the pose for one step only approximately, so
    # evaluate the reward expression's parts directly
    assert dp[0] == pytest.approx(1.0, abs=1e-15)


def test_attitude_error_angle_properties():
    r = np.random.Generator(np.random.PCG64(1))
    n = 200
    q = r.standard_normal((4, n))
    q /= np.linalg.norm(q, axis=0)
    qr = r.standard_normal((4, n))
    qr /= np.linalg.norm(qr, axis=0)
    Rerr = np.transpose(dyn.rotation(q), (0, 2, 1)) @ dyn.rotation(qr)
    th = oenv.rotation_angle(Rerr)
    # scipy's rotation magnitude of R^-1 R_ref
    ref = (Rotation.from_quat(np.stack([q[1], q[2], q[3], q[0]], 1)).inv()
           * Rotation.from_quat(np.stack([qr[1], qr[2], qr[3], qr[0]], 1))).magnitude()
    assert np.allclose(th, ref, atol=1e-12)
    # q and -q are the same attitude
    Rerr2 = np.transpose(dyn.rotation(-q), (0, 2, 1)) @ dyn.rotation(qr)
    assert np.allclose(oenv.rotation_angle(Rerr2), th, atol=1e-14)
    # a 180 degree flip about x
    flip = dyn.rotation(np.array([[0.0], [1.0], [0.0], [0.0]]))
    assert oenv.rotation_angle(flip)[0] == pytest.approx(math.pi, abs=1e-15)


def test_reset_draws_ranges_and_flags():
    e = _env("c2", n_envs=2000)
    assert np.all((e.scales >= 0.8) & (e.scales <= 1.2))
    assert np.all(np.abs(e.c_w) <= 0.3)
    assert np.all(np.abs(e.x[0:3]) <= 2.0) and np.all(np.abs(e.p_goal) <= 2.0)
    assert np.allclose(np.linalg.norm(e.x[3:7], axis=0), 1, atol=1e-14)
    assert np.all(e.x[7:13] == 0.0)
    assert np.all((e.amp >= 0.5) & (e.amp <= 2.0)) and np.all((e.freq >= 0.02) & (e.freq <= 0.1))
    assert np.all((e.phase >= 0) & (e.phase <= np.float32(2 * math.pi)))
    assert np.all(np.abs(e.yaw_rate) <= 0.1) and np.all(np.abs(e.yaw0) <= np.float32(math.pi))
    # every drawn scalar is an fp32 value
    for a in (e.scales, e.c_w, e.x[0:3], e.p_goal, e.amp, e.freq, e.phase, e.yaw_rate, e.yaw0):
        assert np.array_equal(a, a.astype(np.float32).astype(np.float64))
    e0 = _env("c1", n_envs=100)
    assert np.all(e0.scales == 1.0) and np.all(e0.c_w == 0.0)


def test_reset_word_positions():
    """Word k of the 32 reset words feeds draw k of the documented map."""
    e = _env("c4", n_envs=5)
    w = rng.words(e.seed, e.ids, 0, rng.TAG_RESET, 8)
    u = rng.uniform01(w)
    assert np.array_equal(e.x[0], np.float32(-2.0) + np.float32(4.0) * u[6])
    assert np.array_equal(e.scales[2], (np.float64(np.float32(0.8)) + np.float64(np.float32(0.4)) * u[2]).astype(np.float32))
    assert np.array_equal(e.yaw0, (np.float64(np.float32(-math.pi)) + np.float64(np.float32(2 * math.pi)) * u[28]).astype(np.float32))
    q = rng.shoemake(u[15], u[16], u[17])
    assert np.array_equal(e.q_goal, q)


def test_sharding_invariance():
    """An env's draws depend only on (seed, global id, episode): a shard of envs with an
    id offset reproduces the matching slice of the whole batch, step for step."""
    full = _env("c2", n_envs=96)
    part = _env("c2", n_envs=32, env_offset=40)
    for t in range(5):
        a_full = rng.random_actions(full.seed, full.ids, full.global_step)
        a_part = rng.random_actions(part.seed, part.ids, part.global_step)
        assert np.array_equal(a_full[:, 40:72], a_part)
        full.step(a_full)
        part.step(a_part)
    assert np.allclose(full.x[:, 40:72], part.x, atol=0, rtol=0)


def test_auto_reset_at_episode_length():
    e = _env("c2", n_envs=8, episode_len=7)
    p_goal0 = e.p_goal.copy()
    for t in range(7):
        r, d, s, obs = e.step(rng.random_actions(e.seed, e.ids, e.global_step))
        assert d.all() == (t == 6) and d.any() == (t == 6)
        assert s[1] == (8.0 if t == 6 else 0.0)
    assert np.all(e.episode == 1) and np.all(e.ep_step == 0)
    assert not np.allclose(e.p_goal, p_goal0)
    # the post-reset observation is the fresh state's, with a zero previous action
    assert np.all(obs[15:23] == 0.0) and np.all(e.x[7:13] == 0.0)
    assert np.allclose(obs, e.observe()[0])
    # and the fresh draws are those of episode 1
    w = rng.words(e.seed, e.ids, 1, rng.TAG_RESET, 8)
    assert np.array_equal(e.x[0], (np.float32(-2) + np.float32(4) * rng.uniform01(w[6])).astype(np.float64))


def test_stagger_initial_steps():
    e = _env("c5", n_envs=1200)
    assert np.array_equal(e.ep_step, np.arange(1200) % 500)
    done_steps = []
    for t in range(3):
        _, d, _, _ = e.step(np.zeros((8, 1200)))
        done_steps.append(np.nonzero(d)[0])
    assert list(done_steps[0]) == [499, 999]
    assert list(done_steps[1]) == [498, 998] and list(done_steps[2]) == [497, 997]


def test_lissajous_reference():
    e = _env("c4", n_envs=32)
    p_ref, q_ref = e.reference()
    assert np.allclose(p_ref, e.p_goal + e.amp * np.sin(e.phase), atol=1e-15)
    assert np.allclose(q_ref, np.stack([np.cos(e.yaw0 / 2), 0 * e.yaw0, 0 * e.yaw0, np.sin(e.yaw0 / 2)]))
    # level attitude: R_ref e3 = e3; yaw angle recovered by scipy
    R = dyn.rotation(q_ref)
    assert np.allclose(R[:, :, 2], [0, 0, 1], atol=1e-15)
    yaw = Rotation.from_matrix(R).as_euler("ZYX")[:, 0]
    assert np.allclose(np.angle(np.exp(1j * (yaw - e.yaw0))), 0, atol=1e-12)
    # at t = 1/f the position term has gone through a full period
    e.ep_step[:] = 25
    p25, _ = e.reference()
    assert np.allclose(p25, e.p_goal + e.amp * np.sin(2 * math.pi * e.freq * 25 * 0.04 + e.phase))


def test_random_actions_range_and_step():
    a = rng.random_actions(3, np.arange(1000), 17)
    assert a.min() >= -1 and a.max() < 1 and np.all(a == a.astype(np.float32))
    assert not np.array_equal(a, rng.random_actions(3, np.arange(1000), 18))


def test_reward_is_minus_distance_when_aligned_and_idle():
    e = _env("c2", n_envs=10)
    e.x[3:7] = e.q_goal
    e.x[7:13] = 0.0
    vd = W.vehicle_variant()
    obs, dp, th = e.observe(u_prev=np.zeros((8, 10)))
    assert np.allclose(th, 0, atol=1e-7)
    assert np.allclose(dp, np.linalg.norm(e.p_goal - e.x[0:3], axis=0), atol=1e-14)
    assert vd["W"] < vd["B"]


def test_step_reward_parts():
    """Reward of a step = -|dp| - 0.5 theta - 0.01 |u|^2 on the post-step state, with u
    the clipped action (actions beyond +-1 are clipped before thrust and penalty)."""
    e = _env("c2", n_envs=64)
    a = np.full((8, 64), 3.0)
    a[:, ::2] = -0.25
    r, d, s, obs = e.step(a)
    _, dp, th = e.observe()
    u = np.clip(a, -1, 1)
    assert np.allclose(r, -dp - 0.5 * th - 0.01 * (u * u).sum(0), atol=1e-14)
    assert np.allclose(obs[15:23], u)
    assert s[0] == pytest.approx(r.sum()) and s[2] == pytest.approx(dp.sum())
