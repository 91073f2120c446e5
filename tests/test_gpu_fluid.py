"""GPU parity of the paper task with the inertia-box fluid model (auv_task.fluid =
AUV_FLUID_INERTIA_BOX) against the oracle (oracle/fluid.py through paper_task.PaperEnv), and
the model's closed forms on the GPU: terminal surge and heave speeds under a constant
command.  Also one SHAC window on the box model against the SHAC oracle given the same
hydrodynamics."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import fluid as fl
from oracle import mlp as omlp
from oracle import paper_task as P
from oracle import shac as S
from tests.gpu_util import announce, gpu_env, host, quat_aligned, rel_err, require_gpu

pytestmark = pytest.mark.gpu


def _pair(cfg):
    g = gpu_env(cfg)
    g.set_task(W.PAPER_TASK_BOX)
    g.reset()
    o = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK_BOX)
    o.reset()
    return g, o


def test_box_model_random_rollout_matches_oracle():
    n, T = 300 + 5, 80
    cfg = W.config("c6", n_envs=n, episode_len=30)
    announce(f"inertia-box random rollout n={n} T={T}")
    g, o = _pair(cfg)
    bufs = g.rollout_buffers(T, record=("obs", "act", "reward", "done", "traj_state"))
    g.rollout(T, W.MODE_RANDOM, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    rec = o.rollout(T, P.MODE_RANDOM, record_state=True)
    assert np.array_equal(got["act"][0:6], rec["act"].astype(np.float32))
    assert np.array_equal(got["done"], rec["done"].astype(np.float32))
    traj = got["traj_state"].copy()
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    err = rel_err(traj, rec["traj_state"])
    assert err[:, 1].max() <= 1e-4 and err.max() <= 2e-3
    assert rel_err(got["reward"], rec["reward"]).max() <= 2e-3
    go, ro = got["obs"], rec["obs"]
    assert rel_err(go[0:3], ro[0:3]).max() <= 2e-3 and rel_err(go[6:12], ro[6:12]).max() <= 2e-3
    # the box model really is different from the Fossen one
    f = gpu_env(cfg)
    f.set_task(W.PAPER_TASK)
    f.reset()
    fb = f.rollout_buffers(T, record=("traj_state",))
    f.rollout(T, W.MODE_RANDOM, bufs=fb)
    assert np.max(np.abs(host(fb["traj_state"]) - got["traj_state"])) > 1e-2


def test_box_model_policy_rollout_matches_oracle():
    """The 12-256-256-6 policy (mean) in closed loop on the box model, a ragged batch with one
    episode end: every action is a valid bf16-policy output for the observation it was taken
    on, and under the GPU's actions the oracle's box model reproduces every reward, episode end
    and state."""
    require_gpu()
    from paper_2512_13359_amd import upload_mlp
    pol = W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12)
    n, T = 200 + 3, 40
    cfg = W.config("c6", n_envs=n, episode_len=25)
    announce(f"inertia-box policy rollout n={n} T={T}")
    g, o = _pair(cfg)
    bufs = g.rollout_buffers(T, record=("obs", "act", "reward", "done", "traj_state"))
    g.rollout(T, W.MODE_POLICY_MEAN, policy=upload_mlp(pol), bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    act, obs = got["act"][0:6], got["obs"][0:12]
    err = omlp.nearest_valid_error(act.reshape(6, -1), obs.reshape(12, -1).astype(np.float64), pol, 1e-6)
    assert err.max() <= 2e-4
    rec = o.rollout(T, P.MODE_EXTERNAL, external=np.transpose(act, (1, 0, 2)).astype(np.float64), record_state=True)
    assert np.array_equal(got["done"], rec["done"].astype(np.float32))
    traj = got["traj_state"].copy()
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    assert rel_err(traj, rec["traj_state"]).max() <= 1e-3
    assert rel_err(got["reward"], rec["reward"]).max() <= 1e-3


def test_box_model_terminal_speeds():
    """A constant half-scale surge command for 20 s from rest: surge reaches the closed-form
    terminal speed of F = quad v^2 + lin v; heave follows the closed-form speed from rest under
    the net restoring force (B - gamma W per environment; small forces are still far from
    their terminal speed); attitude and rates stay level and zero."""
    n, T = 64, 400
    cfg = W.config("c6", n_envs=n)
    announce(f"inertia-box terminal speeds n={n} T={T}")
    require_gpu()
    g = gpu_env(cfg)
    g.set_task(W.PAPER_TASK_BOX)
    g.reset()
    act = torch.zeros(8, T, n, device="cuda")
    act[0] = 0.5
    bufs = g.rollout_buffers(T, record=("reward",))
    bufs["act"] = act
    g.rollout(T, W.MODE_EXTERNAL, bufs=bufs)
    x = host(g.state)
    c = fl.drag_coefficients(float(np.float32(11.5)), np.float32([0.16] * 3).astype(np.float64), 1000.0,
                             float(np.float32(1e-3)))
    v_surge = fl.terminal_speed(0.5 * 60.0, c["lin"][0], c["quad"][0])
    assert np.max(np.abs(x[7] - v_surge)) <= 1e-4 * v_surge
    gfac = host(g.params)[13].astype(np.float64)
    Fz = -(float(np.float32(114.8)) - gfac * float(np.float32(112.8)))   # (gamma W - B) along +z (down)
    m = float(np.float32(11.5))
    v_heave = np.array([fl.speed_from_rest(f, T * 0.05, m, c["lin"][2], c["quad"][2]) for f in Fz])
    assert np.max(np.abs(x[9] - v_heave)) <= 1e-4 * np.max(np.abs(v_heave)) + 1e-7
    assert np.max(np.abs(x[3] - 1.0)) <= 1e-6 and np.max(np.abs(x[10:13])) <= 1e-6 and np.max(np.abs(x[8])) <= 1e-6


def test_box_model_shac_window_matches_oracle():
    """SHAC on the box model: the SHAC oracle is given the same hydrodynamics as constants of
    its vehicle (no added mass, the box's drag coefficients)."""
    n, h, gamma = 101, 5, 0.99
    announce(f"inertia-box SHAC window n={n} h={h}")
    require_gpu()
    from paper_2512_13359_amd import ShacLearner
    cfg = W.config("c6", n_envs=n)
    g = gpu_env(cfg)
    g.set_task(W.PAPER_TASK_BOX)
    g.reset()
    x0 = W.random_states(n, seed=21)
    g.state.copy_(torch.from_numpy(x0))
    pr, ob = host(g.params), host(g.obs)
    start = dict(x=x0.astype(np.float64), abar=ob[12:18].astype(np.float64), p_goal=pr[6:9].astype(np.float64),
                 q_goal=pr[9:13].astype(np.float64), gfac=pr[13].astype(np.float64), step=0, env_ids=np.arange(n))
    pol = W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12)
    val = W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12)
    L = ShacLearner(g, pol, val, h=h, gamma=gamma)
    gact = torch.zeros(8, h, n, device="cuda")
    L.window(mode=3, out=dict(grad_act=gact))
    c = fl.drag_coefficients(float(np.float32(11.5)), np.float32([0.16] * 3).astype(np.float64), 1000.0,
                             float(np.float32(1e-3)))
    veh = dict(W.VEHICLE, added_mass=np.zeros(6, np.float32), lin_damp=c["lin"].astype(np.float32),
               quad_damp=c["quad"].astype(np.float32))
    want = S.window_grad(start, cfg, veh, W.PAPER_TASK, h, gamma, S.MODE_POLICY_SAMPLE, policy_net=pol,
                         value_net=val, quantize=True)
    ga = np.transpose(host(gact)[0:6], (1, 0, 2))
    assert np.max(np.abs(ga - want["grad_act"])) <= 2e-2 * np.max(np.abs(want["grad_act"]))
    got = host(L.grad)
    gw2 = got[256 * 23:256 * 23 + 256 * 256].reshape(256, 256)
    assert np.max(np.abs(gw2 - want["grad_policy"]["W2"])) <= 5e-3 * np.max(np.abs(want["grad_policy"]["W2"]))
