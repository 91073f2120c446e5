"""GPU parity of the paper's own training task (auv_set_task with AUV_TASK_PAPER) against
the fp64 oracle (oracle/paper_task.py), through the C interface.

The rotation vector of an attitude error near 180 degrees is not unique (its sign flips
with the sign of the error quaternion's scalar part, which floating point decides there),
so observation rows 3-5 are compared only where that scalar part is not tiny; the reward
uses |dtheta|^2 and is unique everywhere."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import mlp as omlp
from oracle import paper_task as P
from oracle import rng
from tests.gpu_util import announce, gpu_env, host, quat_aligned, rel_err, require_gpu

pytestmark = pytest.mark.gpu

DELTA = 1e-6
TOL_VALID = 2e-4
TOL_MU = 2e-3


def _pair(cfg):
    g = gpu_env(cfg)
    g.set_task(W.PAPER_TASK)
    g.reset()
    o = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK)
    o.reset()
    return g, o


def _err_scalar(q, q_goal):
    """|scalar part| of q^* (x) q_goal."""
    return np.abs(np.sum(q * q_goal, axis=0))


def test_paper_reset_parity():
    n = 1000 + 7
    announce(f"paper task reset n={n}")
    g, o = _pair(W.config("c6", n_envs=n))
    params, state, obs = host(g.params), host(g.state), host(g.obs)
    assert np.array_equal(params[13], o.gfac.astype(np.float32))           # affine draws: bit-exact
    assert np.array_equal(params[6:9], o.p_goal.astype(np.float32))
    assert np.max(np.abs(params[9:13] - o.q_goal)) <= 1e-6
    assert np.all(params[0:3] == 1) and np.all(params[3:6] == 0) and np.all(params[14:] == 0)
    want = np.zeros((13, n), np.float32)
    want[3] = 1
    assert np.array_equal(state, want)
    assert np.array_equal(obs[0:3], params[6:9])
    assert np.max(np.abs(obs[3:6] - o.obs[3:6])) <= 1e-5
    assert np.all(obs[6:] == 0)


def test_paper_random_rollout_with_resets():
    """Open loop (Philox actions) over 80 steps with 30-step episodes: actions bit-exact,
    episode ends exact, every state, reward and observation against the oracle."""
    n, T = 300 + 5, 80
    cfg = W.config("c6", n_envs=n, episode_len=30)
    announce(f"paper task random rollout n={n} T={T}")
    g, o = _pair(cfg)
    bufs = g.rollout_buffers(T, record=("obs", "act", "reward", "done", "traj_state", "stats"))
    g.rollout(T, W.MODE_RANDOM, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    rec = o.rollout(T, P.MODE_RANDOM, record_state=True)
    assert np.array_equal(got["act"][0:6], rec["act"].astype(np.float32))
    assert np.array_equal(got["done"], rec["done"].astype(np.float32))
    assert np.array_equal(np.nonzero(got["done"].any(axis=1))[0], [29, 59])
    traj = got["traj_state"].copy()
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    err = rel_err(traj, rec["traj_state"])
    assert err[:, 1].max() <= 1e-4 and err.max() <= 1e-3
    assert rel_err(got["reward"], rec["reward"]).max() <= 1e-3
    assert rel_err(got["reward"][:10], rec["reward"][:10]).max() <= 1e-4
    go, ro = got["obs"], rec["obs"]
    assert rel_err(go[0:3], ro[0:3]).max() <= 1e-3 and rel_err(go[6:12], ro[6:12]).max() <= 1e-3
    unique = np.linalg.norm(ro[3:6], axis=0) < np.pi - 1e-2          # rotation vectors away from 180 deg
    assert rel_err(go[3:6][:, unique], ro[3:6][:, unique]).max() <= 1e-3
    assert np.all(go[12:] == 0)
    s = got["stats"]
    assert np.allclose(s[0], got["reward"].astype(np.float64).sum(1), rtol=1e-5, atol=1e-3)
    assert np.array_equal(s[1], got["done"].sum(1))


def test_paper_one_step_from_identical_state():
    """Random poses, velocities, goals and action averages on both sides, external actions
    including out-of-range ones: state, reward, observation and the new action average 1e-4."""
    n = 2000 + 3
    cfg = W.config("c6", n_envs=n)
    announce(f"paper task one step n={n}")
    g, o = _pair(cfg)
    x0 = W.random_states(n, seed=8)
    r = np.random.default_rng(9)
    ep0 = ((np.arange(n) * 7) % 500).astype(np.int32)
    abar0 = r.uniform(-1, 1, (6, n)).astype(np.float32)
    g.state.copy_(torch.from_numpy(x0))
    g.ep_step.copy_(torch.from_numpy(ep0))
    obs0 = host(g.obs).copy()
    obs0[12:18] = abar0
    g.obs.copy_(torch.from_numpy(obs0))
    pr = host(g.params)
    o.load(x0, pr[13], pr[6:9], pr[9:13], ep0, np.zeros(n), abar0)
    acts = r.uniform(-1.3, 1.3, (6, n)).astype(np.float32)
    a8 = np.zeros((8, n), np.float32)
    a8[0:6] = acts
    reward, done, _ = g.step(W.MODE_EXTERNAL, torch.from_numpy(a8).cuda())
    r_o, d_o, _, obs_o = o.step(acts.astype(np.float64))
    x = host(g.state)
    x[3:7] = quat_aligned(x[3:7], o.x[3:7])
    assert rel_err(x, o.x).max() <= 1e-4
    assert np.array_equal(host(done).astype(bool), d_o)
    assert rel_err(host(reward), r_o).max() <= 1e-4
    go = host(g.obs)
    unique = _err_scalar(o.x[3:7], o.q_goal) > 1e-3
    assert rel_err(go[0:3], obs_o[0:3]).max() <= 1e-4
    assert rel_err(go[3:6][:, unique], obs_o[3:6][:, unique]).max() <= 1e-4
    assert rel_err(go[6:12], obs_o[6:12]).max() <= 1e-4
    assert np.max(np.abs(go[12:18] - o.abar)) <= 1e-6
    assert unique.mean() > 0.99


@pytest.mark.parametrize("mode", [W.MODE_POLICY_MEAN, W.MODE_POLICY_SAMPLE])
def test_paper_policy_rollout(mode):
    """The 12-256-256-6 policy in closed loop (mean or Gaussian sample), a ragged batch, one
    episode end: every action is a valid policy output (plus the oracle's noise) for the
    observation it was taken on, log-probabilities match, and under the GPU's actions the
    oracle reproduces every reward, episode end and state."""
    require_gpu()
    from paper_2512_13359_amd import upload_mlp
    pol = W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12)
    dpol = upload_mlp(pol)
    n, T = 256 + 9, 40
    cfg = W.config("c6", n_envs=n, episode_len=25)
    announce(f"paper task policy rollout mode={mode} n={n} T={T}")
    g, o = _pair(cfg)
    rec_keys = ("obs", "act", "reward", "done", "traj_state") + (("logp",) if mode == W.MODE_POLICY_SAMPLE else ())
    bufs = g.rollout_buffers(T, record=rec_keys)
    g.rollout(T, mode, policy=dpol, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    act = got["act"][0:6]
    obs = got["obs"][0:12]
    if mode == W.MODE_POLICY_SAMPLE:
        sig = np.exp(np.asarray(pol["log_std"], np.float32).astype(np.float64))[:6, None]
        for t in range(T):
            e8 = rng.gaussian8(cfg["seed"], np.arange(n), t)
            eps = np.concatenate([e8[0:6:2], e8[1:6:2]])
            mu = act[:, t] - sig * eps
            assert omlp.nearest_valid_error(mu, obs[:, t].astype(np.float64), pol, DELTA).max() <= TOL_MU
            lp = np.sum(-0.5 * eps * eps - np.log(sig) - 0.5 * np.log(2 * np.pi), axis=0)
            assert np.max(np.abs(got["logp"][t] - lp)) <= 1e-4
    else:
        err = omlp.nearest_valid_error(act.reshape(6, -1), obs.reshape(12, -1).astype(np.float64), pol, DELTA)
        assert err.max() <= TOL_VALID
    rec = o.rollout(T, P.MODE_EXTERNAL, external=np.transpose(act, (1, 0, 2)).astype(np.float64), record_state=True)
    assert np.array_equal(got["done"], rec["done"].astype(np.float32))
    traj = got["traj_state"].copy()
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    assert rel_err(traj, rec["traj_state"]).max() <= 1e-3
    assert rel_err(got["reward"], rec["reward"]).max() <= 1e-3


def test_paper_step_matches_rollout_and_resumes():
    cfg = W.config("c6", n_envs=517, episode_len=4)
    announce("paper task step vs rollout, resume")
    a = gpu_env(cfg)
    b = gpu_env(cfg)
    for e in (a, b):
        e.set_task(W.PAPER_TASK)
        e.reset()
    rs = []
    for _ in range(7):
        r, d, s = a.step(W.MODE_RANDOM)
        rs.append(host(r))
    bufs = b.rollout_buffers(7, record=("reward",))
    b.rollout(3, W.MODE_RANDOM)
    b2 = b.rollout_buffers(4, record=("reward",))
    b.rollout(4, W.MODE_RANDOM, bufs=b2)
    assert np.array_equal(np.stack(rs[3:]), host(b2["reward"]))
    for k in ("state", "params", "ep_step", "episode", "obs"):
        assert torch.equal(getattr(a, k), getattr(b, k)), k
    del bufs


def test_paper_task_rejects_workload_flags():
    require_gpu()
    from paper_2512_13359_amd import AuvError
    g = gpu_env(W.config("c2", n_envs=64))
    with pytest.raises(AuvError):
        g.set_task(W.PAPER_TASK)
    g2 = gpu_env(W.config("c6", n_envs=64))
    with pytest.raises(AuvError):
        g2.set_task({**W.PAPER_TASK, "beta": 1.0})
    with pytest.raises(AuvError):
        g2.set_task({**W.PAPER_TASK, "kind": 7})
