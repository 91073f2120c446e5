"""GPU parity of the bf16 MFMA policy / value MLP and the fused policy rollout against
the fp64 oracle, through the C interface.

bf16 rounding of the hidden activations makes the MLP's result non-unique: where an
exact hidden value lies within the fp32 error bound DELTA of a bf16 rounding midpoint,
both roundings are correct.  The MLP is therefore compared with the nearest of the
oracle's valid outputs (oracle.mlp.mlp_candidates), to a tolerance far below 2e-3.

A closed-loop trajectory inherits that non-uniqueness, so closed-loop runs are checked
for what is unique (episode ends, reset draws) and for validity: every action the GPU
took must be a valid policy output for the observation it was taken on, and every
transition must agree with the oracle's dynamics for that action."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gae as ogae
from oracle import mlp as omlp
from oracle import rng
from tests.gpu_util import (announce, gpu_env, host, oracle_env, quat_aligned, rel_err,
                            require_gpu)

pytestmark = pytest.mark.gpu

TOL_MU = 2e-3      # policy / value outputs against the oracle (bf16 MFMA)
TOL_VALID = 2e-4   # distance to the nearest valid bf16 output
DELTA = 1e-6       # bound on the fp32 error of a hidden value before its bf16 rounding


@pytest.fixture(scope="module")
def nets():
    require_gpu()
    from paper_2512_13359_amd import upload_mlp
    pol = W.mlp_weights(8, W.POLICY_SEED)
    val = W.mlp_weights(1, W.VALUE_SEED)
    return pol, val, upload_mlp(pol), upload_mlp(val)


def _mlp_gpu(dev_net, obs):
    from paper_2512_13359_amd import _abi as A
    n = obs.shape[1]
    out = torch.empty(dev_net["n_out"], n, device="cuda")
    A.auv_mlp_forward(dev_net["struct"], n, torch.from_numpy(np.ascontiguousarray(obs, np.float32)).cuda(), out)
    return host(out)


@pytest.mark.parametrize("n", [1, 64, 1000, 20000])
def test_mlp_forward_parity(nets, n):
    pol, val, dpol, dval = nets
    announce(f"mlp forward n={n}")
    r = np.random.default_rng(n)
    obs = np.concatenate([r.normal(0, 2, (3, n)), r.uniform(-1, 1, (6, n)), r.normal(0, 1, (6, n)),
                          r.uniform(-1, 1, (8, n))]).astype(np.float32)
    mu = _mlp_gpu(dpol, obs)
    err = omlp.nearest_valid_error(mu, obs.astype(np.float64), pol, DELTA)
    assert err.max() <= TOL_VALID
    v = _mlp_gpu(dval, obs)
    err = omlp.nearest_valid_error(v, obs.astype(np.float64), val, DELTA)
    assert err.max() <= TOL_VALID


def test_mlp_single_entry_routing(nets):
    """Single-entry weights: input j -> hidden-1 unit i -> hidden-2 unit k -> output o,
    one case per wave slice, checks orientation and the K-slot order of every tile."""
    from paper_2512_13359_amd import upload_mlp
    cases = [(17, 5, 200, 3), (0, 255, 0, 7), (22, 64, 130, 0), (9, 191, 63, 5)]
    for j, i, k, o in cases:
        def bits(a):
            return torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        W1 = np.zeros((256, 23)); W1[i, j] = 1.0
        W2 = np.zeros((256, 256)); W2[k, i] = 1.0
        W3 = np.zeros((8, 256)); W3[o, k] = 2.0
        net = {"W1": bits(W1), "W2": bits(W2), "W3": bits(W3), "b1": np.zeros(256, np.float32),
               "b2": np.zeros(256, np.float32), "b3": np.zeros(8, np.float32)}
        obs = np.zeros((23, 70), np.float32)
        obs[j] = np.linspace(-2, 2, 70)
        got = _mlp_gpu(upload_mlp(net), obs)
        want = omlp.mlp_forward(obs.astype(np.float64), net)
        assert np.max(np.abs(got - want)) <= TOL_MU, (j, i, k, o)
        assert np.all(np.delete(got, o, axis=0) == 0.0)
        assert np.count_nonzero(got[o]) >= 60


def _policy_rollout(cfg, T, dpol, record, mode=W.MODE_POLICY_MEAN, dval=None):
    g = gpu_env(cfg)
    g.reset()
    bufs = g.rollout_buffers(T, record=record)
    g.rollout(T, mode, policy=dpol, value=dval, bufs=bufs)
    return g, {k: host(v) for k, v in bufs.items()}


def _check_mu_on_gpu_obs(pol, got, sample_idx=None):
    """Largest distance of the GPU's actions to a valid policy output for the observation
    each was taken on (validity of the GPU's own trajectory)."""
    obs, act = got["obs"], got["act"]
    T, n = obs.shape[1], obs.shape[2]
    flat_o = obs.reshape(23, T * n)
    flat_a = act.reshape(8, T * n)
    if sample_idx is not None:
        flat_o, flat_a = flat_o[:, sample_idx], flat_a[:, sample_idx]
    return omlp.nearest_valid_error(flat_a, flat_o.astype(np.float64), pol, DELTA).max()


def test_c3_closed_loop(nets):
    """c3 shape (4096 envs, policy mean) over 120 steps, plus a ragged 1000-env batch."""
    pol, _, dpol, _ = nets
    for n, T in ((4096, 120), (1000 + 17, 60)):
        announce(f"c3 closed loop n={n} T={T}")
        cfg = W.config("c3", n_envs=n)
        g, got = _policy_rollout(cfg, T, dpol, ("obs", "act", "reward", "done", "traj_state", "stats"))
        idx = np.random.default_rng(n).choice(T * n, min(T * n, 12000), replace=False)
        assert _check_mu_on_gpu_obs(pol, got, idx) <= TOL_VALID
        # validity of the transitions: the oracle's dynamics under the GPU's actions
        sl = slice(n - 64, n)
        o = oracle_env(W.config("c3", n_envs=64, env_offset=n - 64))
        o.reset()
        rec = o.rollout(T, W.MODE_EXTERNAL, external=np.transpose(got["act"][:, :, sl], (1, 0, 2)).astype(np.float64),
                        record_state=True)
        traj = got["traj_state"][:, :, sl].copy()
        traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
        err = rel_err(traj, rec["traj_state"])
        assert err[:, 1].max() <= 1e-4 and err.max() <= 1e-3
        assert rel_err(got["reward"][:, sl], rec["reward"]).max() <= 1e-3
        assert rel_err(got["obs"][:, :10, sl], rec["obs"][:, :10]).max() <= 1e-4
        assert np.all(got["done"] == 0)
        s = got["stats"]
        assert np.allclose(s[0], got["reward"].astype(np.float64).sum(1), rtol=1e-5, atol=1e-3)


def _teacher_forced(cfg, got, off, n_slice, T):
    """Worst per-transition errors of envs [off, off + n_slice): each of the T transitions
    against the oracle's control step from the GPU's state under the GPU's action (state,
    reward, next observation; and whether any done flag differs)."""
    sl = slice(off, off + n_slice)
    o = oracle_env(dict(cfg, n_envs=n_slice, env_offset=off))
    o.reset()
    traj = got["traj_state"][:, :, sl].astype(np.float64)
    worst = np.zeros(4)
    for t in range(T):
        o.x = traj[:, t].copy()
        rew, done, _, obs = o.step(got["act"][:, t, sl].astype(np.float64))
        x = traj[:, t + 1].copy()
        x[3:7] = quat_aligned(x[3:7], o.x[3:7])
        e = [rel_err(x, o.x).max(), rel_err(got["reward"][t, sl], rew).max(),
             rel_err(got["obs"][:, t + 1, sl], obs).max() if t + 1 < T else 0.0,
             float(np.any(done != (got["done"][t, sl] == 1)))]
        worst = np.maximum(worst, e)
    return worst


def test_c4_full_size_sampled(nets):
    """c4 at full size, the configuration the benchmark times: 16384 envs x 2000 steps,
    4 substeps, Lissajous references, policy mean.  Episode ends exact for every env; the
    policy valid on 6000 sampled (step, env) observations; every one of the 2000
    transitions agrees with the oracle's control step from the GPU's state under the GPU's
    action (1e-4, the one-step bound) for the 64 envs of one workgroup (all four of its
    physics tiles), and the reset draws of the episode starts agree with the oracle's own."""
    pol, _, dpol, _ = nets
    cfg = W.config("c4")
    n, T = cfg["n_envs"], cfg["T"]
    announce(f"c4 full size n={n} T={T}")
    g, got = _policy_rollout(cfg, T, dpol, ("obs", "act", "reward", "done", "traj_state"))
    r = np.random.default_rng(0)
    idx = r.choice(T * n, 6000, replace=False)
    assert _check_mu_on_gpu_obs(pol, got, idx) <= TOL_VALID
    d = got["done"]
    assert np.array_equal(np.nonzero(d.any(axis=1))[0], [499, 999, 1499, 1999])
    assert np.all(d[[499, 999, 1499, 1999]] == 1)
    off = 141 * 64                  # workgroup 141: tiles 0-3
    sl = slice(off, off + 64)
    worst = _teacher_forced(cfg, got, off, 64, T)
    announce(f"c4 per-transition worst: state {worst[0]:.2e} reward {worst[1]:.2e} obs {worst[2]:.2e}")
    assert worst[3] == 0
    assert worst[0] <= 1e-4 and worst[1] <= 1e-4 and worst[2] <= 1e-4
    x = host(g.state)[:, sl]
    assert np.array_equal(x, got["traj_state"][:, -1, sl])


def test_c5_sampling_value_gae(nets):
    """c5 shape: 65536 envs x 64 steps, Gaussian sampling, staggered episodes, PPO buffer,
    value net and GAE.  Sampled envs checked against the oracle."""
    pol, val, dpol, dval = nets
    cfg = W.config("c5")
    n, T = cfg["n_envs"], cfg["T"]
    announce(f"c5 n={n} T={T}")
    g, got = _policy_rollout(cfg, T, dpol, ("obs", "act", "logp", "value", "reward", "done", "last_value"),
                             mode=W.MODE_POLICY_SAMPLE, dval=dval)
    # dones: env i finishes at step (499 - i mod 500) when that is < T
    want_done = np.zeros((T, n), np.float32)
    ids = np.arange(n)
    first = 499 - ids % 500
    m = first < T
    want_done[first[m], ids[m]] = 1.0
    assert np.array_equal(got["done"], want_done)
    assert abs(want_done.any(0).mean() - 0.128) < 0.01
    r = np.random.default_rng(1)
    envs = np.sort(r.choice(n, 256, replace=False))
    sigma = np.exp(np.float64(np.float32(-0.5)))
    for t in (0, 17, 63):
        o_t = got["obs"][:, t, envs].astype(np.float64)
        eps = rng.gaussian8(cfg["seed"], envs, t)
        # the action minus the oracle's noise must be a valid policy mean for o_t
        mu_gpu = got["act"][:, t, envs] - sigma * eps
        assert omlp.nearest_valid_error(mu_gpu, o_t, pol, DELTA).max() <= TOL_MU
        assert np.max(np.abs(got["logp"][t, envs] - omlp.gaussian_logp(eps, pol["log_std"]))) <= TOL_MU
        assert omlp.nearest_valid_error(got["value"][None, t, envs], o_t, val, DELTA).max() <= TOL_VALID
    lv_err = omlp.nearest_valid_error(got["last_value"][None, envs], host(g.obs)[:, envs].astype(np.float64), val, DELTA)
    assert lv_err.max() <= TOL_VALID
    # GAE on the GPU buffers
    from paper_2512_13359_amd import _abi as A
    dev = {k: torch.from_numpy(np.ascontiguousarray(got[k])).cuda() for k in ("reward", "value", "done", "last_value")}
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    A.auv_gae(T, n, dev["reward"], dev["value"], dev["done"], dev["last_value"], 0.99, 0.95, adv, ret)
    a_o, r_o = ogae.gae(got["reward"], got["value"], got["done"], got["last_value"], 0.99, 0.95)
    assert np.all(np.abs(host(adv) - a_o) <= 1e-4 * (1 + np.abs(a_o)))
    assert np.all(np.abs(host(ret) - r_o) <= 1e-4 * (1 + np.abs(r_o)))
    # teacher-forced dynamics for the first 64 envs (contains staggered resets)
    o = oracle_env(W.config("c5", n_envs=64))
    o.reset()
    rec = o.rollout(T, W.MODE_EXTERNAL, external=np.transpose(got["act"][:, :, :64], (1, 0, 2)).astype(np.float64))
    assert rel_err(got["reward"][:, :64], rec["reward"]).max() <= 1e-3
    assert np.array_equal(got["done"][:, :64], rec["done"].astype(np.float32))


def test_policy_rollout_deterministic_and_resumable(nets):
    _, _, dpol, _ = nets
    cfg = W.config("c4", n_envs=700, T=30, episode_len=11)
    announce("policy rollout determinism / resume")
    a = gpu_env(cfg)
    a.reset()
    a.rollout(30, W.MODE_POLICY_SAMPLE, policy=dpol)
    b = gpu_env(cfg)
    b.reset()
    b.rollout(13, W.MODE_POLICY_SAMPLE, policy=dpol)
    b.rollout(17, W.MODE_POLICY_SAMPLE, policy=dpol)
    for k in ("state", "params", "ep_step", "episode", "obs"):
        assert torch.equal(getattr(a, k), getattr(b, k)), k


@pytest.mark.parametrize("n,T", [(1, 5), (17, 3), (64 + 5, 1)])
def test_policy_rollout_small_and_ragged(nets, n, T):
    """Single environment, a tile that is only partly filled, one-step launches: valid
    actions, the oracle's control step under them, statistics equal to the per-env sums."""
    pol, _, dpol, _ = nets
    announce(f"policy rollout small n={n} T={T}")
    cfg = W.config("c4", n_envs=n, T=T)
    g, got = _policy_rollout(cfg, T, dpol, ("obs", "act", "reward", "done", "traj_state", "stats"))
    assert _check_mu_on_gpu_obs(pol, got) <= TOL_VALID
    o = oracle_env(cfg)
    o.reset()
    rec = o.rollout(T, W.MODE_EXTERNAL, external=np.transpose(got["act"], (1, 0, 2)).astype(np.float64),
                    record_state=True)
    traj = got["traj_state"].copy()
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    assert rel_err(traj, rec["traj_state"]).max() <= 1e-4 * T
    assert rel_err(got["reward"], rec["reward"]).max() <= 1e-3
    assert np.allclose(got["stats"][0], got["reward"].astype(np.float64).sum(1), rtol=1e-5, atol=1e-4)
    assert np.isfinite(got["stats"]).all()


def test_policy_rollout_rejects_zero_steps(nets):
    """T = 0 is an argument error: nothing is enqueued and the state stays as it was."""
    from paper_2512_13359_amd import _abi as A
    _, _, dpol, _ = nets
    cfg = W.config("c4", n_envs=100, T=4)
    g = gpu_env(cfg)
    g.reset()
    before = {k: getattr(g, k).clone() for k in ("state", "params", "ep_step", "episode", "obs")}
    with pytest.raises(A.AuvError):
        g.rollout(0, W.MODE_POLICY_MEAN, policy=dpol)
    for k, v in before.items():
        assert torch.equal(getattr(g, k), v), k


def test_abandoned_waits_end_the_launch(nets):
    """With a one-poll bound, the workgroup's waits give up: the launch still ends normally
    and the abandoned environments hold NaN (never a hang).  The default bound restores
    normal results."""
    from paper_2512_13359_amd import _abi as A
    _, _, dpol, _ = nets
    announce("abandoned waits")
    cfg = W.config("c4", n_envs=128, T=20)
    g = gpu_env(cfg)
    g.reset()
    A.auv_set_sync_poll_limit(g.handle, 1)
    g.rollout(20, W.MODE_POLICY_MEAN, policy=dpol)
    st = host(g.state)
    assert np.isnan(st).any()
    A.auv_set_sync_poll_limit(g.handle, 0)
    g.reset()
    g.rollout(20, W.MODE_POLICY_MEAN, policy=dpol)
    assert np.isfinite(host(g.state)).all()


def _stats_rows_check(got, final_obs, check_dist):
    """Rows of the batch statistics against fp64 sums of the GPU's own per-env values:
    reward and |dp| (the norm of the post-step observation's first three rows, on steps
    without an episode end) to 1e-5 relative, done exactly."""
    s = got["stats"].astype(np.float64)
    rew = got["reward"].astype(np.float64)
    want_r = rew.sum(1)
    assert np.all(np.abs(s[0] - want_r) <= 1e-5 * np.abs(rew).sum(1)), np.abs(s[0] - want_r).max()
    assert np.array_equal(s[1], got["done"].astype(np.float64).sum(1))
    if check_dist:
        post = np.concatenate([got["obs"][0:3, 1:], final_obs[0:3, None]], axis=1).astype(np.float64)
        want_p = np.sqrt((post ** 2).sum(0)).sum(1)
        assert np.all(np.abs(s[2] - want_p) <= 1e-5 * want_p), np.abs(s[2] - want_p).max()


@pytest.mark.parametrize("n", [16384 + 17, 8192 + 37])
def test_rollout_statistics_all_rows(nets, n):
    """Batch statistics of the fused rollout at four and at two tiles per workgroup, the
    configurations of every benchmarked size from 8192 envs up, with a ragged last workgroup
    (tiles partly or wholly empty): 80 steps cross a 64-step row of the partials and end in a
    partial row.  Without episode ends all three rows are checked; with staggered episodes
    (about 16 % of the envs end one within the launch, sampled actions) reward and done."""
    pol, _, dpol, _ = nets
    T = 80
    for stagger in (False, True):
        announce(f"rollout statistics n={n} T={T} stagger={stagger}")
        cfg = W.config("c4", n_envs=n, T=T)
        if stagger:
            cfg["flags"] |= W.FLAG_STAGGER
        mode = W.MODE_POLICY_SAMPLE if stagger else W.MODE_POLICY_MEAN
        g, got = _policy_rollout(cfg, T, dpol, ("obs", "reward", "done", "stats"), mode=mode)
        if stagger:
            assert got["done"].sum() > 0.1 * n
        else:
            assert got["done"].sum() == 0
        _stats_rows_check(got, host(g.obs), check_dist=not stagger)


def test_two_tile_rollout_parity(nets):
    """Two 16-env tiles per workgroup (the instantiation for 8192 to 16383 envs): every action a
    valid policy output on 6000 sampled observations; every transition of the 64 envs of two
    whole workgroups against the oracle's control step (1e-4), across an episode end."""
    pol, _, dpol, _ = nets
    n, T = 8192 + 37, 60
    announce(f"two-tile rollout n={n} T={T}")
    cfg = W.config("c4", n_envs=n, T=T, episode_len=41)
    g, got = _policy_rollout(cfg, T, dpol, ("obs", "act", "reward", "done", "traj_state"))
    idx = np.random.default_rng(2).choice(T * n, 6000, replace=False)
    assert _check_mu_on_gpu_obs(pol, got, idx) <= TOL_VALID
    assert np.array_equal(np.nonzero(got["done"].any(axis=1))[0], [40])
    for off in (32 * 100, n - 37 - 27):    # workgroups 100-101; the last three (the last one ragged)
        worst = _teacher_forced(cfg, got, off, 64, T)
        announce(f"  envs {off}..{off + 63}: state {worst[0]:.2e} reward {worst[1]:.2e} obs {worst[2]:.2e}")
        assert worst[3] == 0 and worst[0] <= 1e-4 and worst[1] <= 1e-4 and worst[2] <= 1e-4
