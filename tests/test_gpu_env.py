"""GPU parity of the environment path (reset, random / external actions, auto-reset,
statistics, GAE) against the fp64 oracle, through the C interface."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import gae as ogae
from oracle import rng
from tests.gpu_util import (announce, gpu_env, host, oracle_env, quat_aligned, rel_err,
                            require_gpu)

pytestmark = pytest.mark.gpu

AFFINE_ROWS = [0, 1, 2, 3, 4, 5, 6, 7, 8, 13, 14, 15, 16, 17, 18, 19, 20, 21, 22, 23]


def _reset_pair(cfg):
    g = gpu_env(cfg)
    g.reset()
    o = oracle_env(cfg)
    o.reset()
    return g, o


@pytest.mark.parametrize("name,n", [("c2", 1000), ("c4", 4096 + 37), ("c5", 777), ("c1", 64)])
def test_reset_parity(name, n):
    require_gpu()
    announce(f"reset parity {name} n={n}")
    cfg = W.config(name, n_envs=n)
    g, o = _reset_pair(cfg)
    params = host(g.params)
    state = host(g.state)
    want = o.params_f32()
    # affine draws and positions: bit-exact
    assert np.array_equal(params[AFFINE_ROWS], want[AFFINE_ROWS])
    assert np.array_equal(state[0:3], o.x[0:3].astype(np.float32))
    assert np.all(state[7:13] == 0.0)
    # Shoemake quaternions: 1e-6
    assert np.max(np.abs(params[9:13] - o.q_goal)) <= 1e-6
    assert np.max(np.abs(state[3:7] - o.x[3:7])) <= 1e-6
    assert np.array_equal(host(g.ep_step), o.ep_step.astype(np.int32))
    assert np.array_equal(host(g.episode), o.episode.astype(np.int32))
    assert np.max(rel_err(host(g.obs), o.obs)) <= 1e-4


def _rollout_random(cfg, T, record):
    g, o = _reset_pair(cfg)
    bufs = g.rollout_buffers(T, record=record)
    g.rollout(T, W.MODE_RANDOM, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    rec = o.rollout(T, W.MODE_RANDOM, record_state="traj_state" in record)
    return g, o, got, rec


def test_c1_full_trajectory():
    """c1: 64 envs x 200 steps, Philox actions, no randomisation: every state of the
    trajectory within 1e-3, actions bit-exact, obs / reward within 1e-4 early on."""
    require_gpu()
    cfg = W.config("c1")
    announce("c1 full trajectory 64 x 200")
    g, o, got, rec = _rollout_random(cfg, 200, ("obs", "act", "reward", "done", "traj_state", "stats"))
    assert np.array_equal(got["act"], rec["act"].astype(np.float32))
    assert np.all(got["done"] == 0) and np.all(rec["done"] == 0)
    traj = got["traj_state"]
    traj[3:7] = quat_aligned(traj[3:7], rec["traj_state"][3:7])
    err = rel_err(traj, rec["traj_state"])
    assert err[:, 1].max() <= 1e-4           # one step from the identical reset state
    assert err[:, -1].max() <= 1e-3          # end of the run
    assert err.max() <= 1e-3
    assert rel_err(got["obs"][:, :20], rec["obs"][:, :20]).max() <= 1e-4
    assert rel_err(got["reward"][:20], rec["reward"][:20]).max() <= 1e-4
    # the env's state buffer holds the last trajectory entry
    assert g.global_step == 200


def test_c2_full_size_sampled_envs():
    """c2 at full size (4096 x 1000, randomisation, current, one auto-reset per env).
    The oracle replays three 64-env slices through its global-id counters."""
    require_gpu()
    cfg = W.config("c2")
    T, n = cfg["T"], cfg["n_envs"]
    announce("c2 4096 x 1000 (GPU), oracle on 3 slices")
    g = gpu_env(cfg)
    g.reset()
    bufs = g.rollout_buffers(T, record=("reward", "done", "stats"))
    g.rollout(T, W.MODE_RANDOM, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    state = host(g.state)
    # dones: exactly at steps 499 and 999 for every env
    d = got["done"]
    assert np.array_equal(np.nonzero(d.any(axis=1))[0], [499, 999]) and np.all(d[[499, 999]] == 1)
    assert np.array_equal(host(g.episode), np.full(n, 2, np.int32))
    # stats: sums of the GPU's own per-env values
    s = got["stats"]
    assert np.allclose(s[0], got["reward"].astype(np.float64).sum(1), rtol=1e-5, atol=1e-3)
    assert np.array_equal(s[1], got["done"].sum(1))
    for off in (0, 2011, n - 64):
        o = oracle_env(W.config("c2", n_envs=64, env_offset=off))
        o.reset()
        rec = o.rollout(T, W.MODE_RANDOM)
        sl = slice(off, off + 64)
        assert np.array_equal(d[:, sl], rec["done"].astype(np.float32))
        x = state[:, sl].copy()
        x[3:7] = quat_aligned(x[3:7], o.x[3:7])
        assert rel_err(x, o.x).max() <= 1e-3
        assert rel_err(got["reward"][-50:, sl], rec["reward"][-50:]).max() <= 1e-3


def test_lane_layout_loop_large_batch():
    """Above 32 envs per SIMD (four SIMDs per CU) the random / external loop keeps one
    environment per lane instead of four lanes per environment.  A batch just past that
    size with a ragged last wave and short episodes (auto-resets inside the run): random
    actions bit-exact, dones exact, rewards and end states of three 64-env slices within
    1e-3 of the oracle, then one external-action step."""
    require_gpu()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n, T, H = 128 * cus + 1000 + 7, 40, 15
    cfg = W.config("c2", n_envs=n, episode_len=H)
    announce(f"lane-per-env loop n={n} T={T} H={H}")
    g = gpu_env(cfg)
    g.reset()
    bufs = g.rollout_buffers(T, record=("act", "reward", "done", "stats"))
    g.rollout(T, W.MODE_RANDOM, bufs=bufs)
    got = {k: host(v) for k, v in bufs.items()}
    s = got["stats"]
    assert np.allclose(s[0], got["reward"].astype(np.float64).sum(1), rtol=1e-5, atol=1e-3)
    assert np.array_equal(s[1], got["done"].sum(1))
    acts = np.random.default_rng(9).uniform(-1.3, 1.3, (8, n)).astype(np.float32)
    reward, done, _ = g.step(W.MODE_EXTERNAL, torch.from_numpy(acts).cuda())
    state = host(g.state)
    for off in (0, n // 2 + 11, n - 64):
        o = oracle_env(W.config("c2", n_envs=64, env_offset=off, episode_len=H))
        o.reset()
        rec = o.rollout(T, W.MODE_RANDOM)
        sl = slice(off, off + 64)
        assert np.array_equal(got["act"][:, :, sl], rec["act"].astype(np.float32))
        assert np.array_equal(got["done"][:, sl], rec["done"].astype(np.float32))
        assert rel_err(got["reward"][:, sl], rec["reward"]).max() <= 1e-3
        r_o, d_o, _, _ = o.step(acts[:, sl].astype(np.float64))
        assert np.array_equal(host(done)[sl].astype(bool), d_o)
        assert rel_err(host(reward)[sl], r_o).max() <= 1e-3
        x = state[:, sl].copy()
        x[3:7] = quat_aligned(x[3:7], o.x[3:7])
        assert rel_err(x, o.x).max() <= 1e-3


def test_one_step_from_identical_state():
    """One control step from the same seeded fp32 states on both sides (random poses and
    velocities; each side's own randomisation draws from the same seed), external seeded
    actions including out-of-range ones: 1e-4 per component."""
    require_gpu()
    n = 3000 + 5
    cfg = W.config("c4", n_envs=n)
    announce(f"one step from identical state n={n} (c4 model, 4 substeps)")
    g, o = _reset_pair(cfg)
    x0 = W.random_states(n, seed=3)
    ep0 = ((np.arange(n) * 7) % 499).astype(np.int32)
    g.state.copy_(torch.from_numpy(x0))
    g.ep_step.copy_(torch.from_numpy(ep0))
    o.x = x0.astype(np.float64)
    o.ep_step = ep0.astype(np.int64)
    acts = np.random.default_rng(5).uniform(-1.3, 1.3, (8, n)).astype(np.float32)
    reward, done, _ = g.step(W.MODE_EXTERNAL, torch.from_numpy(acts).cuda())
    r_o, d_o, _, obs_o = o.step(acts.astype(np.float64))
    x = host(g.state)
    x[3:7] = quat_aligned(x[3:7], o.x[3:7])
    assert rel_err(x, o.x).max() <= 1e-4
    assert np.array_equal(host(done).astype(bool), d_o)
    assert rel_err(host(reward), r_o).max() <= 1e-4
    assert rel_err(host(g.obs), obs_o).max() <= 1e-4


def test_step_api_matches_rollout_and_is_deterministic():
    require_gpu()
    cfg = W.config("c2", n_envs=517, episode_len=3)
    announce("auv_step vs auv_rollout, determinism")
    a = gpu_env(cfg)
    b = gpu_env(cfg)
    a.reset()
    b.reset()
    rs, ds, ss = [], [], []
    for _ in range(5):
        r, d, s = a.step(W.MODE_RANDOM, want_stats=True)
        rs.append(host(r)); ds.append(host(d)); ss.append(host(s))
    bufs = b.rollout_buffers(5, record=("reward", "done", "stats"))
    b.rollout(5, W.MODE_RANDOM, bufs=bufs)
    assert np.array_equal(np.stack(rs), host(bufs["reward"]))
    assert np.array_equal(np.stack(ds).astype(np.float32), host(bufs["done"]))
    assert np.array_equal(np.stack(ss).T, host(bufs["stats"]))
    assert np.array_equal(host(a.state), host(b.state))
    assert np.array_equal(host(a.obs), host(b.obs))
    assert np.array_equal(host(a.params), host(b.params))


def test_checkpoint_resume_bit_exact():
    """T steps in one go equal T/2 steps, a copy of the state buffers and step counter
    into a fresh handle, and T/2 more steps."""
    require_gpu()
    cfg = W.config("c2", n_envs=300, episode_len=40)
    announce("checkpoint / resume")
    a = gpu_env(cfg)
    a.reset()
    a.rollout(100, W.MODE_RANDOM)
    b = gpu_env(cfg)
    b.reset()
    b.rollout(50, W.MODE_RANDOM)
    c = gpu_env(cfg)
    for k in ("state", "params", "ep_step", "episode", "obs"):
        getattr(c, k).copy_(getattr(b, k))
    c.global_step = b.global_step
    c.rollout(50, W.MODE_RANDOM)
    for k in ("state", "params", "ep_step", "episode", "obs"):
        assert torch.equal(getattr(a, k), getattr(c, k)), k


def test_gae_parity():
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    # segmented scan with 16-step segments (T <= 256), 32-step segments (T <= 512), and the
    # one-lane-per-env scan beyond; ragged env counts and partial last segments
    for T, n in ((64, 65536), (37, 1001), (1, 5), (256, 300), (512, 4096), (300, 777), (600, 130)):
        announce(f"gae T={T} n={n}")
        r = np.random.default_rng(T)
        rew = r.normal(size=(T, n)).astype(np.float32)
        val = r.normal(size=(T, n)).astype(np.float32)
        done = (r.random((T, n)) < 0.05).astype(np.float32)
        last = r.normal(size=n).astype(np.float32)
        dev = [torch.from_numpy(x).cuda() for x in (rew, val, done, last)]
        adv = torch.empty(T, n, device="cuda")
        ret = torch.empty(T, n, device="cuda")
        A.auv_gae(T, n, *dev, 0.99, 0.95, adv, ret)
        a_o, r_o = ogae.gae(rew, val, done, last, 0.99, 0.95)
        assert np.all(np.abs(host(adv) - a_o) <= 1e-4 * (1 + np.abs(a_o)))
        assert np.all(np.abs(host(ret) - r_o) <= 1e-4 * (1 + np.abs(r_o)))


def test_invalid_arguments_enqueue_nothing():
    require_gpu()
    from paper_2512_13359_amd import AuvError
    g = gpu_env(W.config("c1"))
    g.reset()
    before = host(g.state).copy()
    with pytest.raises(AuvError):
        g.rollout(0, W.MODE_RANDOM)
    with pytest.raises(AuvError):
        g.step(mode=7)
    with pytest.raises(AuvError):
        g.step(mode=W.MODE_EXTERNAL, actions=None)
    assert np.array_equal(host(g.state), before)
    assert g.global_step == 0


def test_philox_words_through_random_actions():
    """Random-mode actions are 2u - 1 of Philox words (env, step, 1, b): bit-exact for
    large env ids and step counters (sharding offset near 2^32, step near 2^31)."""
    require_gpu()
    cfg = W.config("c1", n_envs=130, env_offset=2**32 - 200)
    g = gpu_env(cfg)
    g.reset()
    g.global_step = 2**31 + 12345
    bufs = g.rollout_buffers(3, record=("act",))
    g.rollout(3, W.MODE_RANDOM, bufs=bufs)
    act = host(bufs["act"])
    ids = np.arange(130) + 2**32 - 200
    for t in range(3):
        want = rng.random_actions(cfg["seed"], ids, 2**31 + 12345 + t)
        assert np.array_equal(act[:, t], want.astype(np.float32))
