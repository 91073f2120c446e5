"""Failure detection (auv_get_status, the non-finite state counter) and the policy modes of
auv_step, through the C interface.

Non-finite values are written into chosen environments' state rows from the host; the
counter must then report exactly the non-finite components the kernels find where an
episode ends and where the launch ends, in each environment kernel (quad-layout loop,
lane-per-environment loop, fused policy rollout).  A policy-mode auv_step is the first step
of a one-step rollout, so k steps must equal a k-step rollout bit for bit."""
import numpy as np
import pytest
import torch

import workloads as W
from tests.gpu_util import announce, gpu_env, host, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dpol():
    require_gpu()
    from paper_2512_13359_amd import upload_mlp
    return upload_mlp(W.mlp_weights(8, W.POLICY_SEED))


def _poison(g, env_ids, rows, value):
    st = host(g.state).copy()
    for i in env_ids:
        st[rows, i] = value
    g.state.copy_(torch.from_numpy(st))


@pytest.mark.parametrize("n", [300, 40000])   # quad-layout loop, lane-per-environment loop
def test_status_counts_nonfinite_state_random_actions(n):
    announce(f"status random actions n={n}")
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    g = gpu_env(W.config("c2", n_envs=n))
    g.reset()
    g.step(W.MODE_RANDOM)
    assert g.get_status() == (0, 0)
    rc, _, _ = A.auv_get_status(g.handle)
    assert rc == A.AUV_OK
    # an infinite position component stays the only non-finite one (nothing in the state
    # depends on p); whole-NaN states stay NaN
    _poison(g, [5], [0], np.inf)
    _poison(g, [17, n - 1], list(range(13)), np.nan)
    g.step(W.MODE_RANDOM)
    rc, nf, ab = A.auv_get_status(g.handle)
    assert rc == A.AUV_ENONFINITE and (nf, ab) == (1 + 2 * 13, 0)
    assert g.get_status() == (0, 0)                  # cleared by the read
    g.rollout(7, W.MODE_RANDOM)
    assert g.get_status() == (1 + 2 * 13, 0)         # counted once, at the launch's end


@pytest.mark.parametrize("n", [300, 40000])
def test_status_counts_at_episode_end_before_reset(n):
    """An environment whose episode ends inside the launch is counted before its reset and is
    finite afterwards (no second count at the launch's end)."""
    announce(f"status episode end n={n}")
    require_gpu()
    g = gpu_env(W.config("c2", n_envs=n, episode_len=5))
    g.reset()
    g.rollout(2, W.MODE_RANDOM)
    _poison(g, [3, 64], list(range(13)), np.nan)     # both end their episode at step 5
    g.rollout(6, W.MODE_RANDOM)
    assert g.get_status() == (2 * 13, 0)
    assert np.isfinite(host(g.state)).all()
    g.rollout(3, W.MODE_RANDOM)
    assert g.get_status() == (0, 0)


def test_status_policy_rollout_and_abandoned_waits(dpol):
    announce("status policy rollout")
    from paper_2512_13359_amd import _abi as A
    n = 16384 + 17
    g = gpu_env(W.config("c4", n_envs=n, T=10))
    g.reset()
    g.rollout(3, W.MODE_POLICY_MEAN, policy=dpol)
    assert g.get_status() == (0, 0)
    _poison(g, [0, 9000, n - 1], list(range(13)), np.nan)
    g.rollout(4, W.MODE_POLICY_SAMPLE, policy=dpol)
    assert g.get_status() == (3 * 13, 0)
    small = gpu_env(W.config("c4", n_envs=128, T=20))
    small.reset()
    A.auv_set_sync_poll_limit(small.handle, 1)
    small.rollout(20, W.MODE_POLICY_MEAN, policy=dpol)
    nf, ab = small.get_status()
    st = host(small.state)
    assert ab >= 1 and nf == int(np.count_nonzero(~np.isfinite(st)))
    A.auv_set_sync_poll_limit(small.handle, 0)
    small.reset()
    small.rollout(20, W.MODE_POLICY_MEAN, policy=dpol)
    assert small.get_status() == (0, 0)


@pytest.mark.parametrize("mode", [W.MODE_POLICY_MEAN, W.MODE_POLICY_SAMPLE])
@pytest.mark.parametrize("n", [700, 16384 + 17])
def test_step_policy_mode_equals_rollout(dpol, mode, n):
    """k policy-mode auv_step calls equal one k-step rollout bit for bit: environment buffers,
    per-step reward and done flags, and the statistics of a one-step launch."""
    announce(f"auv_step policy mode={mode} n={n}")
    k = 6
    cfg = W.config("c4", n_envs=n, T=k, episode_len=4)
    a = gpu_env(cfg)
    a.reset()
    bufs = a.rollout_buffers(k, record=("reward", "done", "stats"))
    a.rollout(k, mode, policy=dpol, bufs=bufs)
    b = gpu_env(cfg)
    b.reset()
    rews, dones, stats = [], [], []
    for _ in range(k):
        r, d, s = b.step(mode, want_stats=True, policy=dpol)
        rews.append(host(r).copy())
        dones.append(host(d).copy())
        stats.append(host(s).copy())
    for key in ("state", "params", "ep_step", "episode", "obs"):
        assert torch.equal(getattr(a, key), getattr(b, key)), key
    assert np.array_equal(np.stack(rews), host(bufs["reward"]))
    assert np.array_equal(np.stack(dones).astype(np.float32), host(bufs["done"]))
    assert np.stack(dones)[3].all() and not np.stack(dones)[:3].any()
    assert np.array_equal(np.stack(stats, axis=1), host(bufs["stats"]))
    assert a.global_step == b.global_step == k
