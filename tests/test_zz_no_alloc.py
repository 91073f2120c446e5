"""auv_rollout_static, the rollout entry point that allocates nothing, through the C
interface: its results equal auv_rollout's (which takes a caller-provided statistics
workspace) bit for bit, on two calls in a row, the second smaller than the first (so the
library's array holds the first call's partials when the second starts); requests beyond the
array and a given workspace are refused before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from tests.gpu_util import announce, gpu_env, host, require_gpu

pytestmark = pytest.mark.gpu


def _pair(cfg, T, mode, dpol, record):
    from paper_2512_13359_amd import _abi as A
    a, b = gpu_env(cfg), gpu_env(cfg)
    a.reset()
    b.reset()
    ba = a.rollout_buffers(T, record=record)
    a.rollout(T, mode, policy=dpol, bufs=ba)
    bb = b.rollout_buffers(T, record=record)
    bb.pop("stats_work", None)
    A.auv_rollout_static(b.handle, T, mode, None if dpol is None else dpol["struct"], None,
                         A.make_rollout_buffers(**bb))
    torch.cuda.synchronize()
    return a, b, ba, bb


def _same(a, b, ba, bb):
    for k in bb:
        assert torch.equal(ba[k], bb[k]), k
    for k in ("state", "params", "ep_step", "episode", "obs"):
        assert torch.equal(getattr(a, k), getattr(b, k)), k
    assert a.global_step == b.global_step


def test_static_rollout_matches_rollout_twice():
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    from paper_2512_13359_amd import upload_mlp
    dpol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    rec = ("obs", "act", "reward", "done", "stats")
    # first: four tiles per workgroup, ragged, 300 steps (4.7 rows of 64); second: smaller
    for n, T, ep in ((16384 + 17, 300, 120), (1000, 70, 33)):
        announce(f"static rollout n={n} T={T}")
        a, b, ba, bb = _pair(W.config("c4", n_envs=n, T=T, episode_len=ep), T, W.MODE_POLICY_MEAN, dpol, rec)
        _same(a, b, ba, bb)
        assert host(bb["done"]).sum() > 0 and np.isfinite(host(bb["stats"])).all()
    # the random-action loop through the same array (two calls, the second smaller)
    for n, T in ((5000, 200), (300, 9)):
        announce(f"static random rollout n={n} T={T}")
        a, b, ba, bb = _pair(W.config("c2", n_envs=n, episode_len=50), T, W.MODE_RANDOM, None, ("reward", "stats"))
        _same(a, b, ba, bb)
    # refused before anything is enqueued: too many partials, a workspace given
    g = gpu_env(W.config("c4", n_envs=65536, T=1000))
    g.reset()
    before = host(g.state).copy()
    stats = torch.empty(3, 1000, device="cuda")
    rb = A.make_rollout_buffers(stats=stats)
    rc = A.lib.auv_rollout_static(g.handle, 1000, W.MODE_POLICY_MEAN, ctypes.byref(dpol["struct"]), None,
                                  ctypes.byref(rb), None)
    assert rc == A.AUV_EINVAL and "maximum" in A.auv_last_error()
    work = torch.empty(A.auv_stats_work_floats(65536, 10), device="cuda")
    rb2 = A.make_rollout_buffers(stats=stats, stats_work=work)
    rc = A.lib.auv_rollout_static(g.handle, 10, W.MODE_POLICY_MEAN, ctypes.byref(dpol["struct"]), None,
                                  ctypes.byref(rb2), None)
    assert rc == A.AUV_EINVAL and "stats_work" in A.auv_last_error()
    assert np.array_equal(host(g.state), before) and g.global_step == 0
