"""C interface checks that need no GPU: the library loads, exports every function the
header declares, and auv_create validates its arguments (it makes no GPU call)."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    txt = open(os.path.join(ROOT, "include", "auv.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(auv_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    from paper_2512_13359_amd import _abi as A
    names = _header_functions()
    assert "auv_rollout" in names and "auv_create" in names and len(names) >= 11
    raw = ctypes.CDLL(A.LIB_PATH)
    for name in names:
        assert hasattr(raw, name), name


def _cfg(**kw):
    from paper_2512_13359_amd import _abi as A
    base = dict(n_envs=64, substeps=1, episode_len=500, dt_control=0.02, seed=1, flags=0)
    base.update(kw)
    return A.make_config(**base)


def _bufs(addr=0x10000):
    from paper_2512_13359_amd import _abi as A
    # fake device addresses: auv_create only checks them, it never dereferences them
    return A.AuvEnvBuffers(addr, addr + 0x1000, addr + 0x2000, addr + 0x3000, addr + 0x4000)


def test_create_validates_without_gpu():
    from paper_2512_13359_amd import _abi as A
    veh = A.make_vehicle(W.VEHICLE, W.ALLOC)
    h = A.auv_create(_cfg(), veh, _bufs())
    assert A.auv_get_global_step(h) == 0
    A.auv_set_global_step(h, 123)
    assert A.auv_get_global_step(h) == 123
    A.auv_destroy(h)
    bad = [(_cfg(n_envs=0), veh, _bufs(), "n_envs"),
           (_cfg(substeps=0), veh, _bufs(), "substeps"),
           (_cfg(episode_len=0), veh, _bufs(), "episode_len"),
           (_cfg(dt_control=-1.0), veh, _bufs(), "dt_control"),
           (_cfg(flags=1 << 10), veh, _bufs(), "flag"),
           (_cfg(), veh, _bufs(0x10004), "aligned"),
           (_cfg(), veh, A.AuvEnvBuffers(0x10000, None, 0x20000, 0x30000, 0x40000), "NULL"),
           (_cfg(), veh, A.AuvEnvBuffers(0x10000, 0x11000, 0x12000, 0x13000, 0x14000, 0x15002), "status")]
    v2 = A.make_vehicle(W.vehicle_variant(m=-1.0), W.ALLOC)
    bad.append((_cfg(), v2, _bufs(), "mass"))
    v3 = A.make_vehicle(W.vehicle_variant(W=float("nan")), W.ALLOC)
    bad.append((_cfg(), v3, _bufs(), "finite"))
    c4 = _cfg()
    c4.env_offset = 2**32 - 10
    bad.append((c4, veh, _bufs(), "env_offset"))
    for cfg, v, b, word in bad:
        with pytest.raises(A.AuvError) as ei:
            A.auv_create(cfg, v, b)
        assert ei.value.code == A.AUV_EINVAL
        assert word in str(ei.value), (word, str(ei.value))


def test_argument_errors_before_any_launch():
    from paper_2512_13359_amd import _abi as A
    h = A.auv_create(_cfg(), A.make_vehicle(W.VEHICLE, W.ALLOC), _bufs())
    rc = A.lib.auv_rollout(h, 0, A.AUV_ACT_RANDOM, None, None, None, None)
    assert rc == A.AUV_EINVAL and "T must be" in A.auv_last_error()
    rc = A.lib.auv_step(h, 9, None, None, None, None, None, None, None)
    assert rc == A.AUV_EINVAL and "mode" in A.auv_last_error()
    rc = A.lib.auv_step(h, A.AUV_ACT_EXTERNAL, None, None, None, None, None, None, None)
    assert rc == A.AUV_EINVAL and "actions" in A.auv_last_error()
    rc = A.lib.auv_step(h, A.AUV_ACT_POLICY_MEAN, None, None, None, None, None, None, None)
    assert rc == A.AUV_EINVAL and "policy" in A.auv_last_error()
    mlp = A.AuvMlp(0x1000, 0x2000, 0x3000, 8)
    rc = A.lib.auv_step(h, A.AUV_ACT_RANDOM, None, ctypes.byref(mlp), None, None, None, None, None)
    assert rc == A.AUV_EINVAL and "policy" in A.auv_last_error()
    bad_net = A.AuvMlp(0x1000, 0x2000, 0x3000, 3)
    rc = A.lib.auv_step(h, A.AUV_ACT_POLICY_MEAN, None, ctypes.byref(bad_net), None, None, None, None, None)
    assert rc == A.AUV_EINVAL and "n_out" in A.auv_last_error()
    # a handle without a status buffer has nothing to read: refused before any GPU call
    nf = ctypes.c_uint32(7)
    rc = A.lib.auv_get_status(h, ctypes.byref(nf), None, None)
    assert rc == A.AUV_EINVAL and "status" in A.auv_last_error() and nf.value == 7
    rc = A.lib.auv_rollout(h, 10, A.AUV_ACT_RANDOM, None, None,
                           ctypes.byref(A.AuvRolloutBuffers(stats=0x1000)), None)
    assert rc == A.AUV_EINVAL and "stats_work" in A.auv_last_error()
    rc = A.lib.auv_gae(0, 10, *([0x1000] * 4), 0.99, 0.95, 0x1000, 0x1000, None)
    assert rc == A.AUV_EINVAL
    assert A.auv_get_global_step(h) == 0
    A.auv_destroy(h)
    assert A.auv_stats_work_floats(4096, 10) == 3 * 10 * 4 * 64
    assert A.auv_stats_work_floats(65, 2) == 3 * 2 * 4 * 2


def test_value_regression_sizes_and_argument_errors():
    """auv_ppo_fit_work_bytes: -1 outside 16 <= M <= 2^28, 1 <= batches <= M / 16; else the
    minibatch workspace plus two index slots.  auv_ppo_fit_value rejects bad arguments on the
    host (no GPU needed)."""
    from paper_2512_13359_amd import _abi as A
    assert A.auv_ppo_fit_work_bytes(15, 1) == -1 and A.auv_ppo_fit_work_bytes(64, 5) == -1
    assert A.auv_ppo_fit_work_bytes(64, 0) == -1 and A.auv_ppo_fit_work_bytes((1 << 28) + 16, 1) == -1
    M, b = 131072, 4
    B = M // 16 // b * 16
    base = A.auv_ppo_work_bytes(B)
    assert A.auv_ppo_fit_work_bytes(M, b) == (base + 255) // 256 * 256 + 2 * M * 4
    cfg = A.make_ppo_config(vf_coef=2.0, ent_coef=0.0, max_grad_norm=0.0, normalize_adv=False)
    net = A.AuvPpoNet(0x1000, 0x1000, 0x1000, 0x1000, 1)
    mlp = A.AuvMlp()
    batch = A.AuvPpoBatch()
    rc = A.lib.auv_ppo_fit_value(ctypes.byref(cfg), ctypes.byref(mlp), ctypes.byref(net), ctypes.byref(batch), 1, 1, 0,
                                 0, 0x1000, 0x1000, 0x1000, 0x1000, None)
    assert rc == A.AUV_EINVAL


def test_binding_structs_match_header_sizes():
    from paper_2512_13359_amd import _abi as A
    assert ctypes.sizeof(A.AuvVehicle) == 4 * (1 + 3 + 6 + 6 + 6 + 2 + 3 + 1 + 48)
    assert ctypes.sizeof(A.AuvConfig) == 32
    assert ctypes.sizeof(A.AuvRolloutBuffers) == 80
    assert ctypes.sizeof(A.AuvEnvBuffers) == 48
    v = A.make_vehicle(W.VEHICLE, W.ALLOC)
    assert np.allclose(np.array(v.alloc).reshape(6, 8), W.ALLOC)
