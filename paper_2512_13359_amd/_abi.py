"""ctypes binding of libauv's C interface (include/auv.h), same names, marshalling only.

Device buffers are torch tensors on the GPU; the binding passes their addresses and the
current HIP stream.  Every compute step runs in libauv's HIP kernels; if the library is
missing the import of this module fails loudly (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # noqa: F401  (brings up the HIP runtime before libauv registers its kernels)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libauv.so")

AUV_OK, AUV_EINVAL, AUV_ENODEV, AUV_ELAUNCH, AUV_ERUNTIME, AUV_ENONFINITE = 0, -1, -2, -3, -4, -5
AUV_ACT_EXTERNAL, AUV_ACT_RANDOM, AUV_ACT_POLICY_MEAN, AUV_ACT_POLICY_SAMPLE = 0, 1, 2, 3
AUV_F_DR, AUV_F_CURRENT, AUV_F_LISSAJOUS, AUV_F_STAGGER = 1, 2, 4, 8
AUV_TASK_WORKLOAD, AUV_TASK_PAPER = 0, 1
AUV_FLUID_FOSSEN, AUV_FLUID_INERTIA_BOX = 0, 1
AUV_STATIC_STATS_FLOATS = 2 * 1024 * 1024
AUV_CONV_UNIFORM, AUV_CONV_UNIFORM_OPEN0, AUV_CONV_AFFINE, AUV_CONV_BF16 = 0, 1, 2, 3
AUV_PROBE_EXP, AUV_PROBE_RCP, AUV_PROBE_FMA, AUV_PROBE_MFMA_BF16 = 0, 1, 2, 3
OBS_DIM, ACT_DIM, STATE_DIM, PARAM_DIM, HIDDEN, ENVS_PER_GROUP = 23, 8, 13, 24, 256, 64

_f = ctypes.c_float
_vp = ctypes.c_void_p


class AuvConfig(ctypes.Structure):
    _fields_ = [("n_envs", ctypes.c_int32), ("substeps", ctypes.c_int32),
                ("episode_len", ctypes.c_int32), ("dt_control", _f), ("seed", ctypes.c_uint64),
                ("flags", ctypes.c_uint32), ("env_offset", ctypes.c_uint32)]


class AuvVehicle(ctypes.Structure):
    _fields_ = [("m", _f), ("inertia", _f * 3), ("added_mass", _f * 6), ("lin_damp", _f * 6),
                ("quad_damp", _f * 6), ("W", _f), ("B", _f), ("r_b", _f * 3), ("f_max", _f),
                ("alloc", _f * 48)]


class AuvEnvBuffers(ctypes.Structure):
    _fields_ = [("state", _vp), ("params", _vp), ("ep_step", _vp), ("episode", _vp), ("obs", _vp), ("status", _vp)]


class AuvMlp(ctypes.Structure):
    _fields_ = [("w", _vp), ("b", _vp), ("log_std", _vp), ("n_out", ctypes.c_int32)]


class AuvRolloutBuffers(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("obs", "act", "logp", "value", "reward", "done", "last_value",
                                   "traj_state", "stats", "stats_work")]


class AuvTask(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("f_max", _f), ("tau_max", _f), ("w_pos", _f), ("d_pos", _f * 3),
                ("w_att", _f), ("w_act", _f), ("w_vel", _f), ("w_mavg", _f), ("beta", _f), ("gamma_lo", _f),
                ("gamma_span", _f), ("euler_max", _f), ("fluid", ctypes.c_int32), ("density", _f),
                ("viscosity", _f)]


class AuvPpoConfig(ctypes.Structure):
    _fields_ = [("clip_eps", _f), ("vf_coef", _f), ("ent_coef", _f), ("max_grad_norm", _f), ("lr", _f),
                ("beta1", _f), ("beta2", _f), ("adam_eps", _f), ("normalize_adv", ctypes.c_int32),
                ("n_actions", ctypes.c_int32)]


class AuvPpoBatch(ctypes.Structure):
    _fields_ = [("obs", _vp), ("act", _vp), ("logp", _vp), ("adv", _vp), ("ret", _vp), ("M", ctypes.c_int64)]


class AuvPpoNet(ctypes.Structure):
    _fields_ = [("theta", _vp), ("adam_m", _vp), ("adam_v", _vp), ("w_bf16", _vp), ("n_out", ctypes.c_int32)]


class AuvShacConfig(ctypes.Structure):
    _fields_ = [("h", ctypes.c_int32), ("mode", ctypes.c_int32), ("gamma", _f), ("max_grad_norm", _f)]


class AuvShacBuffers(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("actions", "obs", "act", "reward", "done", "grad_act", "value_last",
                                   "grad_state0")]


def ppo_nw(n_out: int) -> int:
    """AUV_PPO_NW: packed offset of b1 (the weight matrices' length)."""
    return 256 * 23 + 256 * 256 + n_out * 256


def ppo_nparam(n_out: int) -> int:
    """AUV_PPO_NPARAM: length of a network's packed parameter vector."""
    return ppo_nw(n_out) + 512 + n_out + (8 if n_out == 8 else 0)


class AuvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libauv error {code}: {msg}")
        self.code = code


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2512_13359_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, P = ctypes.c_int32, ctypes.c_int64, ctypes.POINTER
    sig = {
        "auv_stats_work_floats": (i64, [i32, i32]),
        "auv_create": (ctypes.c_int, [P(AuvConfig), P(AuvVehicle), P(AuvEnvBuffers), P(_vp)]),
        "auv_destroy": (ctypes.c_int, [_vp]),
        "auv_reset": (ctypes.c_int, [_vp, _vp]),
        "auv_step": (ctypes.c_int, [_vp, ctypes.c_int, _vp, P(AuvMlp), _vp, _vp, _vp, _vp, _vp]),
        "auv_get_status": (ctypes.c_int, [_vp, P(ctypes.c_uint32), P(ctypes.c_uint32), _vp]),
        "auv_rollout": (ctypes.c_int, [_vp, i32, ctypes.c_int, P(AuvMlp), P(AuvMlp), P(AuvRolloutBuffers), _vp]),
        "auv_rollout_static": (ctypes.c_int, [_vp, i32, ctypes.c_int, P(AuvMlp), P(AuvMlp), P(AuvRolloutBuffers),
                                              _vp]),
        "auv_convert": (ctypes.c_int, [ctypes.c_int, i64, _vp, _f, _f, _vp, _vp]),
        "auv_probe_rate": (ctypes.c_int, [ctypes.c_int, i32, i32, _vp, _vp]),
        "auv_gae": (ctypes.c_int, [i32, i32, _vp, _vp, _vp, _vp, _f, _f, _vp, _vp, _vp]),
        "auv_mlp_forward": (ctypes.c_int, [P(AuvMlp), i32, _vp, _vp, _vp]),
        "auv_get_global_step": (i64, [_vp]),
        "auv_set_global_step": (ctypes.c_int, [_vp, i64]),
        "auv_set_sync_poll_limit": (ctypes.c_int, [_vp, ctypes.c_uint32]),
        "auv_set_task": (ctypes.c_int, [_vp, P(AuvTask)]),
        "auv_ppo_work_bytes": (i64, [i32]),
        "auv_ppo_grad": (ctypes.c_int, [P(AuvPpoConfig), P(AuvMlp), P(AuvMlp), P(AuvPpoBatch), _vp, i32, _vp, _vp,
                                        _vp, _vp, _vp]),
        "auv_ppo_adam": (ctypes.c_int, [P(AuvPpoConfig), i64, P(AuvPpoNet), P(AuvPpoNet), _vp, _vp, _vp, _vp]),
        "auv_ppo_fit_work_bytes": (i64, [i64, i32]),
        "auv_ppo_fit_value": (ctypes.c_int, [P(AuvPpoConfig), P(AuvMlp), P(AuvPpoNet), P(AuvPpoBatch), i32, i32,
                                             ctypes.c_uint64, i64, _vp, _vp, _vp, _vp, _vp]),
        "auv_shac_work_bytes": (i64, [i32, i32]),
        "auv_shac_window": (ctypes.c_int, [_vp, P(AuvShacConfig), P(AuvMlp), P(AuvMlp), P(AuvShacBuffers), _vp, _vp,
                                           _vp, _vp]),
        "auv_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


lib = _load()


def _check(rc: int) -> None:
    if rc != AUV_OK:
        raise AuvError(rc, lib.auv_last_error().decode())


def ptr(t) -> int | None:
    """Device address of a tensor (None for None)."""
    return None if t is None else t.data_ptr()


def stream_ptr(stream=None) -> int | None:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream or None


# ---- the C entry points, same names ---------------------------------------------------

def auv_stats_work_floats(n_envs: int, T: int) -> int:
    return int(lib.auv_stats_work_floats(n_envs, T))


def auv_create(cfg: AuvConfig, veh: AuvVehicle, bufs: AuvEnvBuffers) -> int:
    h = _vp()
    _check(lib.auv_create(ctypes.byref(cfg), ctypes.byref(veh), ctypes.byref(bufs), ctypes.byref(h)))
    return h.value


def auv_destroy(h: int) -> None:
    _check(lib.auv_destroy(h))


def auv_reset(h: int, stream=None) -> None:
    _check(lib.auv_reset(h, stream_ptr(stream)))


def auv_step(h: int, mode: int, actions=None, policy: AuvMlp | None = None, reward=None, done=None, stats=None,
             stats_work=None, stream=None) -> None:
    _check(lib.auv_step(h, mode, ptr(actions), None if policy is None else ctypes.byref(policy), ptr(reward),
                        ptr(done), ptr(stats), ptr(stats_work),
                        stream_ptr(stream)))


def auv_get_status(h: int, stream=None) -> tuple[int, int, int]:
    """(return code, non-finite state components, abandoned waits); AUV_ENONFINITE is a
    result here, not an exception (other failures raise)."""
    nf, ab = ctypes.c_uint32(0), ctypes.c_uint32(0)
    rc = lib.auv_get_status(h, ctypes.byref(nf), ctypes.byref(ab), stream_ptr(stream))
    if rc not in (AUV_OK, AUV_ENONFINITE):
        _check(rc)
    return rc, nf.value, ab.value


def auv_rollout(h: int, T: int, mode: int, policy: AuvMlp | None = None, value: AuvMlp | None = None,
                rbufs: AuvRolloutBuffers | None = None, stream=None) -> None:
    _check(lib.auv_rollout(h, T, mode, None if policy is None else ctypes.byref(policy),
                           None if value is None else ctypes.byref(value),
                           None if rbufs is None else ctypes.byref(rbufs), stream_ptr(stream)))


def auv_rollout_static(h: int, T: int, mode: int, policy: AuvMlp | None = None, value: AuvMlp | None = None,
                       rbufs: AuvRolloutBuffers | None = None, stream=None) -> None:
    _check(lib.auv_rollout_static(h, T, mode, None if policy is None else ctypes.byref(policy),
                                  None if value is None else ctypes.byref(value),
                                  None if rbufs is None else ctypes.byref(rbufs), stream_ptr(stream)))


def auv_convert(kind: int, n: int, inp, lo: float, span: float, out, stream=None) -> None:
    _check(lib.auv_convert(kind, n, ptr(inp), lo, span, ptr(out), stream_ptr(stream)))


def auv_probe_rate(kind: int, blocks: int, iters: int, sink, stream=None) -> None:
    _check(lib.auv_probe_rate(kind, blocks, iters, ptr(sink), stream_ptr(stream)))


def auv_gae(T: int, n_envs: int, reward, value, done, last_value, gamma: float, lam: float,
            adv, ret, stream=None) -> None:
    _check(lib.auv_gae(T, n_envs, ptr(reward), ptr(value), ptr(done), ptr(last_value), gamma, lam,
                       ptr(adv), ptr(ret), stream_ptr(stream)))


def auv_mlp_forward(net: AuvMlp, n_envs: int, obs, out, stream=None) -> None:
    _check(lib.auv_mlp_forward(ctypes.byref(net), n_envs, ptr(obs), ptr(out), stream_ptr(stream)))


def auv_get_global_step(h: int) -> int:
    return int(lib.auv_get_global_step(h))


def auv_set_global_step(h: int, step: int) -> None:
    _check(lib.auv_set_global_step(h, step))


def auv_set_sync_poll_limit(h: int, polls: int) -> None:
    _check(lib.auv_set_sync_poll_limit(h, polls))


def auv_set_task(h: int, task: AuvTask) -> None:
    _check(lib.auv_set_task(h, ctypes.byref(task)))


def auv_ppo_work_bytes(B: int) -> int:
    return int(lib.auv_ppo_work_bytes(B))


def auv_ppo_grad(cfg: AuvPpoConfig, policy: AuvMlp | None, value: AuvMlp, batch: AuvPpoBatch, idx, B: int,
                 grad_policy, grad_value, stats, work, stream=None) -> None:
    _check(lib.auv_ppo_grad(ctypes.byref(cfg), ctypes.byref(policy) if policy is not None else None,
                            ctypes.byref(value), ctypes.byref(batch),
                            ptr(idx), B, ptr(grad_policy), ptr(grad_value), ptr(stats), ptr(work),
                            stream_ptr(stream)))


def auv_ppo_adam(cfg: AuvPpoConfig, t: int, policy: AuvPpoNet | None, value: AuvPpoNet | None, grad_policy,
                 grad_value, stats, stream=None) -> None:
    ref = lambda n: ctypes.byref(n) if n is not None else None  # noqa: E731
    _check(lib.auv_ppo_adam(ctypes.byref(cfg), t, ref(policy), ref(value), ptr(grad_policy), ptr(grad_value),
                            ptr(stats), stream_ptr(stream)))


def auv_ppo_fit_work_bytes(M: int, batches: int) -> int:
    return int(lib.auv_ppo_fit_work_bytes(M, batches))


def auv_ppo_fit_value(cfg: AuvPpoConfig, value: AuvMlp, value_net: AuvPpoNet, batch: AuvPpoBatch, iterations: int,
                      batches: int, seed: int, t0: int, host_stage, grad_value, stats, work, stream=None) -> None:
    """host_stage: pinned CPU int32 tensor of 2 * 16 * (M // 16) entries."""
    _check(lib.auv_ppo_fit_value(ctypes.byref(cfg), ctypes.byref(value), ctypes.byref(value_net), ctypes.byref(batch),
                                 iterations, batches, seed, t0, ptr(host_stage), ptr(grad_value), ptr(stats), ptr(work),
                                 stream_ptr(stream)))


def auv_shac_work_bytes(n_envs: int, h: int) -> int:
    return int(lib.auv_shac_work_bytes(n_envs, h))


def auv_shac_window(h: int, cfg: AuvShacConfig, policy: AuvMlp | None, value: AuvMlp | None,
                    out: AuvShacBuffers | None, grad_policy, stats, work, stream=None) -> None:
    _check(lib.auv_shac_window(h, ctypes.byref(cfg), ctypes.byref(policy) if policy is not None else None,
                               ctypes.byref(value) if value is not None else None,
                               ctypes.byref(out) if out is not None else None, ptr(grad_policy), ptr(stats), ptr(work),
                               stream_ptr(stream)))


def auv_last_error() -> str:
    return lib.auv_last_error().decode()


# ---- struct builders (marshalling) ---------------------------------------------------

def make_config(n_envs, substeps, episode_len, dt_control, seed, flags, env_offset=0) -> AuvConfig:
    return AuvConfig(n_envs, substeps, episode_len, float(np.float32(dt_control)), seed, flags, env_offset)


def make_vehicle(vehicle: dict, alloc) -> AuvVehicle:
    v = AuvVehicle()
    v.m = float(vehicle["m"])
    for name in ("inertia", "added_mass", "lin_damp", "quad_damp", "r_b"):
        arr = np.asarray(vehicle[name], np.float32).ravel()
        getattr(v, name)[:] = [float(x) for x in arr]
    v.W, v.B, v.f_max = float(vehicle["W"]), float(vehicle["B"]), float(vehicle["f_max"])
    v.alloc[:] = [float(x) for x in np.asarray(alloc, np.float32).ravel()]
    return v


def make_mlp(w, b, log_std, n_out: int) -> AuvMlp:
    return AuvMlp(ptr(w), ptr(b), ptr(log_std), n_out)


def make_env_buffers(state, params, ep_step, episode, obs, status=None) -> AuvEnvBuffers:
    return AuvEnvBuffers(ptr(state), ptr(params), ptr(ep_step), ptr(episode), ptr(obs), ptr(status))


def make_task(task: dict) -> AuvTask:
    """auv_task from a dict (kind, f_max, tau_max, w_pos, d_pos, w_att, w_act, w_vel, w_mavg, beta,
    gamma_lo, gamma_span, euler_max; fluid, density, viscosity)."""
    t = AuvTask()
    for k, v in task.items():
        if k == "d_pos":
            t.d_pos[:] = [float(x) for x in v]
        else:
            setattr(t, k, v)
    return t


def make_ppo_config(clip_eps=0.2, vf_coef=0.5, ent_coef=0.0, max_grad_norm=0.5, lr=3e-4, beta1=0.9,
                    beta2=0.999, adam_eps=1e-8, normalize_adv=True, n_actions=8) -> AuvPpoConfig:
    return AuvPpoConfig(clip_eps, vf_coef, ent_coef, max_grad_norm, lr, beta1, beta2, adam_eps, int(bool(normalize_adv)),
                        n_actions)


def make_ppo_batch(obs, act, logp, adv, ret, M: int) -> AuvPpoBatch:
    return AuvPpoBatch(ptr(obs), ptr(act), ptr(logp), ptr(adv), ptr(ret), M)


def make_shac_config(h: int, mode: int, gamma: float, max_grad_norm: float = 0.0) -> AuvShacConfig:
    return AuvShacConfig(h, mode, float(np.float32(gamma)), float(np.float32(max_grad_norm)))


def make_shac_buffers(**kw) -> AuvShacBuffers:
    return AuvShacBuffers(**{k: ptr(v) for k, v in kw.items()})


def make_rollout_buffers(**kw) -> AuvRolloutBuffers:
    return AuvRolloutBuffers(**{k: ptr(v) for k, v in kw.items()})
