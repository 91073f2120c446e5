"""Benchmark of the batched AUV rollout on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4]

One bench step is one auv_rollout launch over the whole workload: for the headline
workload (16384 envs x 2000 control steps, 4 RK4 substeps per 0.04 s step, Lissajous
references, randomisation and current, bf16 MFMA policy mean, per-step batch statistics)
that is 32.8 M env-steps of physics + policy.  Inputs (env state, weights) are resident
in HBM before the timed region.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "env-steps/sec (physics+policy) at 16384 envs; % of FP32/MFMA roofline"

# Algorithmic work per env-step of the headline workload (formula counts, padding
# excluded): bf16 MFMA FLOP of the 23-256-256-8 MLP, fp32 VALU FLOP of physics +
# observation + reward, transcendental ops (512 tanh = exp + reciprocal each).
F_MFMA = 2 * (23 * 256 + 256 * 256 + 256 * 8)      # 146,944
F_VALU = 4815
N_TRANS = 1024
# MI355X peaks: published dense bf16 MFMA and fp32 vector rates; transcendentals
# (v_exp_f32, v_rcp_f32) issue at a quarter of the fp32 FMA lane rate, 8 lanes per SIMD per
# clock: 256 CU x 4 SIMD x 8 lanes x 2.4 GHz (auv_probe_rate measures 0.86 of it,
# profiles/unit_rate_probe.txt).
P_MFMA = 2.5e15
P_VALU = 157.3e12
P_TRANS = 256 * 4 * 8 * 2.4e9
HBM_PEAK = 8.0e12

# The translation unit of the rollout kernel (auv_policy.hip and everything it includes).
KERNEL_SOURCES = ["auv_policy.hip", "auv_internal.hpp", "auv_device.hpp", "env_lane.hpp", "quad_env.hpp",
                  "mlp_mfma.hpp", "mlp_tile.hpp"]
COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_policy_rollout_c4_counters.txt")


def rollout_flags() -> list:
    """The compile flags of the rollout's source, as the build script sets them."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("auv_build", os.path.join(ROOT, "paper_2512_13359_amd", "build.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return list(m.HIPCC_FLAGS) + list(m.EXTRA_FLAGS.get(KERNEL_SOURCES[0], []))


def source_hash() -> str:
    """Hash of the rollout kernel's sources and of its compile flags."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2512_13359_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    h.update(" ".join(rollout_flags()).encode())
    return h.hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per launch of the rollout kernel from the committed counter summary,
    or None if it is missing or was taken on different kernel sources."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    kv = {}
    for line in open(COUNTERS_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(cfg: dict, n_steps: int) -> dict:
    """The fp64 oracle on a bounded sample of the same workload (host cores): all envs of the
    workload over a prefix of n_steps control steps (min(T, 100) for the closed-loop
    workloads), BLAS threads = the cores this process may run on."""
    import numpy as np
    import threadpoolctl

    import workloads as W
    from oracle import env as oenv

    n = cfg["n_envs"]
    cores = len(os.sched_getaffinity(0))
    with threadpoolctl.threadpool_limits(limits=cores):
        info = threadpoolctl.threadpool_info()
        blas = [f"{i.get('internal_api', '?')} {i.get('version', '?')} ({i.get('num_threads', '?')} threads)"
                for i in info if i.get("user_api") == "blas"]
        pol = W.mlp_weights(8, W.POLICY_SEED)
        e = oenv.Env(cfg, W.VEHICLE, W.ALLOC)
        e.reset()
        t0 = time.perf_counter()
        e.rollout(n_steps, cfg["mode"], policy=pol)
        dt = time.perf_counter() - t0
    return {"value": n * n_steps / dt, "unit": "env-steps/s", "cores": cores, "kind": "oracle",
            "sample": f"{n} envs x the first {n_steps} control steps of the same workload (fp64 NumPy, "
                      f"{dt:.1f} s)",
            "cpu_model": _cpu_model(), "numpy": np.__version__, "blas": blas}


def c5_measure(reps: int = 3, rollout_reps: int = 7) -> dict:
    """PPO-buffer workload (65536 envs x 64 steps, sampled actions, value head, staggered
    episodes): rollout time and write bandwidth of the structure-of-arrays buffer, then the
    GAE scan with its inputs evicted from the Infinity Cache (cold) and resident (warm), each
    timed over six back-to-back scans."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp
    from paper_2512_13359_amd import _abi as A

    cfg = W.config("c5")
    n, T = cfg["n_envs"], cfg["T"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    pol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    val = upload_mlp(W.mlp_weights(1, W.VALUE_SEED))
    bufs = env.rollout_buffers(T, record=("obs", "act", "logp", "value", "reward", "done", "last_value"))
    ev = lambda: torch.cuda.Event(enable_timing=True)
    times = []
    for k in range(rollout_reps + 1):   # median of seven launches after one warm-up
        env.reset()
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        env.rollout(T, cfg["mode"], policy=pol, value=val, bufs=bufs)
        e1.record()
        torch.cuda.synchronize()
        if k:
            times.append(e0.elapsed_time(e1) * 1e-3)
    t_roll = sorted(times)[len(times) // 2]
    buf_bytes = (A.OBS_DIM + A.ACT_DIM + 4) * 4 * T * n + 4 * n
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    # 512 MiB swept by a read before a cold measurement: it evicts the 256 MB Infinity Cache and,
    # unlike a write, leaves no dirty lines whose write-back the measured scans would pay for
    scratch = torch.ones(1 << 27, device="cuda")
    gae_bytes = 20 * T * n + 4 * n
    # K copies of the scan's inputs (6 x 50 MB, more than the Infinity Cache holds): cold = K
    # back-to-back scans of the K copies after the cache was flushed, warm = K scans of one
    # resident copy; per-scan time = events around the K launches / K (launch overhead amortised)
    K = 6
    copies = [[bufs[k].clone() for k in ("reward", "value", "done", "last_value")] for _ in range(K)]
    res = {}
    for kind in ("cold", "warm"):
        ts = []
        for _ in range(reps):
            if kind == "cold":
                scratch.sum()
            else:
                A.auv_gae(T, n, *copies[0], 0.99, 0.95, adv, ret)
            torch.cuda.synchronize()
            e0, e1 = ev(), ev()
            e0.record()
            for c in range(K):
                A.auv_gae(T, n, *copies[c if kind == "cold" else 0], 0.99, 0.95, adv, ret)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3 / K)
        res[kind] = sorted(ts)[len(ts) // 2]
    del copies
    return {"workload": f"c5: {n} envs x {T} steps, sampled actions + value head, staggered episodes, "
                        f"PPO buffer (obs 23, act 8, logp, value, reward, done fp32), GAE gamma 0.99 lambda 0.95",
            "rollout_ms": t_roll * 1e3, "env_steps_per_s": n * T / t_roll,
            "buffer_bytes": buf_bytes, "buffer_write_GBps": buf_bytes / t_roll / 1e9,
            "gae_bytes": gae_bytes, "gae_ms_cold": res["cold"] * 1e3, "gae_GBps_cold": gae_bytes / res["cold"] / 1e9,
            "gae_ms_warm": res["warm"] * 1e3, "gae_GBps_warm": gae_bytes / res["warm"] / 1e9,
            "gae_hbm_frac_cold": gae_bytes / res["cold"] / 8e12}


# algorithmic MFMA work of one PPO sample: forward and backward (dW and dX products, no
# input gradient) of the 23-256-256-8 policy and the 23-256-256-1 value net
PPO_FLOP_PER_SAMPLE = (2 * (23 * 256 + 256 * 256 + 256 * 8) + 2 * 2 * 8 * 256 + 2 * 2 * 256 * 256 + 2 * 256 * 23
                       + 2 * (23 * 256 + 256 * 256 + 256) + 2 * 2 * 256 + 2 * 2 * 256 * 256 + 2 * 256 * 23)


def ppo_measure(reps: int = 5) -> dict:
    """PPO update (gradient of both networks + Adam) on minibatches of 262144 samples drawn
    in 16-sample blocks from a c5-sized buffer (65536 envs x 64 steps) of synthetic data."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import PpoLearner

    P = W.PPO
    M, B = P["M"], P["B"]
    g = torch.Generator(device="cuda").manual_seed(21)
    obs = torch.rand(23, M, device="cuda", generator=g) * 2 - 1
    act = torch.randn(8, M, device="cuda", generator=g) * 0.6
    logp = torch.randn(M, device="cuda", generator=g) * 0.1 - 6.0
    adv = torch.randn(M, device="cuda", generator=g)
    ret = torch.randn(M, device="cuda", generator=g)
    hp = {k: P[k] for k in ("clip_eps", "vf_coef", "ent_coef", "max_grad_norm", "lr", "beta1", "beta2", "adam_eps",
                            "normalize_adv")}
    L = PpoLearner(W.mlp_weights(8, W.POLICY_SEED), W.mlp_weights(1, W.VALUE_SEED), **hp)
    batch = L.batch(obs, act, logp, adv, ret)
    idx = [torch.from_numpy(W.ppo_minibatch_idx(M, B, seed=100 + k)).cuda() for k in range(reps + 1)]
    ev = lambda: torch.cuda.Event(enable_timing=True)
    times = []
    for k in range(reps + 1):
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        L.update(batch, idx[k])
        e1.record()
        torch.cuda.synchronize()
        if k:
            times.append(e0.elapsed_time(e1) * 1e-3)
    t = sorted(times)[len(times) // 2]
    # the same updates enqueued back to back, as a training loop runs them (the single-update
    # time above also holds the wait for the host to issue its first kernels)
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for k in range(1, reps + 1):
        L.update(batch, idx[k])
    e1.record()
    torch.cuda.synchronize()
    t_b2b = e0.elapsed_time(e1) * 1e-3 / reps
    st = L.stats.cpu().numpy()
    assert (st == st).all(), "non-finite PPO statistics"
    ach = PPO_FLOP_PER_SAMPLE * B / t
    return {"workload": f"PPO update: minibatch {B} of a {M}-sample buffer (16-sample blocks), clipped surrogate "
                        f"+ value loss, both 23-256-256 MLPs forward + backward on bf16 MFMA, global-norm clip, Adam",
            "minibatch": B, "update_ms": t * 1e3, "samples_per_s": B / t,
            "mfma_flop_per_sample": PPO_FLOP_PER_SAMPLE, "achieved_TFLOPs": ach / 1e12,
            "frac_of_bf16_peak": ach / P_MFMA,
            "back_to_back": {"updates": reps, "update_ms": t_b2b * 1e3, "samples_per_s": B / t_b2b,
                             "achieved_TFLOPs": PPO_FLOP_PER_SAMPLE * B / t_b2b / 1e12}}


def paper_task_measure(reps: int = 3) -> dict:
    """The paper's own task (12-D observation, 6-D wrench, five-term reward) at the paper's
    training scale: 4096 envs x one 512-step episode, policy mean (12-256-256-6) and random
    actions on the Fossen model, and the policy on the inertia-box fluid model of the paper's
    MJX simulation; env-steps/s per launch."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp

    cfg = W.config("c6")
    n, T = cfg["n_envs"], cfg["T"]
    pol = upload_mlp(W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12))
    out = {"workload": f"c6: paper task, {n} envs x {T} steps (one episode), {cfg['substeps']} RK4 substeps "
                       f"per {cfg['dt_control']} s, gravity randomisation, goals within 2 m / 60 deg"}
    runs = (("policy", W.MODE_POLICY_MEAN, pol, W.PAPER_TASK), ("random", W.MODE_RANDOM, None, W.PAPER_TASK),
            ("policy_inertia_box", W.MODE_POLICY_MEAN, pol, W.PAPER_TASK_BOX))
    for name, mode, p, task in runs:
        env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
        env.set_task(task)
        ts = []
        for k in range(reps + 1):
            env.reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            env.rollout(T, mode, policy=p)
            e1.record()
            torch.cuda.synchronize()
            if k:
                ts.append(e0.elapsed_time(e1) * 1e-3)
        t = sorted(ts)[len(ts) // 2]
        out[name] = {"launch_ms": t * 1e3, "env_steps_per_s": n * T / t}
    return out


def paper_training_measure(reps: int = 2, epochs: int = 4, minibatch: int = 262144) -> dict:
    """One PPO training iteration on the paper's own task at its training scale: a sampled
    rollout of 4096 envs x one 512-step episode with the value head, GAE, then `epochs`
    passes of minibatch updates (gradient + Adam) over the 2.1 M samples."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, PpoLearner
    from paper_2512_13359_amd import _abi as A

    cfg = W.config("c6")
    n, T = cfg["n_envs"], cfg["T"]
    M = n * T
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    P = W.PPO
    L = PpoLearner(W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.VALUE_SEED, n_in=12),
                   **{k: P[k] for k in ("clip_eps", "vf_coef", "ent_coef", "max_grad_norm", "lr", "beta1", "beta2",
                                        "adam_eps", "normalize_adv")})
    bufs = env.rollout_buffers(T, record=("obs", "act", "logp", "value", "reward", "done", "last_value"), value=True)
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    batch = L.batch(bufs["obs"].reshape(23, M), bufs["act"].reshape(8, M), bufs["logp"].reshape(M), adv.reshape(M),
                    ret.reshape(M))
    n_mb = M // minibatch
    idx = [torch.from_numpy(W.ppo_minibatch_idx(M, M, seed=200 + e)).cuda() for e in range(epochs)]
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    times, parts = [], []
    for k in range(reps + 1):
        torch.cuda.synchronize()
        e = [ev() for _ in range(4)]
        e[0].record()
        env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
        e[1].record()
        A.auv_gae(T, n, bufs["reward"], bufs["value"], bufs["done"], bufs["last_value"], 0.99, 0.95, adv, ret)
        e[2].record()
        for ep in range(epochs):
            for j in range(n_mb):
                L.update(batch, idx[ep][j * minibatch:(j + 1) * minibatch])
        e[3].record()
        torch.cuda.synchronize()
        if k:
            times.append(e[0].elapsed_time(e[3]) * 1e-3)
            parts.append([e[i].elapsed_time(e[i + 1]) for i in range(3)])
    st = L.stats.cpu().numpy()
    assert (st == st).all(), "non-finite PPO statistics"
    t = sorted(times)[len(times) // 2]
    p = parts[times.index(t)]
    return {"workload": f"paper task PPO iteration: {n} envs x {T}-step episode (sampled, value head), GAE, "
                        f"{epochs} epochs x {n_mb} minibatches of {minibatch}",
            "iteration_ms": t * 1e3, "rollout_ms": p[0], "gae_ms": p[1], "ppo_ms": p[2],
            "hundred_episodes_s": 100 * t}


def paper_learning_measure(iters: int = 150, epochs: int = 4, minibatch: int = 262144) -> dict:
    """PPO training on the paper's own task at its training scale (4096 envs x one 512-step
    episode per iteration, GAE, `epochs` passes of minibatch updates), from the seeded initial
    networks: the mean step reward of each iteration's rollout, and the wall clock of the whole
    run (host work included)."""
    import time

    import numpy as np
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, PpoLearner
    from paper_2512_13359_amd import _abi as A

    cfg = W.config("c6")
    n, T = cfg["n_envs"], cfg["T"]
    M = n * T
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    P = W.PPO
    L = PpoLearner(W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.VALUE_SEED, n_in=12),
                   **{k: P[k] for k in ("clip_eps", "vf_coef", "ent_coef", "max_grad_norm", "lr", "beta1", "beta2",
                                        "adam_eps", "normalize_adv")})
    bufs = env.rollout_buffers(T, record=("obs", "act", "logp", "value", "reward", "done", "last_value"), value=True)
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    batch = L.batch(bufs["obs"].reshape(23, M), bufs["act"].reshape(8, M), bufs["logp"].reshape(M), adv.reshape(M),
                    ret.reshape(M))
    n_mb = M // minibatch
    rng = np.random.default_rng(0)
    perms = [torch.from_numpy(W.ppo_minibatch_idx(M, M, seed=int(rng.integers(1 << 30)))).cuda() for _ in range(16)]
    rewards = torch.empty(iters, device="cuda")
    torch.cuda.synchronize()
    t0 = time.time()
    for it in range(iters):
        env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
        A.auv_gae(T, n, bufs["reward"], bufs["value"], bufs["done"], bufs["last_value"], 0.99, 0.95, adv, ret)
        rewards[it] = bufs["reward"].mean()
        for ep in range(epochs):
            perm = perms[(it * epochs + ep) % len(perms)]
            for j in range(n_mb):
                L.update(batch, perm[j * minibatch:(j + 1) * minibatch])
    torch.cuda.synchronize()
    wall = time.time() - t0
    r = rewards.cpu().numpy()
    st = L.stats.cpu().numpy()
    assert np.isfinite(r).all() and (st == st).all(), "non-finite training statistics"
    marks = sorted({0, iters // 3, 2 * iters // 3, iters - 1})
    return {"workload": f"paper task PPO training from the seeded networks: {iters} iterations of {n} envs x {T} "
                        f"steps (sampled, value head), GAE, {epochs} epochs x {n_mb} minibatches of {minibatch}",
            "iterations": iters, "wall_s": wall, "ms_per_iteration": wall / iters * 1e3,
            "mean_step_reward": {str(k): float(r[k]) for k in marks},
            "last_value_loss": float(st[1]), "last_entropy": float(st[2]), "last_approx_kl": float(st[3])}


# Dense-contraction work per env-step of a SHAC window on the paper task's 12-256-256-6
# policy (padding excluded): the forward, the input gradient (the same matrices
# transposed) and the weight gradient.
SHAC_FLOP_PER_STEP = 3 * 2 * (12 * 256 + 256 * 256 + 256 * 6)


def shac_measure(n_envs: int, reps: int = 16) -> dict:
    """SHAC on the paper task: windows of h = 32 control steps of n_envs environments with the
    sampled policy in the loop and a terminal value (auv_shac_window: forward, reverse sweep
    through RK4 + Fossen and the policy, parameter gradient), the actor's Adam step, and the
    critic's regression on the window's TD(lambda) targets (16 passes x 4 minibatches of
    value-only gradient + Adam).  Consecutive windows tile the 512-step episodes."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, ShacLearner

    cfg = W.config("c6", n_envs=n_envs)
    h = W.SHAC["h"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    L = ShacLearner(env, W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12),
                    h=h, gamma=W.SHAC["gamma"], max_grad_norm=W.SHAC["max_grad_norm"])
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    win, stp, crit = [], [], []
    for k in range(reps + 1):
        torch.cuda.synchronize()
        e = [ev() for _ in range(4)]
        e[0].record()
        L.window()
        e[1].record()
        L.step()
        e[2].record()
        if k < 6:   # the critic's regression (16 passes x 4 minibatches) on the first windows only:
            # five timed, since one host stall among its 256 launches can double a sample
            L.critic_update(iterations=16, batches=4, seed=k)
        e[3].record()
        torch.cuda.synchronize()
        if k:
            win.append(e[0].elapsed_time(e[1]) * 1e-3)
            stp.append(e[1].elapsed_time(e[2]) * 1e-3)
            if k < 6:
                crit.append(e[2].elapsed_time(e[3]) * 1e-3)
    st = L.stats.cpu().numpy()
    assert (st == st).all(), "non-finite SHAC statistics"
    tw = sorted(win)[len(win) // 2]
    ts = sorted(stp)[len(stp) // 2]
    tc = sorted(crit)[len(crit) // 2]
    steps = n_envs * h
    windows_per_episode = cfg["episode_len"] // h
    return {"workload": f"SHAC on the paper task: {n_envs} envs, windows of {h} steps (sampled policy, terminal "
                        f"value), actor gradient through RK4 + Fossen and the 12-256-256-6 policy, Adam step",
            "n_envs": n_envs, "h": h, "window_ms": tw * 1e3, "actor_step_ms": ts * 1e3,
            "env_steps_per_s": steps / tw, "mfma_flop_per_env_step": SHAC_FLOP_PER_STEP,
            "achieved_TFLOPs": SHAC_FLOP_PER_STEP * steps / tw / 1e12,
            "frac_of_bf16_peak": SHAC_FLOP_PER_STEP * steps / tw / P_MFMA,
            "critic_ms": tc * 1e3, "iteration_ms": (tw + ts + tc) * 1e3,
            "hundred_episodes_actor_s": 100 * windows_per_episode * (tw + ts),
            "hundred_episodes_s": 100 * windows_per_episode * (tw + ts + tc)}


def shac_learning_measure(n_envs: int, windows: int = 320) -> dict:
    """SHAC training on the paper task from the seeded networks: `windows` iterations (window,
    actor step, critic update of 16 x 4 minibatches), consecutive windows tiling the 512-step
    episodes; the mean step reward of each window and of each episode's 16 windows, and the
    wall clock of the whole run (host work included)."""
    import time

    import numpy as np
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, ShacLearner

    cfg = W.config("c6", n_envs=n_envs)
    h = W.SHAC["h"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    L = ShacLearner(env, W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12),
                    h=h, gamma=W.SHAC["gamma"], max_grad_norm=W.SHAC["max_grad_norm"])
    r = torch.empty(windows, device="cuda")
    torch.cuda.synchronize()
    t0 = time.time()
    for k in range(windows):
        L.window()
        r[k] = L.rec["reward"].mean()
        L.step()
        L.critic_update(iterations=16, batches=4, seed=k)
    torch.cuda.synchronize()
    wall = time.time() - t0
    rr = r.cpu().numpy()
    wpe = cfg["episode_len"] // h
    ep = rr[:(windows // wpe) * wpe].reshape(-1, wpe).mean(axis=1)
    assert np.isfinite(rr).all() and np.isfinite(L.stats.cpu().numpy()).all(), "non-finite SHAC training"
    return {"workload": f"SHAC training on the paper task from the seeded networks: {n_envs} envs, {windows} windows "
                        f"of {h} steps ({len(ep)} episodes), actor step and critic update (16 x 4 minibatches) each",
            "n_envs": n_envs, "windows": windows, "wall_s": wall, "ms_per_window": wall / windows * 1e3,
            "first_windows_mean_step_reward": [float(x) for x in rr[:4]],
            "episode_mean_step_reward": {str(i): float(ep[i]) for i in sorted({0, 1, len(ep) // 2, len(ep) - 1})}}


def small_configs_measure(reps: int = 3) -> dict:
    """The 4096-env workloads (random actions c2, policy mean c3): env-steps/s per launch.
    4096 envs are 256 one-wave blocks of the quad-layout loop (c2) or 256 one-tile workgroups of
    the fused rollout (c3): a quarter of the SIMDs carry physics, so both are capped by N."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp

    out = {}
    pol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    for name in ("c2", "c3"):
        cfg = W.config(name)
        n, T = cfg["n_envs"], cfg["T"]
        env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
        bufs = env.rollout_buffers(T, record=("stats",))
        ts = []
        for k in range(reps + 1):
            env.reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            env.rollout(T, cfg["mode"], policy=pol if cfg["mode"] >= W.MODE_POLICY_MEAN else None, bufs=bufs)
            e1.record()
            torch.cuda.synchronize()
            if k:
                ts.append(e0.elapsed_time(e1) * 1e-3)
        t = sorted(ts)[len(ts) // 2]
        out[name] = {"n_envs": n, "control_steps": T, "launch_ms": t * 1e3, "env_steps_per_s": n * T / t}
    return out


def probe_rates(reps: int = 3) -> dict:
    """Throughput of the units that bound the rollout (auv_probe_rate): v_exp_f32, v_rcp_f32
    and v_fma_f32 in lane operations per second, bf16 MFMA in FLOP/s, each from the median of
    reps launches of 2048 workgroups (eight waves per SIMD) after one warm-up."""
    import torch

    from paper_2512_13359_amd import _abi as A

    blocks = 2048
    sink = torch.empty(blocks * 256, device="cuda")
    out = {}
    for name, kind, iters in (("exp_lane_ops_per_s", A.AUV_PROBE_EXP, 20000), ("rcp_lane_ops_per_s", A.AUV_PROBE_RCP, 20000),
                              ("fma_lane_ops_per_s", A.AUV_PROBE_FMA, 40000),
                              ("mfma_bf16_flop_per_s", A.AUV_PROBE_MFMA_BF16, 200)):
        times = []
        for k in range(reps + 1):
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            A.auv_probe_rate(kind, blocks, iters, sink)
            e1.record()
            torch.cuda.synchronize()
            if k:
                times.append(e0.elapsed_time(e1) * 1e-3)
        t = sorted(times)[len(times) // 2]
        ops = blocks * 4 * 8 * iters * 16384 if kind == A.AUV_PROBE_MFMA_BF16 else blocks * 256 * 8 * iters
        out[name] = ops / t
        out[name.replace("_per_s", "_ms")] = t * 1e3
    return out


SWEEP_ENVS = (64, 256, 1024, 4096, 8192, 16384, 32768, 65536)


def sweep_measure(reps: int = 3) -> list:
    """The headline workload's rollout (policy mean, 4 RK4 substeps, Lissajous references,
    2000 control steps) at environment counts from 64 to 65536: launch time by HIP events
    (median of reps after one warm-up launch), env-steps/s and the fraction of the same
    per-env-step lower bound as the headline line (report only)."""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp

    pol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    t_lb = F_MFMA / P_MFMA + F_VALU / P_VALU + N_TRANS / P_TRANS
    out = []
    for n in SWEEP_ENVS:
        cfg = W.config("c4", n_envs=n)
        T = cfg["T"]
        env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
        env.reset()
        bufs = env.rollout_buffers(T, record=("stats",))
        times = []
        for k in range(reps + 1):
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            env.rollout(T, cfg["mode"], policy=pol, bufs=bufs)
            e1.record()
            torch.cuda.synchronize()
            if k:
                times.append(e0.elapsed_time(e1) * 1e-3)
        t = sorted(times)[len(times) // 2]
        assert torch.isfinite(bufs["stats"]).all(), f"non-finite statistics at {n} envs"
        out.append({"n_envs": n, "control_steps": T, "launch_ms": t * 1e3, "env_steps_per_s": n * T / t,
                    "frac": t_lb * n * T / t})
        print(json.dumps({"sweep_point": out[-1]}), file=sys.stderr, flush=True)
        del env, bufs
    return out


def spin_up(seconds: float = 0.4) -> None:
    """Run the headline rollout for a moment before anything is measured, so that every mode
    (also the short ones: --ppo-only, --c5-only, ...) measures in the clock state the full
    run's later sections see (after the headline rollout), not while the clock is still
    ramping up from idle.  (A bf16 GEMM load instead left the clock about 9 % lower.)"""
    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp

    cfg = W.config("c4")
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.reset()
    pol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        env.rollout(cfg["T"], cfg["mode"], policy=pol)
        torch.cuda.synchronize()
    del env, pol


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c4", choices=["c3", "c4"])
    ap.add_argument("--cpu-steps", type=int, default=100,
                    help="oracle control steps for the CPU baseline, at most T (0: skip)")
    ap.add_argument("--no-c5", action="store_true", help="skip the PPO-buffer (c5) rollout and GAE measurement")
    ap.add_argument("--no-ppo", action="store_true", help="skip the PPO-update measurement")
    ap.add_argument("--ppo-only", action="store_true", help="only measure the PPO update and print it")
    ap.add_argument("--paper-only", action="store_true",
                    help="only measure the paper task (c6, training iteration, 150 training iterations)")
    ap.add_argument("--shac-only", action="store_true", help="only measure the SHAC windows (4096 and 512 envs)")
    ap.add_argument("--c5-only", action="store_true", help="only measure the PPO-buffer rollout and GAE (c5)")
    ap.add_argument("--sweep", action="store_true",
                    help="only measure the headline rollout at 64 to 65536 envs and print it")
    ap.add_argument("--probe-rates", action="store_true",
                    help="only measure the exp / rcp / fma / bf16 MFMA unit rates (auv_probe_rate) and print them")
    ap.add_argument("--no-spin-up", action="store_true",
                    help="skip the 0.4 s of headline rollouts run before anything is measured")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run one plain device copy of MIB MiB (counter calibration) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        src = torch.ones(args.calibrate_copy * (1 << 18), device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": src.numel() * 4}))
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (the rollout has no cross-GPU step to measure); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        return 2

    import torch

    import workloads as W
    from paper_2512_13359_amd import AuvEnv, upload_mlp

    torch.cuda.set_device(0)
    if not args.no_spin_up:
        spin_up()
    if args.ppo_only:
        print(json.dumps({"ppo": ppo_measure()}), flush=True)
        return 0
    if args.paper_only:
        print(json.dumps({"c6": paper_task_measure(), "paper_training": paper_training_measure(),
                          "paper_learning": paper_learning_measure()}), flush=True)
        return 0
    if args.c5_only:
        print(json.dumps({"c5": c5_measure()}), flush=True)
        return 0
    if args.sweep:
        print(json.dumps({"sweep": sweep_measure()}), flush=True)
        return 0
    if args.probe_rates:
        print(json.dumps({"unit_rates": probe_rates()}), flush=True)
        return 0
    if args.shac_only:
        print(json.dumps({"shac": [shac_measure(W.SHAC["n_envs"]), shac_measure(W.SHAC["n_envs_small"])]}),
              flush=True)
        return 0
    cfg = W.config(args.workload)
    n, T = cfg["n_envs"], cfg["T"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.reset()
    pol = upload_mlp(W.mlp_weights(8, W.POLICY_SEED))
    bufs = env.rollout_buffers(T, record=("stats",))
    for _ in range(args.warmup):
        env.rollout(T, cfg["mode"], policy=pol, bufs=bufs)
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record()
        env.rollout(T, cfg["mode"], policy=pol, bufs=bufs)
        ends[k].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_s = sum(s.elapsed_time(e) for s, e in zip(starts, ends)) / args.steps * 1e-3
    stats = bufs["stats"].cpu().numpy()
    assert stats.shape == (3, T) and (stats == stats).all(), "non-finite statistics"

    env_steps = n * T
    value = env_steps * args.steps / wall
    per_env_step_s = launch_s / env_steps
    t_lb = F_MFMA / P_MFMA + F_VALU / P_VALU + N_TRANS / P_TRANS
    # the bound's work in bf16-MFMA-equivalent FLOP: each unit's work scaled to the time it
    # takes at its peak, expressed at the MFMA peak (so peak = the published 2.5 PFLOP/s)
    f_eq = t_lb * P_MFMA
    traffic = recorded_traffic()
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "env-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+bf16",
        "data": "synthetic (seeded Philox resets, seeded N(0,1/fan_in) bf16 weights)",
        "config": {
            "workload": f"{args.workload}: {n} envs x {T} control steps, {cfg['substeps']} RK4 substeps per "
                        f"{cfg['dt_control']} s step, randomisation + current"
                        + (", Lissajous references" if cfg["flags"] & W.FLAG_LISSAJOUS else "")
                        + ", bf16 MFMA policy 23-256-256-8 (mean), batch statistics",
            "n_envs": n, "control_steps": T, "substeps": cfg["substeps"],
            "env_steps_per_launch": env_steps,
        },
        "roofline": {
            "bound": "alu",
            "achieved": f_eq / per_env_step_s / 1e12,
            "peak": P_MFMA / 1e12,
            "unit": "TFLOP/s",
            "unit_note": "bf16-MFMA-equivalent: per env-step MFMA FLOP + fp32 VALU FLOP x (2500/157.3) + "
                         "transcendentals x (2500/19.66), the sum-of-units bound at the MFMA peak",
            "frac": t_lb / per_env_step_s,
            "traffic": traffic,
            "kernel": "k_policy_rollout",
            "launch_ms": launch_s * 1e3,
            "unit_peaks": {"mfma_bf16_tflops": P_MFMA / 1e12, "valu_fp32_tflops": P_VALU / 1e12,
                           "trans_tops": P_TRANS / 1e12},
            "per_env_step": {"mfma_flop": F_MFMA, "valu_flop": F_VALU, "trans_ops": N_TRANS},
            "unit_utilisation": {
                "mfma": F_MFMA / per_env_step_s / P_MFMA,
                "valu": F_VALU / per_env_step_s / P_VALU,
                "trans": N_TRANS / per_env_step_s / P_TRANS,
            },
            "max_of_units_frac": max(F_MFMA / P_MFMA, F_VALU / P_VALU, N_TRANS / P_TRANS) / per_env_step_s,
        },
    }
    if not args.no_c5:
        line["c5"] = c5_measure()
        line.update(small_configs_measure())
        line["sweep"] = sweep_measure()
    if not args.no_ppo and not args.no_c5:
        line["ppo"] = ppo_measure()
        line["c6"] = paper_task_measure()
        line["paper_training"] = paper_training_measure()
        line["paper_learning"] = paper_learning_measure()
        line["shac"] = [shac_measure(W.SHAC["n_envs"]), shac_measure(W.SHAC["n_envs_small"])]
        line["shac_learning"] = shac_learning_measure(W.SHAC["n_envs"])
    if args.cpu_steps > 0:
        line["cpu_baseline"] = cpu_baseline(cfg, min(args.cpu_steps, T))
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
