"""Helpers shared by the GPU parity tests."""
import numpy as np
import torch

import workloads as W
from oracle import env as oenv


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2512_13359_amd  # noqa: F401  (fails loudly if libauv.so is missing)


def gpu_env(cfg, vehicle=None, alloc=None):
    from paper_2512_13359_amd import AuvEnv
    return AuvEnv(cfg, W.VEHICLE if vehicle is None else vehicle, W.ALLOC if alloc is None else alloc)


def oracle_env(cfg, vehicle=None, alloc=None):
    e = oenv.Env(cfg, W.VEHICLE if vehicle is None else vehicle, W.ALLOC if alloc is None else alloc)
    return e


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def rel_err(got, want):
    """|got - want| / max(|want|, 1), elementwise."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    return np.abs(got - want) / np.maximum(np.abs(want), 1.0)


def quat_aligned(q_got, q_ref):
    """Quaternions of the GPU trajectory, sign-aligned to the oracle's (q ~ -q)."""
    s = np.sign(np.sum(q_got * q_ref, axis=0, keepdims=True))
    s[s == 0] = 1
    return q_got * s


def announce(msg):
    print(f"[gpu-test] {msg}", flush=True)
