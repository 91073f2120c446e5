"""AuvEnv: owns the device buffers (torch tensors) of one batch of environments and calls
libauv through the C binding.  Memory management and argument marshalling only."""
from __future__ import annotations

import numpy as np
import torch

from . import _abi as A


def pad_to_kernel_layout(net: dict) -> dict:
    """A 12-input or 6-output network in the 23-input / 8-output layout the kernels read:
    zero W1 columns past the inputs, zero W3 rows, b3 entries and log_std past the outputs
    (exactly the same function on the inputs it has)."""
    W1 = np.asarray(net["W1"], np.uint16)
    W3 = np.asarray(net["W3"], np.uint16)
    out = dict(net)
    if W1.shape[1] < 23:
        out["W1"] = np.concatenate([W1, np.zeros((W1.shape[0], 23 - W1.shape[1]), np.uint16)], axis=1)
    if 1 < W3.shape[0] < 8:
        k = W3.shape[0]
        out["W3"] = np.concatenate([W3, np.zeros((8 - k, W3.shape[1]), np.uint16)])
        out["b3"] = np.concatenate([np.asarray(net["b3"], np.float32), np.zeros(8 - k, np.float32)])
        if "log_std" in net:
            out["log_std"] = np.concatenate([np.asarray(net["log_std"], np.float32)[:k], np.zeros(8 - k, np.float32)])
    return out


def upload_mlp(net: dict, device="cuda") -> dict:
    """Copy an MLP parameter dict (bf16 bits W1, W2, W3; fp32 b1, b2, b3; log_std) into
    contiguous device buffers in the layout auv_mlp expects (12-input / 6-output networks of
    the paper task are padded, see pad_to_kernel_layout)."""
    net = pad_to_kernel_layout(net)
    w = np.concatenate([np.asarray(net[k], np.uint16).ravel() for k in ("W1", "W2", "W3")])
    b = np.concatenate([np.asarray(net[k], np.float32).ravel() for k in ("b1", "b2", "b3")])
    n_out = int(np.asarray(net["W3"]).shape[0])
    d = {"w": torch.from_numpy(w.view(np.int16).copy()).to(device),
         "b": torch.from_numpy(b).to(device),
         "log_std": torch.from_numpy(np.asarray(net.get("log_std", np.zeros(8)), np.float32)).to(device),
         "n_out": n_out}
    d["struct"] = A.make_mlp(d["w"], d["b"], d["log_std"], n_out)
    return d


class AuvEnv:
    def __init__(self, cfg: dict, vehicle: dict, alloc, device="cuda"):
        self.cfg = dict(cfg)
        self.n = n = int(cfg["n_envs"])
        self.device = device
        f32 = dict(dtype=torch.float32, device=device)
        self.state = torch.zeros(A.STATE_DIM, n, **f32)
        self.params = torch.zeros(A.PARAM_DIM, n, **f32)
        self.ep_step = torch.zeros(n, dtype=torch.int32, device=device)
        self.episode = torch.zeros(n, dtype=torch.int32, device=device)
        self.obs = torch.zeros(A.OBS_DIM, n, **f32)
        self.status = torch.zeros(2, dtype=torch.int32, device=device)   # failure counters (uint32)
        self._cfg = A.make_config(n, int(cfg["substeps"]), int(cfg["episode_len"]), cfg["dt_control"],
                                  int(cfg["seed"]), int(cfg["flags"]), int(cfg.get("env_offset", 0)))
        self._veh = A.make_vehicle(vehicle, alloc)
        self._bufs = A.make_env_buffers(self.state, self.params, self.ep_step, self.episode, self.obs, self.status)
        self.handle = A.auv_create(self._cfg, self._veh, self._bufs)

    def close(self):
        if getattr(self, "handle", None):
            A.auv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def global_step(self) -> int:
        return A.auv_get_global_step(self.handle)

    @global_step.setter
    def global_step(self, step: int):
        A.auv_set_global_step(self.handle, step)

    def set_task(self, task: dict):
        """Select the task (a dict for make_task, e.g. workloads.PAPER_TASK); before reset()."""
        self._task = A.make_task(task)
        A.auv_set_task(self.handle, self._task)

    def reset(self):
        A.auv_reset(self.handle)

    def step(self, mode=A.AUV_ACT_RANDOM, actions=None, want_stats=False, policy=None):
        """One control step (policy: an upload_mlp dict in the policy modes); returns
        (reward [N], done uint8 [N], stats [3] or None)."""
        reward = torch.empty(self.n, dtype=torch.float32, device=self.device)
        done = torch.empty(self.n, dtype=torch.uint8, device=self.device)
        stats = work = None
        if want_stats:
            stats = torch.empty(3, dtype=torch.float32, device=self.device)
            work = torch.empty(A.auv_stats_work_floats(self.n, 1), dtype=torch.float32, device=self.device)
        A.auv_step(self.handle, mode, actions, None if policy is None else policy["struct"], reward, done, stats, work)
        return reward, done, stats

    def get_status(self):
        """(non-finite state components, abandoned waits) since the last call; synchronises."""
        _, nf, ab = A.auv_get_status(self.handle)
        return nf, ab

    def rollout_buffers(self, T, record=("obs", "act", "reward", "done", "stats"), value=False):
        """Allocate the per-step output buffers named in `record`."""
        n, f32 = self.n, dict(dtype=torch.float32, device=self.device)
        shapes = {"obs": (A.OBS_DIM, T, n), "act": (A.ACT_DIM, T, n), "logp": (T, n), "value": (T, n),
                  "reward": (T, n), "done": (T, n), "last_value": (n,),
                  "traj_state": (A.STATE_DIM, T + 1, n), "stats": (3, T)}
        out = {k: torch.empty(shapes[k], **f32) for k in record}
        if "stats" in out:
            out["stats_work"] = torch.empty(A.auv_stats_work_floats(n, T), **f32)
        return out

    def rollout(self, T, mode, policy=None, value=None, bufs=None):
        """T control steps in one launch; bufs from rollout_buffers() (or None)."""
        bufs = bufs or {}
        rb = A.make_rollout_buffers(**bufs)
        A.auv_rollout(self.handle, T, mode, None if policy is None else policy["struct"],
                      None if value is None else value["struct"], rb)
        return bufs
