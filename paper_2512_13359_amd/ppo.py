"""PpoNet / PpoLearner: device buffers of the PPO update (packed fp32 parameters, Adam
moments, bf16 weight copies, gradients, workspace) and calls of auv_ppo_grad /
auv_ppo_adam through the C binding.  Memory management and argument marshalling only."""
from __future__ import annotations

import numpy as np
import torch

from . import _abi as A


class PpoNet:
    """One trainable MLP: theta packed W1 | W2 | W3 | b1 | b2 | b3 [| log_std], its Adam
    moments and gradient, and the bf16 copy of W1 | W2 | W3.  `mlp` is the auv_mlp view
    (bf16 weights, fp32 biases and log_std inside theta) that auv_rollout and auv_ppo_grad
    read."""

    def __init__(self, net: dict, device="cuda"):
        from .env import pad_to_kernel_layout
        self.n_actions = int(np.asarray(net["W3"]).shape[0])   # before padding (6 for the paper task)
        net = pad_to_kernel_layout(net)
        n_out = int(np.asarray(net["W3"]).shape[0])
        self.n_out = n_out
        self.nw = A.ppo_nw(n_out)
        bits = np.concatenate([np.asarray(net[k], np.uint16).ravel() for k in ("W1", "W2", "W3")])
        wvals = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
        parts = [wvals] + [np.asarray(net[k], np.float32).ravel() for k in ("b1", "b2", "b3")]
        if n_out == 8:
            parts.append(np.asarray(net["log_std"], np.float32).ravel())
        theta = np.concatenate(parts)
        assert theta.size == A.ppo_nparam(n_out)
        self.theta = torch.from_numpy(theta).to(device)
        self.adam_m = torch.zeros_like(self.theta)
        self.adam_v = torch.zeros_like(self.theta)
        self.grad = torch.zeros_like(self.theta)
        self.w_bf16 = torch.from_numpy(bits.view(np.int16).copy()).to(device)
        self.b = self.theta[self.nw:]
        self.log_std = self.theta[self.nw + 512 + n_out:] if n_out == 8 else None
        self.mlp = A.make_mlp(self.w_bf16, self.b, self.log_std, n_out)
        self.net = A.AuvPpoNet(A.ptr(self.theta), A.ptr(self.adam_m), A.ptr(self.adam_v), A.ptr(self.w_bf16), n_out)


class PpoLearner:
    """Policy and value networks with one Adam state; update(batch, idx) = auv_ppo_grad on
    the minibatch idx of the rollout buffer, then auv_ppo_adam."""

    def __init__(self, policy: dict, value: dict, device="cuda", **hp):
        self.pol = PpoNet(policy, device)
        self.val = PpoNet(value, device)
        hp.setdefault("n_actions", self.pol.n_actions)
        self.cfg = A.make_ppo_config(**hp)
        self.t = 0
        self.device = device
        self.stats = torch.zeros(8, dtype=torch.float32, device=device)
        self._work = None

    def work(self, B: int) -> torch.Tensor:
        n = A.auv_ppo_work_bytes(B)
        if self._work is None or self._work.numel() < n:
            self._work = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self._work

    @staticmethod
    def batch(obs, act, logp, adv, ret) -> A.AuvPpoBatch:
        """Rollout buffers as [23][M], [8][M] and [M] tensors (any [k][T][N] buffer viewed flat)."""
        M = int(logp.numel())
        return A.make_ppo_batch(obs, act, logp, adv, ret, M)

    def grad(self, batch: A.AuvPpoBatch, idx: torch.Tensor, stream=None) -> None:
        B = int(idx.numel())
        A.auv_ppo_grad(self.cfg, self.pol.mlp, self.val.mlp, batch, idx, B, self.pol.grad, self.val.grad,
                       self.stats, self.work(B), stream)

    def step(self, stream=None) -> None:
        self.t += 1
        A.auv_ppo_adam(self.cfg, self.t, self.pol.net, self.val.net, self.pol.grad, self.val.grad, self.stats,
                       stream)

    def update(self, batch: A.AuvPpoBatch, idx: torch.Tensor, stream=None) -> None:
        self.grad(batch, idx, stream)
        self.step(stream)
