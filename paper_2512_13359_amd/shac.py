"""ShacLearner: the SHAC actor update on the paper task through the C binding.

Holds the policy as a PpoNet (packed fp32 parameters, Adam moments, bf16 weight copy), an
optional value net for the terminal estimate, the gradient, statistics and workspace
buffers, and calls auv_shac_window (one window's loss and policy gradient) and
auv_ppo_adam with the value net left out (the actor step).  Memory management and argument
marshalling only."""
from __future__ import annotations

import torch

from . import _abi as A
from .ppo import PpoNet


class ShacLearner:
    """SHAC actor of one AuvEnv running the paper task.  window() runs h control steps with
    the policy in the loop and leaves the gradient of the window's objective in self.grad
    and its statistics in self.stats; step() applies one clipped Adam step to the policy."""

    def __init__(self, env, policy: dict, value: dict | None = None, h: int = 32, gamma: float = 0.99,
                 max_grad_norm: float = 1.0, lr: float = 2e-3, beta1: float = 0.7, beta2: float = 0.95,
                 device="cuda"):
        self.env = env
        self.pol = PpoNet(policy, device)
        self.val = PpoNet(value, device) if value is not None else None
        self.h = int(h)
        self.gamma = float(gamma)
        self.max_grad_norm = float(max_grad_norm)
        self.adam = A.make_ppo_config(lr=lr, beta1=beta1, beta2=beta2, max_grad_norm=max_grad_norm,
                                      n_actions=self.pol.n_actions)
        self.grad = torch.zeros(A.ppo_nparam(8), dtype=torch.float32, device=device)
        self.stats = torch.zeros(8, dtype=torch.float32, device=device)
        n = int(env.state.shape[1])
        self.work = torch.empty(A.auv_shac_work_bytes(n, self.h), dtype=torch.uint8, device=device)
        self.t = 0

    def window(self, mode: int = A.AUV_ACT_POLICY_SAMPLE, out: dict | None = None, grad: bool = True,
               stream=None) -> None:
        """One window; out: optional tensors keyed like auv_shac_buffers (actions, obs, act,
        reward, done, grad_act, value_last, grad_state0)."""
        cfg = A.make_shac_config(self.h, mode, self.gamma, self.max_grad_norm)
        bufs = A.make_shac_buffers(**(out or {}))
        policy = self.pol.mlp if mode != A.AUV_ACT_EXTERNAL else None
        value = self.val.mlp if self.val is not None else None
        A.auv_shac_window(self.env.handle, cfg, policy, value, bufs, self.grad if (grad and policy is not None) else None,
                          self.stats, self.work, stream)

    def step(self, stream=None) -> None:
        self.t += 1
        A.auv_ppo_adam(self.adam, self.t, self.pol.net, None, self.grad, None, self.stats, stream)
