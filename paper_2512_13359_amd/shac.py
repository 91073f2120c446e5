"""ShacLearner: SHAC on the paper task through the C binding.

Holds the policy and the value net as PpoNets (packed fp32 parameters, Adam moments, bf16
weight copy), the gradients, statistics and workspace buffers, and the window's recorded
observations, rewards and values.  Calls auv_shac_window (one window's actor loss and policy
gradient), auv_ppo_adam with the value net left out (the actor step), and for the critic
auv_mlp_forward (values of the window's observations), auv_gae (TD(lambda) targets) and
auv_ppo_fit_value (the value regression).  Memory management
and argument marshalling only."""
from __future__ import annotations

import torch

from . import _abi as A
from .ppo import PpoNet


class ShacLearner:
    """SHAC actor and critic of one AuvEnv running the paper task.

    window() runs h control steps with the policy in the loop, leaves the gradient of the
    window's actor objective in self.grad and its statistics in self.stats, and records the
    window's observations and rewards; step() applies one clipped Adam step to the policy;
    critic_update() fits the value net to the window's TD(lambda) targets."""

    def __init__(self, env, policy: dict, value: dict | None = None, h: int = 32, gamma: float = 0.99,
                 max_grad_norm: float = 1.0, lr: float = 2e-3, beta1: float = 0.7, beta2: float = 0.95,
                 critic_lr: float = 2e-3, lam: float = 0.95, device="cuda"):
        self.env = env
        self.pol = PpoNet(policy, device)
        self.val = PpoNet(value, device) if value is not None else None
        self.h = int(h)
        self.gamma = float(gamma)
        self.lam = float(lam)
        self.max_grad_norm = float(max_grad_norm)
        self.adam = A.make_ppo_config(lr=lr, beta1=beta1, beta2=beta2, max_grad_norm=max_grad_norm,
                                      n_actions=self.pol.n_actions)
        # value regression: L = (vf_coef / 2) mean (V - R)^2 with vf_coef 2, no gradient clipping
        self.critic_cfg = A.make_ppo_config(vf_coef=2.0, ent_coef=0.0, max_grad_norm=0.0, lr=critic_lr, beta1=beta1,
                                            beta2=beta2, normalize_adv=False)
        self.grad = torch.zeros(A.ppo_nparam(8), dtype=torch.float32, device=device)
        self.grad_v = torch.zeros(A.ppo_nparam(1), dtype=torch.float32, device=device)
        self.stats = torch.zeros(8, dtype=torch.float32, device=device)
        self.critic_stats = torch.zeros(8, dtype=torch.float32, device=device)
        n = int(env.state.shape[1])
        self.n = n
        self.work = torch.empty(A.auv_shac_work_bytes(n, self.h), dtype=torch.uint8, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.rec = {"obs": torch.zeros(A.OBS_DIM, self.h, n, **f32), "reward": torch.zeros(self.h, n, **f32),
                    "done": torch.zeros(self.h, n, **f32), "value_last": torch.zeros(n, **f32)}
        self.values = torch.zeros(self.h, n, **f32)
        self.adv = torch.zeros(self.h, n, **f32)
        self.ret = torch.zeros(self.h, n, **f32)
        self._no_done = torch.zeros(self.h, n, **f32)
        self._critic_work = None
        self._critic_shape = None
        self._idx_host = None
        self.t = 0
        self.t_critic = 0

    def window(self, mode: int = A.AUV_ACT_POLICY_SAMPLE, out: dict | None = None, grad: bool = True,
               stream=None) -> None:
        """One window; out: optional tensors keyed like auv_shac_buffers (actions, obs, act,
        reward, done, grad_act, value_last, grad_state0); observations, rewards and the final
        value are recorded for the critic unless out provides its own."""
        cfg = A.make_shac_config(self.h, mode, self.gamma, self.max_grad_norm)
        bufs = dict(self.rec)
        bufs.update(out or {})
        policy = self.pol.mlp if mode != A.AUV_ACT_EXTERNAL else None
        value = self.val.mlp if self.val is not None else None
        A.auv_shac_window(self.env.handle, cfg, policy, value, A.make_shac_buffers(**bufs),
                          self.grad if (grad and policy is not None) else None, self.stats, self.work, stream)
        self._last = bufs

    def step(self, stream=None) -> None:
        """One clipped Adam step of the policy on the last window's gradient."""
        self.t += 1
        A.auv_ppo_adam(self.adam, self.t, self.pol.net, None, self.grad, None, self.stats, stream)

    def targets(self, stream=None) -> None:
        """TD(lambda) targets of the last window's observations: values from the current value
        net, then R_t = A_t + V_t with A from generalised advantage estimation, bootstrapped on
        V(o(s_h)) before any reset (the window's end, also at an episode's time limit)."""
        b = self._last
        M = self.h * self.n
        A.auv_mlp_forward(self.val.mlp, M, b["obs"], self.values, stream)
        A.auv_gae(self.h, self.n, b["reward"], self.values, self._no_done, b["value_last"], self.gamma, self.lam,
                  self.adv, self.ret, stream)

    def critic_update(self, iterations: int = 16, batches: int = 4, seed: int = 0, stream=None) -> None:
        """Value regression on the last window (auv_ppo_fit_value): `iterations` passes, each
        over `batches` minibatches of a seeded shuffle of the window's h N samples (16-sample
        blocks), each a value-only gradient and Adam step of the value net."""
        self.targets(stream)
        M = self.h * self.n
        if A.auv_ppo_fit_work_bytes(M, batches) < 0:
            raise ValueError("too few samples for this many minibatches")
        if self._critic_work is None or self._critic_shape != (M, batches):
            self._critic_work = torch.empty(A.auv_ppo_fit_work_bytes(M, batches), dtype=torch.uint8,
                                            device=self.values.device)
            self._idx_host = torch.empty(2 * 16 * (M // 16), dtype=torch.int32, pin_memory=True)
            self._critic_shape = (M, batches)
        b = self._last
        batch = A.make_ppo_batch(b["obs"], b["obs"], self.values, self.adv, self.ret, M)
        A.auv_ppo_fit_value(self.critic_cfg, self.val.mlp, self.val.net, batch, iterations, batches, seed,
                            self.t_critic, self._idx_host, self.grad_v, self.critic_stats, self._critic_work, stream)
        self.t_critic += iterations * batches
