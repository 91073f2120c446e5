"""GPU parity of the SHAC window (auv_shac_window) against the float64 oracle
(oracle/shac.py), through the C interface.

Open loop (external actions): rewards, the terminal value, the action and initial-state
gradients through reward, observation, RK4 + Fossen and the terminal value, and the
environment update.  Closed loop (policy mean / sample): every policy parameter's gradient,
dL/dmu_t, the actions.  Episode end at the window's last step: terminal value before the
reset, the reset itself, and the refusal of a window that would cross an episode end.  At
the full 4096-environment, 32-step size: sampled environments against the oracle run on
those environments alone (each environment's window depends only on itself); every gradient
block of 32- and 64-step windows against the oracle at 256 and 33 environments.

Tolerances: the kernel carries the adjoint in fp32 against the oracle's fp64; where a
cotangent or activation sits within fp32 error of a bf16 rounding midpoint, the two sides
may round it to neighbouring bf16 values (2^-8 relative apart), which moves the products it
feeds by a fraction of that.  In closed loop such a flip in the forward also moves the
trajectory a little.  Gradient blocks are compared by their largest deviation relative to
the block's largest entry."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import mlp as omlp
from oracle import paper_task as P
from oracle import shac as S
from tests.gpu_util import announce, gpu_env, host, quat_aligned, rel_err, require_gpu

pytestmark = pytest.mark.gpu


def _nets():
    return W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12)


def _setup(n, seed=8, episode_len=512, moving=True):
    """A paper-task env on the GPU, optionally moved off its reset state (random poses,
    velocities and action averages), and the oracle's window start for the same values."""
    cfg = W.config("c6", n_envs=n, episode_len=episode_len)
    g = gpu_env(cfg)
    g.set_task(W.PAPER_TASK)
    g.reset()
    if moving:
        x0 = W.random_states(n, seed=seed)
        r = np.random.default_rng(seed)
        obs = host(g.obs).copy()
        obs[12:18] = r.uniform(-0.6, 0.6, (6, n)).astype(np.float32)
        g.state.copy_(torch.from_numpy(x0))
        g.obs.copy_(torch.from_numpy(obs))
    pr, st, ob = host(g.params), host(g.state), host(g.obs)
    start = dict(x=st.astype(np.float64), abar=ob[12:18].astype(np.float64), p_goal=pr[6:9].astype(np.float64),
                 q_goal=pr[9:13].astype(np.float64), gfac=pr[13].astype(np.float64), step=g.global_step,
                 env_ids=np.arange(n))
    return cfg, g, start


def _learner(g, h, gamma=0.97):
    from paper_2512_13359_amd import ShacLearner
    pol, val = _nets()
    return ShacLearner(g, pol, val, h=h, gamma=gamma, max_grad_norm=1.0)


def _dev(*shape):
    return torch.zeros(*shape, dtype=torch.float32, device="cuda")


def _unpad(grad: np.ndarray) -> dict:
    """Packed 23-256-256-8 gradient -> blocks of the 12-256-256-6 net, and its padding."""
    o = 0
    out = {}
    for k, n in (("W1", 256 * 23), ("W2", 256 * 256), ("W3", 8 * 256), ("b1", 256), ("b2", 256), ("b3", 8),
                 ("log_std", 8)):
        out[k] = grad[o:o + n]
        o += n
    assert o == grad.size
    W1, W3 = out["W1"].reshape(256, 23), out["W3"].reshape(8, 256)
    pad = np.concatenate([W1[:, 12:].ravel(), W3[6:].ravel(), out["b3"][6:], out["log_std"][6:]])
    return dict(W1=W1[:, :12], W2=out["W2"].reshape(256, 256), W3=W3[:6], b1=out["b1"], b2=out["b2"],
                b3=out["b3"][:6], log_std=out["log_std"][:6]), pad


def _block_err(got, want):
    return np.max(np.abs(np.asarray(got, np.float64) - want)) / max(np.max(np.abs(want)), 1e-30)


def test_shac_open_loop_window_matches_oracle():
    n, h, gamma = 101, 6, 0.97
    announce(f"SHAC external window n={n} h={h}")
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    cfg, g, start = _setup(n)
    _, val = _nets()
    ext = np.zeros((8, h, n), np.float32)
    ext[0:6] = np.random.default_rng(3).uniform(-1.2, 1.2, (6, h, n))
    L = _learner(g, h, gamma)
    out = dict(actions=torch.from_numpy(ext).cuda(), reward=_dev(h, n), done=_dev(h, n), grad_act=_dev(8, h, n),
               value_last=_dev(n), grad_state0=_dev(13, n), obs=_dev(23, h, n), act=_dev(8, h, n))
    L.window(mode=A.AUV_ACT_EXTERNAL, out=out)
    got = {k: host(v) for k, v in out.items()}
    stats = host(L.stats)
    want = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_EXTERNAL, value_net=val,
                         external=np.transpose(ext[0:6], (1, 0, 2)).astype(np.float64), quantize=True)
    assert rel_err(got["reward"], want["rewards"]).max() <= 1e-4
    assert np.all(got["done"] == 0)
    assert np.max(np.abs(got["value_last"] - want["v_last"])) <= 5e-3
    assert np.array_equal(got["act"][0:6], ext[0:6]) and np.all(got["act"][6:] == 0)
    assert np.all(got["obs"][12:] == 0)
    ga = np.transpose(got["grad_act"][0:6], (1, 0, 2))
    assert _block_err(ga, want["grad_act"]) <= 5e-3
    assert np.all(got["grad_act"][6:] == 0)
    assert np.all(ga[np.abs(np.transpose(ext[0:6], (1, 0, 2))) > 1.0] == 0)
    assert _block_err(got["grad_state0"], want["grad_state0"]) <= 5e-3
    assert abs(stats[0] - want["loss"]) <= 1e-3 * abs(want["loss"])
    assert np.isclose(stats[1], np.mean(want["J"] - gamma ** h * want["v_last"]), rtol=1e-4)
    assert stats[7] == 1.0
    # the environment after the window: final state, action average, counters
    x = host(g.state)
    x[3:7] = quat_aligned(x[3:7], want["x"][3:7])
    assert rel_err(x, want["x"]).max() <= 1e-4
    assert np.max(np.abs(host(g.obs)[12:18] - want["abar"])) <= 1e-5
    assert np.all(host(g.ep_step) == h) and g.global_step == h


@pytest.mark.parametrize("mode", [2, 3])
def test_shac_policy_gradient_matches_oracle(mode):
    """Closed loop with the policy (2: mean, 3: Gaussian sample): the packed policy gradient
    block by block (padding rows and columns exactly 0), dL/dmu_t and the actions."""
    n, h, gamma = 101, 5, 0.99
    announce(f"SHAC policy window mode={mode} n={n} h={h}")
    require_gpu()
    cfg, g, start = _setup(n, seed=9)
    pol, val = _nets()
    L = _learner(g, h, gamma)
    out = dict(grad_act=_dev(8, h, n), act=_dev(8, h, n), reward=_dev(h, n), obs=_dev(23, h, n))
    L.window(mode=mode, out=out)
    got = {k: host(v) for k, v in out.items()}
    blocks, pad = _unpad(host(L.grad))
    want = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, mode, policy_net=pol, value_net=val,
                         quantize=True)
    assert np.all(pad == 0)
    # every action is a valid bf16-MLP output (plus the oracle's noise) for the observation it was taken on
    mu = got["act"][0:6].astype(np.float64)
    if mode == 3:
        sig = np.exp(np.asarray(pol["log_std"], np.float32)[:6].astype(np.float64))[:, None, None]
        mu = mu - sig * np.transpose(np.stack([S.noise(cfg["seed"], np.arange(n), t) for t in range(h)]), (1, 0, 2))
    err = omlp.nearest_valid_error(mu.reshape(6, -1), got["obs"][0:12].reshape(12, -1).astype(np.float64), pol, 1e-6)
    assert err.max() <= 2e-3
    assert np.max(np.abs(np.transpose(got["act"][0:6], (1, 0, 2)) - want["acts"])) <= 1e-2
    assert rel_err(got["reward"], want["rewards"]).max() <= 1e-3
    ga = np.transpose(got["grad_act"][0:6], (1, 0, 2))
    assert _block_err(ga, want["grad_act"]) <= 2e-2
    errs = {k: _block_err(blocks[k], want["grad_policy"][k]) for k in blocks if k != "log_std" or mode == 3}
    announce(f"  block errors {errs}")
    for k, e in errs.items():
        assert e <= 5e-3, (k, e)
    if mode == 2:
        assert np.all(blocks["log_std"] == 0)
    stats = host(L.stats)
    assert abs(stats[0] - want["loss"]) <= 1e-3 * abs(want["loss"])
    gn = np.sqrt(sum(float(np.sum(want["grad_policy"][k] ** 2)) for k in want["grad_policy"]))
    assert abs(np.sqrt(stats[5]) - gn) <= 1e-2 * gn
    assert np.isclose(stats[7], min(1.0, 1.0 / (np.sqrt(stats[5]) + 1e-6)), rtol=1e-6)


@pytest.mark.parametrize("n,h", [(1, 1), (17, 2), (16, 3)])
def test_shac_small_and_ragged(n, h):
    """One environment and a one-step window (15 idle slots of the workgroup), a batch one
    environment past a workgroup (a second group with one live slot), and exactly one group:
    sampled-policy windows against the oracle, with the same tolerances as the larger test."""
    gamma = 0.99
    announce(f"SHAC small window n={n} h={h}")
    require_gpu()
    cfg, g, start = _setup(n, seed=31 + n)
    pol, val = _nets()
    L = _learner(g, h, gamma)
    out = dict(grad_act=_dev(8, h, n), reward=_dev(h, n))
    L.window(mode=3, out=out)
    want = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, 3, policy_net=pol, value_net=val,
                         quantize=True)
    assert rel_err(host(out["reward"]), want["rewards"]).max() <= 1e-3
    ga = np.transpose(host(out["grad_act"])[0:6], (1, 0, 2))
    assert _block_err(ga, want["grad_act"]) <= 2e-2
    blocks, pad = _unpad(host(L.grad))
    assert np.all(pad == 0)
    for k in blocks:
        assert _block_err(blocks[k], want["grad_policy"][k]) <= 5e-3, k
    assert abs(host(L.stats)[0] - want["loss"]) <= 1e-3 * abs(want["loss"])


def test_shac_window_ends_episode_then_resets():
    """8-step episodes, 4-step windows: the second window ends the episode at its last step;
    its terminal value is taken before the reset, then every env starts episode 1 as the
    oracle's reset draws say; a 5-step window at step 4 of 8 is refused."""
    n, h = 70, 4
    announce(f"SHAC episode end n={n} h={h}")
    require_gpu()
    from paper_2512_13359_amd import AuvError
    from paper_2512_13359_amd import _abi as A
    cfg, g, start = _setup(n, seed=10, episode_len=8)
    pol, val = _nets()
    L = _learner(g, h, 0.99)
    L.window(mode=A.AUV_ACT_POLICY_MEAN, grad=False)
    mid = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_MEAN, policy_net=pol,
                        value_net=val, quantize=True)
    out = dict(done=_dev(h, n), value_last=_dev(n), reward=_dev(h, n))
    L.window(mode=A.AUV_ACT_POLICY_MEAN, out=out)
    got = {k: host(v) for k, v in out.items()}
    start2 = dict(start, x=mid["x"], abar=mid["abar"], step=h)
    end = S.window_grad(start2, cfg, W.VEHICLE, W.PAPER_TASK, h, 0.99, S.MODE_POLICY_MEAN, policy_net=pol,
                        value_net=val, quantize=True)
    assert np.array_equal(got["done"][h - 1], np.ones(n, np.float32)) and np.all(got["done"][:h - 1] == 0)
    assert np.max(np.abs(got["value_last"] - end["v_last"])) <= 5e-3
    assert rel_err(got["reward"], end["rewards"]).max() <= 1e-3
    # the reset: episode 1 draws of the oracle
    o = P.PaperEnv(cfg, W.VEHICLE, W.PAPER_TASK)
    o.reset()
    o.episode[:] = 1
    o._draw(np.arange(n))
    pr = host(g.params)
    assert np.array_equal(pr[6:9], o.p_goal.astype(np.float32)) and np.array_equal(pr[13], o.gfac.astype(np.float32))
    assert np.max(np.abs(pr[9:13] - o.q_goal)) <= 1e-6
    want_x = np.zeros((13, n), np.float32)
    want_x[3] = 1
    assert np.array_equal(host(g.state), want_x)
    ob = host(g.obs)
    assert np.all(ob[12:18] == 0) and np.max(np.abs(ob[0:3] - o.p_goal)) <= 1e-6
    assert np.all(host(g.ep_step) == 0) and np.all(host(g.episode) == 1) and g.global_step == 2 * h
    # the next episode: a window of 5 from step 4 of 8 would cross its end
    L.window(mode=A.AUV_ACT_POLICY_MEAN, grad=False)
    L5 = _learner(g, 5)
    with pytest.raises(AuvError):
        L5.window(mode=A.AUV_ACT_POLICY_MEAN)


def test_shac_rejects_invalid_use():
    require_gpu()
    from paper_2512_13359_amd import AuvError, ShacLearner
    from paper_2512_13359_amd import _abi as A
    pol, val = _nets()
    g = gpu_env(W.config("c2", n_envs=64))          # workload task
    g.reset()
    with pytest.raises(AuvError):
        ShacLearner(g, pol, val, h=4).window()
    gs = gpu_env(W.config("c6", n_envs=64, flags=W.FLAG_STAGGER))
    gs.set_task(W.PAPER_TASK)
    gs.reset()
    with pytest.raises(AuvError):
        ShacLearner(gs, pol, val, h=4).window()
    _, g6, _ = _setup(64)
    L = ShacLearner(g6, pol, val, h=4)
    cfg = A.make_shac_config(4, A.AUV_ACT_EXTERNAL, 0.99, 1.0)
    acts = _dev(8, 4, 64)
    with pytest.raises(AuvError):   # no policy gradient in external mode
        A.auv_shac_window(g6.handle, cfg, None, L.val.mlp, A.make_shac_buffers(actions=acts), L.grad, L.stats, L.work)
    with pytest.raises(AuvError):   # external mode needs actions
        A.auv_shac_window(g6.handle, cfg, None, None, None, None, L.stats, L.work)
    bad = A.make_shac_config(4, A.AUV_ACT_POLICY_MEAN, 1.5, 1.0)
    with pytest.raises(AuvError):
        A.auv_shac_window(g6.handle, bad, L.pol.mlp, None, None, L.grad, L.stats, L.work)
    assert A.auv_shac_work_bytes(64, 65) == -1 and A.auv_shac_work_bytes(0, 8) == -1
    assert g6.global_step == 0


def test_shac_is_deterministic():
    n, h = 130, 3
    require_gpu()
    grads = []
    for _ in range(2):
        _, g, _ = _setup(n, seed=12)
        L = _learner(g, h)
        L.window()
        grads.append(host(L.grad).copy())
    assert np.array_equal(grads[0], grads[1])


def _states_from_obs(obs, p_goal, q_goal):
    """States [13, ...] behind paper-task observations [12, ...]: p = p_goal - R dp_b, q = q_goal
    (x) q_err^-1 with q_err = exp(rotation vector / 2), v and omega as observed (scipy's
    rotations; the sign of q is immaterial to the dynamics' outputs)."""
    from scipy.spatial.transform import Rotation
    shp = obs.shape[1:]
    o = obs.reshape(12, -1).astype(np.float64)
    m = o.shape[1]
    pg = np.broadcast_to(p_goal[:, None, :], (3,) + shp).reshape(3, m) if len(shp) == 2 else p_goal
    qg = np.broadcast_to(q_goal[:, None, :], (4,) + shp).reshape(4, m) if len(shp) == 2 else q_goal
    Rg = Rotation.from_quat(np.stack([qg[1], qg[2], qg[3], qg[0]], axis=1))
    R = Rg * Rotation.from_rotvec(o[3:6].T).inv()
    qx = R.as_quat()
    x = np.zeros((13, m))
    x[0:3] = pg - R.apply(o[0:3].T).T
    x[3:7] = np.stack([qx[:, 3], qx[:, 0], qx[:, 1], qx[:, 2]])
    x[7:13] = o[6:12]
    return x.reshape((13,) + shp)


@pytest.mark.parametrize("n,h", [(256, 32), (33, 64)])
def test_shac_long_window_matches_oracle(n, h):
    """Windows of the benchmark's length (32 steps, at 256 environments) and of the longest
    allowed (64 steps): every block of the policy gradient, dL/dmu_t, the rewards, the loss and
    the gradient norm against the oracle (sample mode).  These windows run the checkpoint ring
    of the forward sweep and the reverse sweep over every stored substep.  Over this many
    closed-loop steps bf16 rounding flips let the GPU's and the oracle's trajectories drift
    apart (both correct), so the oracle is teacher-forced onto the GPU's trajectory: its states
    rebuilt from the recorded observations (and the final state buffer), its actions the
    recorded ones; the gradient is then the objective's along that trajectory."""
    gamma = W.SHAC["gamma"]
    announce(f"SHAC long window n={n} h={h}")
    require_gpu()
    cfg, g, start = _setup(n, seed=40 + h)
    pol, val = _nets()
    L = _learner(g, h, gamma)
    out = dict(grad_act=_dev(8, h, n), reward=_dev(h, n), obs=_dev(23, h, n), act=_dev(8, h, n))
    L.window(mode=3, out=out)
    got = {k: host(v) for k, v in out.items()}
    xs = np.concatenate([_states_from_obs(got["obs"][0:12, 1:], start["p_goal"], start["q_goal"]),
                         host(g.state).astype(np.float64)[:, None]], axis=1)           # [13, h, n]
    forced = dict(x=np.transpose(xs, (1, 0, 2)), a=np.transpose(got["act"][0:6], (1, 0, 2)).astype(np.float64))
    want = S.window_grad(start, cfg, W.VEHICLE, W.PAPER_TASK, h, gamma, 3, policy_net=pol, value_net=val,
                         quantize=True, forced=forced)
    rerr = rel_err(got["reward"], want["rewards"]).max()
    ga = np.transpose(got["grad_act"][0:6], (1, 0, 2))
    ga_err = _block_err(ga, want["grad_act"])
    blocks, pad = _unpad(host(L.grad))
    assert np.all(pad == 0)
    errs = {k: _block_err(blocks[k], want["grad_policy"][k]) for k in blocks}
    announce(f"  reward {rerr:.2e}, dL/dmu {ga_err:.2e}, block errors {errs}")
    assert rerr <= 1e-4
    assert ga_err <= 2e-2
    for k, e in errs.items():
        assert e <= 5e-3, (k, e)
    stats = host(L.stats)
    assert abs(stats[0] - want["loss"]) <= 1e-3 * abs(want["loss"])
    gn = np.sqrt(sum(float(np.sum(want["grad_policy"][k] ** 2)) for k in want["grad_policy"]))
    assert abs(np.sqrt(stats[5]) - gn) <= 1e-2 * gn


def test_shac_full_size_sampled_envs():
    """4096 environments x 32 steps (sample mode): 24 sampled environments against the
    oracle run on those environments alone (every gradient block at this window length is
    compared with the oracle at 256 environments, test_shac_long_window_matches_oracle)."""
    n, h, gamma = W.SHAC["n_envs"], W.SHAC["h"], W.SHAC["gamma"]
    announce(f"SHAC full size n={n} h={h}")
    require_gpu()
    cfg, g, start = _setup(n, seed=13)
    pol, val = _nets()
    L = _learner(g, h, gamma)
    out = dict(grad_act=_dev(8, h, n), reward=_dev(h, n))
    L.window(mode=3, out=out)
    got = {k: host(v) for k, v in out.items()}
    blocks, pad = _unpad(host(L.grad))
    assert np.all(pad == 0) and all(np.all(np.isfinite(v)) for v in blocks.values())
    stats = host(L.stats)
    assert np.all(np.isfinite(stats)) and 0.0 < stats[7] <= 1.0
    ga = np.transpose(got["grad_act"][0:6], (1, 0, 2)).astype(np.float64)
    # sampled environments: the oracle on those columns alone (the loss scale 1/(N h) is the full N's)
    idx = np.unique(np.concatenate([np.linspace(0, n - 1, 22).astype(int), [1, n - 2]]))
    sub = {k: (v[..., idx] if isinstance(v, np.ndarray) and v.shape[-1] == n else v) for k, v in start.items()}
    sub["env_ids"] = idx
    want = S.window_grad(sub, dict(cfg, n_envs=idx.size), W.VEHICLE, W.PAPER_TASK, h, gamma, S.MODE_POLICY_SAMPLE,
                         policy_net=pol, value_net=val, quantize=True)
    scale = idx.size / n
    assert rel_err(got["reward"][:, idx], want["rewards"]).max() <= 2e-3
    assert _block_err(ga[:, :, idx], want["grad_act"] * scale) <= 5e-2


def test_shac_critic_regression():
    """The critic's value-only gradient equals the value part of a full PPO gradient call on
    the same minibatch (same kernels, bit for bit); TD(lambda) targets are consistent
    (R = A + V); fitting the window's targets lowers the value loss."""
    n, h = 130, 6
    announce(f"SHAC critic n={n} h={h}")
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    _, g, _ = _setup(n, seed=14)
    L = _learner(g, h)
    L.window()
    L.targets()
    assert float(torch.max(torch.abs(L.ret - L.values - L.adv))) <= 1e-6 * float(torch.max(torch.abs(L.ret)))
    M = h * n
    b = L._last
    batch = A.make_ppo_batch(b["obs"], b["obs"], L.values, L.adv, L.ret, M)
    idx = torch.arange(0, 256, dtype=torch.int32, device="cuda")
    work = torch.empty(A.auv_ppo_work_bytes(256), dtype=torch.uint8, device="cuda")
    gv1, st1 = torch.zeros_like(L.grad_v), torch.zeros(8, device="cuda")
    A.auv_ppo_grad(L.critic_cfg, None, L.val.mlp, batch, idx, 256, None, gv1, st1, work)
    gp, gv2, st2 = torch.zeros_like(L.grad), torch.zeros_like(L.grad_v), torch.zeros(8, device="cuda")
    pbatch = A.make_ppo_batch(b["obs"], torch.zeros(8, M, device="cuda"), torch.zeros(M, device="cuda"), L.adv, L.ret, M)
    A.auv_ppo_grad(L.critic_cfg, L.pol.mlp, L.val.mlp, pbatch, idx, 256, gp, gv2, st2, work)
    assert torch.equal(gv1, gv2)
    assert host(st1)[1] == host(st2)[1] and host(st1)[0] == 0.0
    before = float(torch.mean((L.values - L.ret) ** 2))
    L.critic_update(iterations=8, batches=4)
    A.auv_mlp_forward(L.val.mlp, M, b["obs"], L.values)
    after = float(torch.mean((L.values - L.ret) ** 2))
    assert after < 0.8 * before, (before, after)


def _splitmix64(state):
    """SplitMix64 (Steele, Lea and Flood 2014): (next state, output)."""
    m = (1 << 64) - 1
    state = (state + 0x9E3779B97F4A7C15) & m
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return state, z ^ (z >> 31)


def _fit_indices(M, iterations, seed):
    """The passes' sample orders of auv_ppo_fit_value, restated: Fisher-Yates over the M // 16
    blocks (j uniform in [0, i] by the multiply-shift of the draw's high 32 bits)."""
    nb, st, out = M // 16, seed, []
    for _ in range(iterations):
        perm = list(range(nb))
        for i in range(nb - 1, 0, -1):
            st, r = _splitmix64(st)
            j = ((r >> 32) * (i + 1)) >> 32
            perm[i], perm[j] = perm[j], perm[i]
        out.append((np.array(perm, np.int64)[:, None] * 16 + np.arange(16)).ravel().astype(np.int32))
    return out


def test_ppo_fit_value_back_to_back_calls():
    """Two auv_ppo_fit_value calls issued back to back on one workspace, with no
    synchronisation between them, equal the same steps issued one call at a time (bit for
    bit): the second call's first index upload (slot 0) waits for the first call's last pass,
    which read slot 0 too."""
    n, h, iterations, batches = 130, 6, 3, 4
    announce(f"PPO fit value back to back n={n} h={h} iterations={iterations}")
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    from paper_2512_13359_amd.ppo import PpoNet
    _, g, _ = _setup(n, seed=15)
    L = _learner(g, h)
    L.window()
    L.targets()
    M = h * n
    b = L._last
    batch = A.make_ppo_batch(b["obs"], b["obs"], L.values, L.adv, L.ret, M)
    val = W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12)
    net1, net2 = PpoNet(val, "cuda"), PpoNet(val, "cuda")
    work = torch.empty(A.auv_ppo_fit_work_bytes(M, batches), dtype=torch.uint8, device="cuda")
    stage = torch.empty(2 * 16 * (M // 16), dtype=torch.int32, pin_memory=True)
    g1, s1 = torch.zeros(A.ppo_nparam(1), device="cuda"), torch.zeros(8, device="cuda")
    seeds = (777, 778)
    A.auv_ppo_fit_value(L.critic_cfg, net1.mlp, net1.net, batch, iterations, batches, seeds[0], 0, stage, g1, s1, work)
    A.auv_ppo_fit_value(L.critic_cfg, net1.mlp, net1.net, batch, iterations, batches, seeds[1], iterations * batches,
                        stage, g1, s1, work)
    B = (M // 16 // batches) * 16
    g2, s2 = torch.zeros_like(g1), torch.zeros_like(s1)
    w2 = torch.empty(A.auv_ppo_work_bytes(B), dtype=torch.uint8, device="cuda")
    t = 0
    for seed in seeds:
        for order in _fit_indices(M, iterations, seed):
            idx = torch.from_numpy(order).cuda()
            for j in range(batches):
                A.auv_ppo_grad(L.critic_cfg, None, net2.mlp, batch, idx[j * B:(j + 1) * B], B, None, g2, s2, w2)
                t += 1
                A.auv_ppo_adam(L.critic_cfg, t, None, net2.net, None, g2, s2)
    torch.cuda.synchronize()
    d = (net1.theta - net2.theta).abs()
    assert torch.equal(net1.theta, net2.theta), (float(d.max()), int((d > 0).sum()), int(d.numel()))
    assert torch.equal(g1, g2) and torch.equal(s1, s2)


def test_ppo_fit_value_large_minibatches_match_stepwise_calls():
    """Minibatches of 131072 samples (4096 steps of 32: the value-only weight gradient in its
    128-row form with q(h1) recomputed, 64 chunks, then the reduce with the fused Adam step):
    auv_ppo_fit_value equals the same gradient + Adam calls issued one at a time, bit for bit.
    Synthetic seeded batch of 262144 samples, two passes of two minibatches."""
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    from paper_2512_13359_amd.ppo import PpoNet
    M, iterations, batches, seed = 262144, 2, 2, 777
    announce(f"PPO fit value large minibatches M={M} batches={batches} iterations={iterations}")
    rng = np.random.default_rng(31)
    obs = torch.from_numpy(rng.standard_normal((23, M)).astype(np.float32)).cuda()
    val_old = torch.from_numpy(rng.standard_normal(M).astype(np.float32)).cuda()
    adv = torch.from_numpy(rng.standard_normal(M).astype(np.float32)).cuda()
    ret = torch.from_numpy(rng.standard_normal(M).astype(np.float32)).cuda()
    batch = A.make_ppo_batch(obs, obs, val_old, adv, ret, M)
    cfg = A.make_ppo_config(vf_coef=2.0, ent_coef=0.0, max_grad_norm=0.0, lr=1e-3, normalize_adv=False)
    val = W.mlp_weights(1, W.VALUE_SEED)
    net1, net2 = PpoNet(val, "cuda"), PpoNet(val, "cuda")
    work = torch.empty(A.auv_ppo_fit_work_bytes(M, batches), dtype=torch.uint8, device="cuda")
    stage = torch.empty(2 * M, dtype=torch.int32, pin_memory=True)
    g1, s1 = torch.zeros(A.ppo_nparam(1), device="cuda"), torch.zeros(8, device="cuda")
    A.auv_ppo_fit_value(cfg, net1.mlp, net1.net, batch, iterations, batches, seed, 0, stage, g1, s1, work)
    B = M // batches
    g2, s2 = torch.zeros_like(g1), torch.zeros_like(s1)
    w2 = torch.empty(A.auv_ppo_work_bytes(B), dtype=torch.uint8, device="cuda")
    t = 0
    for order in _fit_indices(M, iterations, seed):
        idx = torch.from_numpy(order).cuda()
        for j in range(batches):
            A.auv_ppo_grad(cfg, None, net2.mlp, batch, idx[j * B:(j + 1) * B], B, None, g2, s2, w2)
            t += 1
            A.auv_ppo_adam(cfg, t, None, net2.net, None, g2, s2)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(net1.theta).all())
    d = (net1.theta - net2.theta).abs()
    assert torch.equal(net1.theta, net2.theta), (float(d.max()), int((d > 0).sum()), int(d.numel()))
    assert torch.equal(net1.w_bf16, net2.w_bf16)
    assert torch.equal(g1, g2) and torch.equal(s1, s2)


def test_ppo_fit_value_matches_stepwise_calls():
    """auv_ppo_fit_value equals the same value-only gradient + Adam steps issued one call at
    a time with the shuffles restated in Python (bit for bit; the index uploads reuse each of
    their two slots), and rejects bad sizes."""
    n, h, iterations, batches, seed = 130, 6, 6, 4, 12345   # six passes: each index slot reused twice
    announce(f"PPO fit value n={n} h={h} iterations={iterations}")
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    from paper_2512_13359_amd.ppo import PpoNet
    _, g, _ = _setup(n, seed=14)
    L = _learner(g, h)
    L.window()
    L.targets()
    M = h * n
    b = L._last
    batch = A.make_ppo_batch(b["obs"], b["obs"], L.values, L.adv, L.ret, M)
    val = W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12)
    net1, net2 = PpoNet(val, "cuda"), PpoNet(val, "cuda")
    work = torch.empty(A.auv_ppo_fit_work_bytes(M, batches), dtype=torch.uint8, device="cuda")
    stage = torch.empty(2 * 16 * (M // 16), dtype=torch.int32, pin_memory=True)
    g1, s1 = torch.zeros(A.ppo_nparam(1), device="cuda"), torch.zeros(8, device="cuda")
    A.auv_ppo_fit_value(L.critic_cfg, net1.mlp, net1.net, batch, iterations, batches, seed, 5, stage, g1, s1, work)
    B = (M // 16 // batches) * 16
    g2, s2 = torch.zeros_like(g1), torch.zeros_like(s1)
    w2 = torch.empty(A.auv_ppo_work_bytes(B), dtype=torch.uint8, device="cuda")
    t = 5
    for order in _fit_indices(M, iterations, seed):
        idx = torch.from_numpy(order).cuda()
        for j in range(batches):
            A.auv_ppo_grad(L.critic_cfg, None, net2.mlp, batch, idx[j * B:(j + 1) * B], B, None, g2, s2, w2)
            t += 1
            A.auv_ppo_adam(L.critic_cfg, t, None, net2.net, None, g2, s2)
    torch.cuda.synchronize()
    d = (net1.theta - net2.theta).abs()
    assert torch.equal(net1.theta, net2.theta), (float(d.max()), int((d > 0).sum()), int(d.numel()))
    assert torch.equal(net1.w_bf16, net2.w_bf16)
    assert torch.equal(g1, g2) and torch.equal(s1, s2)
    assert A.auv_ppo_fit_work_bytes(15, 1) == -1 and A.auv_ppo_fit_work_bytes(64, 5) == -1
    with pytest.raises(A.AuvError):
        A.auv_ppo_fit_value(L.critic_cfg, net1.mlp, net1.net, batch, 0, batches, seed, 0, stage, g1, s1, work)


def test_shac_learns_the_paper_task():
    """End-to-end learning: SHAC on the paper task from the seeded networks at 512 envs, 160
    windows (ten 512-step episodes), each followed by the actor's Adam step and the critic's
    regression.  The reward gradient through the simulation improves the policy within the
    first few windows, and the episodes' mean step reward keeps improving after that."""
    require_gpu()
    announce("shac learns the paper task")
    from paper_2512_13359_amd import AuvEnv, ShacLearner
    cfg = W.config("c6", n_envs=512)
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    L = ShacLearner(env, W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.PAPER_VALUE_SEED, n_in=12),
                    h=W.SHAC["h"], gamma=W.SHAC["gamma"], max_grad_norm=W.SHAC["max_grad_norm"])
    r = []
    for k in range(160):
        L.window()
        r.append(float(L.rec["reward"].mean()))
        L.step()
        L.critic_update(iterations=16, batches=4, seed=k)
    r = np.array(r)
    ep = r.reshape(-1, cfg["episode_len"] // W.SHAC["h"]).mean(axis=1)
    print(f"    first windows {np.round(r[:4], 3)}, episode means {np.round(ep, 3)}")
    assert np.isfinite(r).all() and np.isfinite(host(L.stats)).all()
    assert r[0] < -4.0 and r[3] > 0.5 * r[0]
    assert ep[-1] > 0.5 * ep[0] and ep[-1] > ep[1] + 0.02
