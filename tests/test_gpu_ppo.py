"""GPU parity of the PPO update (auv_ppo_grad, auv_ppo_adam) against the fp64 oracle
(oracle/ppo.py with the bf16 quantisation points of the MFMA path), through the C
interface.

Inputs: seeded draws (workloads.ppo_draws) turned into actions and old log-probabilities
by the oracle's own policy evaluation; target ratios stay 0.03 away from the clip bounds so
that the GPU and the oracle take every clipping decision the same way.

Tolerance of the gradients.  The oracle's quantised gradient differs from the exact one by
about 1-2 units of 2^-8 of each tensor's scale (bf16 rounding of layer inputs and of the
back-propagated values; pinned in test_oracle_ppo).  The GPU computes the same quantised
quantity; it differs from the oracle only where its fp32 value before a bf16 rounding
falls on the other side of a rounding midpoint than the oracle's fp64 value, and by fp32
accumulation.  Those differences are a fraction of the quantisation effect itself, so each
tensor must agree to 2^-8 of its scale (max-abs) and 2^-9 in norm."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import ppo as oppo
from oracle.mlp import bf16_bits_to_f64, bf16_round
from tests.gpu_util import announce, host, require_gpu

pytestmark = pytest.mark.gpu

SHAPES = {8: (23, 256, 8, True), 1: (23, 256, 1, False)}


def _oracle_params(net: dict) -> dict:
    p = {k: bf16_bits_to_f64(net[k]) for k in ("W1", "W2", "W3")}
    for k in ("b1", "b2", "b3"):
        p[k] = np.asarray(net[k], np.float32).astype(np.float64)
    if "log_std" in net and p["W3"].shape[0] == 8:
        p["log_std"] = np.asarray(net["log_std"], np.float32).astype(np.float64)
    return p


def _buffer(M: int, seed: int, pol: dict):
    """Synthetic rollout buffer: act = mu + sigma eps and logp_old from the oracle policy."""
    d = W.ppo_draws(M, seed)
    mu, _ = oppo.mlp_forward_cache(d["obs"].astype(np.float64), pol, quantize=True)
    sig = np.exp(pol["log_std"])[:, None]
    act = (mu + sig * d["eps"]).astype(np.float32)
    logp = oppo.gaussian_logp(act.astype(np.float64), mu, pol["log_std"])
    logp_old = (logp - np.log(d["ratio"])).astype(np.float32)
    return dict(obs=d["obs"], act=act, logp=logp_old, adv=d["adv"], ret=d["ret"])


@pytest.fixture(scope="module")
def setup():
    require_gpu()
    from paper_2512_13359_amd import PpoLearner
    netp = W.mlp_weights(8, W.POLICY_SEED)
    netv = W.mlp_weights(1, W.VALUE_SEED)
    pol, val = _oracle_params(netp), _oracle_params(netv)
    M = 6000
    buf = _buffer(M, 11, pol)
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in buf.items()}
    return netp, netv, pol, val, buf, dev, M, PpoLearner


def _check_grads(got: np.ndarray, want: np.ndarray, n_out: int, what: str):
    g, w = oppo.unpack(got, *SHAPES[n_out]), oppo.unpack(want, *SHAPES[n_out])
    for k in g:
        scale = np.abs(w[k]).max()
        err = np.abs(g[k] - w[k]).max()
        nerr = np.linalg.norm(g[k] - w[k]) / max(np.linalg.norm(w[k]), 1e-30)
        print(f"    {what} {k}: max-abs {err / scale / 2 ** -8:.3f} x 2^-8 of scale, norm {nerr / 2 ** -9:.3f} x 2^-9")
        assert err <= 2.0 ** -8 * scale, (what, k, err / scale)
        assert nerr <= 2.0 ** -9, (what, k, nerr)


@pytest.mark.parametrize("B,normalize", [(1000, True), (1000, False), (64, True), (17, True), (1, False)])
def test_ppo_grad_parity(setup, B, normalize):
    netp, netv, pol, val, buf, dev, M, PpoLearner = setup
    announce(f"ppo grad parity B={B} normalize={normalize}")
    L = PpoLearner(netp, netv, normalize_adv=normalize, ent_coef=0.01)
    idx = W.ppo_minibatch_idx(M, B, seed=B)
    batch = L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"])
    L.grad(batch, torch.from_numpy(idx).cuda())
    st = host(L.stats)
    cols = idx.astype(np.int64)
    want = oppo.ppo_loss_grad(buf["obs"][:, cols], buf["act"][:, cols], buf["logp"][cols], buf["adv"][cols],
                              buf["ret"][cols], pol, val, dict(normalize_adv=normalize, ent_coef=0.01),
                              quantize=True)
    _check_grads(host(L.pol.grad), want["grad_pol"], 8, "policy")
    _check_grads(host(L.val.grad), want["grad_val"], 1, "value")
    assert abs(st[0] - want["pg_loss"]) <= 2e-3 * max(1.0, abs(want["pg_loss"]))
    assert abs(st[1] - want["v_loss"]) <= 2e-3 * max(1.0, abs(want["v_loss"]))
    assert abs(st[2] - want["entropy"]) <= 1e-5 * abs(want["entropy"])
    assert abs(st[3] - want["approx_kl"]) <= 2e-3
    assert st[4] == pytest.approx(want["clip_frac"], abs=0.5 / B)
    gp, gv = host(L.pol.grad).astype(np.float64), host(L.val.grad).astype(np.float64)
    assert st[5] == pytest.approx(np.sum(gp * gp), rel=1e-4)
    assert st[6] == pytest.approx(np.sum(gv * gv), rel=1e-4)
    assert st[7] == pytest.approx(oppo.clip_scale([gp, gv], 0.5), rel=1e-6)


def test_ppo_grad_deterministic_and_block_independent(setup):
    """Same inputs, same bits; and the result does not depend on how the minibatch is
    ordered within its 16-sample tiles beyond fp32 summation order (permuted tiles give
    the same gradient to fp32 rounding)."""
    netp, netv, pol, val, buf, dev, M, PpoLearner = setup
    announce("ppo grad determinism")
    L = PpoLearner(netp, netv)
    idx = W.ppo_minibatch_idx(M, 4096, seed=3)
    batch = L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"])
    L.grad(batch, torch.from_numpy(idx).cuda())
    a = host(L.pol.grad).copy(), host(L.val.grad).copy(), host(L.stats).copy()
    L.grad(batch, torch.from_numpy(idx).cuda())
    b = host(L.pol.grad), host(L.val.grad), host(L.stats)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    perm = np.random.default_rng(0).permutation(idx.size // 16)
    idx2 = idx.reshape(-1, 16)[perm].ravel()
    L.grad(batch, torch.from_numpy(np.ascontiguousarray(idx2)).cuda())
    c = host(L.pol.grad)
    assert np.max(np.abs(c - a[0])) <= 1e-5 * np.abs(a[0]).max()


def test_ppo_adam_parity_two_steps(setup):
    """Two Adam steps from seeded parameters and moments on seeded gradients with a
    clipping factor: theta, m, v to fp32 rounding of the fp64 update; the bf16 copy is the
    round-to-nearest-even of the GPU's own fp32 theta, bit for bit."""
    netp, netv, pol, val, buf, dev, M, PpoLearner = setup
    announce("ppo adam parity")
    from paper_2512_13359_amd import _abi as A
    L = PpoLearner(netp, netv, lr=1e-3)
    r = np.random.default_rng(5)
    # the device receives the hyperparameters as fp32: the oracle takes those values exactly
    hp = {k: float(np.float32(v)) for k, v in dict(lr=1e-3, beta1=0.9, beta2=0.999, adam_eps=1e-8).items()}
    ref = {}
    for net in (L.pol, L.val):
        P = A.ppo_nparam(net.n_out)
        th = host(net.theta).astype(np.float64)
        m0 = (r.standard_normal(P) * 1e-3).astype(np.float32)
        v0 = (r.random(P) * 1e-6).astype(np.float32)
        net.adam_m.copy_(torch.from_numpy(m0))
        net.adam_v.copy_(torch.from_numpy(v0))
        ref[net.n_out] = [th, m0.astype(np.float64), v0.astype(np.float64)]
    stats = torch.zeros(8, device="cuda")
    scales = {}
    for t, scale in ((1, 0.37), (2, 1.0)):
        stats[7] = scale
        L.stats.copy_(stats)
        for net in (L.pol, L.val):
            g = (r.standard_normal(net.theta.numel()) * 10.0 ** r.uniform(-5, -1, net.theta.numel())).astype(np.float32)
            net.grad.copy_(torch.from_numpy(g))
            th, m, v = ref[net.n_out]
            gs = np.float32(scale) * g.astype(np.float64)
            # sums of the magnitudes of every term a moment has accumulated (the fp32 rounding
            # of each step is relative to its terms and carries into the next step)
            sm0, sv0 = scales.get(net.n_out, (np.abs(m), v))
            scales[net.n_out] = (hp["beta1"] * sm0 + (1 - hp["beta1"]) * np.abs(gs),
                                 hp["beta2"] * sv0 + (1 - hp["beta2"]) * gs * gs)
            ref[net.n_out] = list(oppo.adam_step(th, g.astype(np.float64), m, v, t, hp, scale=np.float32(scale)))
        L.t = t - 1
        L.step()
        for net in (L.pol, L.val):
            th, m, v = ref[net.n_out]
            gt, gm, gv = host(net.theta), host(net.adam_m), host(net.adam_v)
            sm, sv = scales[net.n_out]
            rm = np.abs(gm - m) / sm
            rv = np.abs(gv - v) / (sv + 1e-30)
            rt = np.abs(gt - th) / (2e-7 * np.abs(th) + 1e-3 * hp["lr"])
            k = int(np.argmax(rm))
            print(f"    t={t} n_out={net.n_out}: m {rm.max():.3g} (at {k}: got {gm[k]!r} want {m[k]!r} scale {sm[k]!r}), "
                  f"v {rv.max():.3g}, theta {rt.max():.3g}")
            assert rm.max() <= 4e-7 and rv.max() <= 4e-7 and rt.max() <= 1.0
            bits = host(net.w_bf16).view(np.uint16)
            want_bits = bf16_round(gt[:net.nw].astype(np.float64)).astype(np.float32).view(np.uint32) >> 16
            assert np.array_equal(bits, want_bits.astype(np.uint16))


def test_ppo_invalid_arguments(setup):
    netp, netv, pol, val, buf, dev, M, PpoLearner = setup
    from paper_2512_13359_amd import AuvError, _abi as A
    L = PpoLearner(netp, netv)
    batch = L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"])
    idx = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(AuvError):
        A.auv_ppo_grad(L.cfg, L.pol.mlp, L.val.mlp, batch, idx, 0, L.pol.grad, L.val.grad, L.stats, L.work(16))
    with pytest.raises(AuvError):   # networks swapped: wrong n_out
        A.auv_ppo_grad(L.cfg, L.val.mlp, L.pol.mlp, batch, idx, 16, L.pol.grad, L.val.grad, L.stats, L.work(16))
    with pytest.raises(AuvError):
        A.auv_ppo_adam(L.cfg, 0, L.pol.net, L.val.net, L.pol.grad, L.val.grad, L.stats)
    assert A.auv_ppo_work_bytes(0) == -1


def test_ppo_full_minibatch_size(setup):
    """The benchmark's minibatch (262144 samples, the launch configuration it times) from a
    larger buffer: every gradient tensor and loss statistic against the oracle."""
    netp, netv, pol, val, _, _, _, PpoLearner = setup
    B = W.PPO["B"]
    M = B + 16 * 256
    announce(f"ppo full minibatch B={B} M={M}")
    buf = _buffer(M, 12, pol)
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in buf.items()}
    L = PpoLearner(netp, netv)
    idx = W.ppo_minibatch_idx(M, B, seed=7)
    L.grad(L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"]), torch.from_numpy(idx).cuda())
    st = host(L.stats)
    cols = idx.astype(np.int64)
    want = oppo.ppo_loss_grad(buf["obs"][:, cols], buf["act"][:, cols], buf["logp"][cols], buf["adv"][cols],
                              buf["ret"][cols], pol, val, quantize=True)
    _check_grads(host(L.pol.grad), want["grad_pol"], 8, "policy")
    _check_grads(host(L.val.grad), want["grad_val"], 1, "value")
    assert abs(st[0] - want["pg_loss"]) <= 2e-3 * max(1.0, abs(want["pg_loss"]))
    assert st[4] == pytest.approx(want["clip_frac"], abs=0.5 / B)


def test_ppo_grad_ragged_past_the_recompute_switch(setup):
    """131072 - 100 samples: padded to 4096 steps of 32, where the value net's weight gradient
    switches to 128-row blocks with q(h1) recomputed from q(x); 100 padding samples run through
    that path (zero dz2, tanh(b1) as q(h1)) and must add nothing.  Every gradient tensor
    against the oracle."""
    netp, netv, pol, val, _, _, _, PpoLearner = setup
    B = 131072 - 100
    M = B + 16 * 64 + 5
    announce(f"ppo ragged minibatch past the recompute switch B={B} M={M}")
    buf = _buffer(M, 21, pol)
    dev = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in buf.items()}
    L = PpoLearner(netp, netv)
    idx = np.random.default_rng(21).permutation(M)[:B].astype(np.int32)
    L.grad(L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"]), torch.from_numpy(idx).cuda())
    cols = idx.astype(np.int64)
    want = oppo.ppo_loss_grad(buf["obs"][:, cols], buf["act"][:, cols], buf["logp"][cols], buf["adv"][cols],
                              buf["ret"][cols], pol, val, quantize=True)
    _check_grads(host(L.pol.grad), want["grad_pol"], 8, "policy")
    _check_grads(host(L.val.grad), want["grad_val"], 1, "value")


def test_adam_writes_the_weights_the_rollout_reads(setup):
    """After an Adam step the auv_mlp view of a PpoNet (bf16 copy + fp32 tail of theta) is the
    updated network: auv_mlp_forward through it matches the oracle forward of the updated
    parameters (nearest valid bf16 output)."""
    netp, netv, pol, val, buf, dev, M, PpoLearner = setup
    announce("ppo view after adam")
    from oracle.mlp import nearest_valid_error
    from paper_2512_13359_amd import _abi as A
    L = PpoLearner(netp, netv, lr=1e-2)
    idx = W.ppo_minibatch_idx(M, 512, seed=9)
    L.update(L.batch(dev["obs"], dev["act"], dev["logp"], dev["adv"], dev["ret"]), torch.from_numpy(idx).cuda())
    th = host(L.pol.theta)
    new = dict(netp)
    wb = host(L.pol.w_bf16).view(np.uint16)
    n1, n2 = 256 * 23, 256 * 256
    new["W1"], new["W2"], new["W3"] = wb[:n1].reshape(256, 23), wb[n1:n1 + n2].reshape(256, 256), wb[n1 + n2:].reshape(8, 256)
    nw = L.pol.nw
    new["b1"], new["b2"], new["b3"] = th[nw:nw + 256], th[nw + 256:nw + 512], th[nw + 512:nw + 520]
    assert not np.array_equal(wb[:n1], netp["W1"].ravel())           # the step changed the weights
    obs = buf["obs"][:, :300]
    out = torch.empty(8, 300, device="cuda")
    A.auv_mlp_forward(L.pol.mlp, 300, dev["obs"][:, :300].contiguous(), out)
    err = nearest_valid_error(host(out), obs.astype(np.float64), new, 1e-6)
    assert err.max() <= 2e-4, err.max()


def test_ppo_training_loop_on_rollouts():
    """Rollout with sampling and the value head, GAE, then PPO epochs over the rollout buffer,
    all through the C interface: statistics finite, the loss on a fixed minibatch falls over a
    few updates, and the next rollout runs on the updated weights."""
    require_gpu()
    announce("ppo training loop on c5-shaped rollouts")
    from paper_2512_13359_amd import AuvEnv, PpoLearner
    from paper_2512_13359_amd import _abi as A
    cfg = W.config("c5", n_envs=2048, T=32)
    n, T = cfg["n_envs"], cfg["T"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.reset()
    L = PpoLearner(W.mlp_weights(8, W.POLICY_SEED), W.mlp_weights(1, W.VALUE_SEED), lr=1e-3)
    bufs = env.rollout_buffers(T, record=("obs", "act", "logp", "value", "reward", "done", "last_value"), value=True)
    env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    A.auv_gae(T, n, bufs["reward"], bufs["value"], bufs["done"], bufs["last_value"], 0.99, 0.95, adv, ret)
    M = T * n
    batch = L.batch(bufs["obs"].reshape(23, M), bufs["act"].reshape(8, M), bufs["logp"].reshape(M), adv.reshape(M),
                    ret.reshape(M))
    fixed = torch.from_numpy(W.ppo_minibatch_idx(M, 8192, seed=0)).cuda()
    L.grad(batch, fixed)
    first = host(L.stats).copy()
    assert abs(first[3]) < 1e-3            # ratio 1 on fresh samples: approx KL ~ 0 (bf16 policy re-evaluated)
    for k in range(6):
        L.update(batch, fixed)
    L.grad(batch, fixed)
    last = host(L.stats)
    assert np.all(np.isfinite(last))
    assert last[0] + last[1] < first[0] + first[1]
    env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
    r = host(bufs["reward"])
    assert np.all(np.isfinite(r))


def _pad_grad(g: np.ndarray, n_in: int, n_out: int, policy: bool) -> np.ndarray:
    """Gradient of a 12-input / 6-output network in the padded 23 / 8 device layout."""
    p = oppo.unpack(g, n_in, 256, n_out, policy)
    q = {"W1": np.zeros((256, 23)), "W2": p["W2"], "b1": p["b1"], "b2": p["b2"]}
    q["W1"][:, :n_in] = p["W1"]
    no = 8 if n_out > 1 else 1
    q["W3"] = np.zeros((no, 256))
    q["W3"][:n_out] = p["W3"]
    q["b3"] = np.zeros(no)
    q["b3"][:n_out] = p["b3"]
    if policy:
        q["log_std"] = np.zeros(8)
        q["log_std"][:n_out] = p["log_std"]
    return oppo.pack(q)


@pytest.mark.parametrize("M,B", [(5000, 2000), (W.PPO["B"] + 16 * 64 + 3, W.PPO["B"] - 37)])
def test_ppo_six_action_policy_of_the_paper_task(M, B):
    """The paper task's 12-256-256-6 policy and 12-256-256-1 value net in the padded layout:
    gradients against the oracle of the unpadded networks (padding entries exactly zero),
    with NaN in the unused action rows and zeros in observation rows 12-22 (as a paper-task
    rollout records them).  B = 2000 takes the small-minibatch path (q(h1) stored); 262144 - 37,
    the paper-task training minibatch made ragged, the full-size path (q(h1) recomputed)."""
    require_gpu()
    announce(f"ppo six-action policy M={M} B={B}")
    from paper_2512_13359_amd import PpoLearner
    netp = W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12)
    netv = W.mlp_weights(1, W.VALUE_SEED, n_in=12)
    pol, val = _oracle_params(netp), _oracle_params(netv)
    pol["log_std"] = np.asarray(netp["log_std"], np.float32)[:6].astype(np.float64)
    d = W.ppo_draws(M, 21)
    obs12 = d["obs"][:12]
    mu, _ = oppo.mlp_forward_cache(obs12.astype(np.float64), pol, quantize=True)
    act6 = (mu + np.exp(pol["log_std"])[:, None] * d["eps"][:6]).astype(np.float32)
    logp = (oppo.gaussian_logp(act6.astype(np.float64), mu, pol["log_std"]) - np.log(d["ratio"])).astype(np.float32)
    obs23 = np.zeros((23, M), np.float32)
    obs23[:12] = obs12
    act8 = np.full((8, M), np.nan, np.float32)
    act8[:6] = act6
    dev = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (obs23, act8, logp, d["adv"], d["ret"])]
    L = PpoLearner(netp, netv, ent_coef=0.01)
    assert L.cfg.n_actions == 6
    idx = W.ppo_minibatch_idx(M, B, seed=4)
    L.grad(L.batch(*dev), torch.from_numpy(idx).cuda())
    c = idx.astype(np.int64)
    want = oppo.ppo_loss_grad(obs12[:, c], act6[:, c], logp[c], d["adv"][c], d["ret"][c], pol, val,
                              dict(ent_coef=0.01), quantize=True)
    gp, gv = host(L.pol.grad), host(L.val.grad)
    wp, wv = _pad_grad(want["grad_pol"], 12, 6, True), _pad_grad(want["grad_val"], 12, 1, False)
    pad_p = wp == 0.0
    assert np.all(gp[pad_p] == 0.0) and np.all(gv[wv == 0.0] == 0.0)
    _check_grads(gp, wp, 8, "policy")
    _check_grads(gv, wv, 1, "value")
    st = host(L.stats)
    assert abs(st[2] - want["entropy"]) <= 1e-5 * abs(want["entropy"])
    assert abs(st[0] - want["pg_loss"]) <= 2e-3 * max(1.0, abs(want["pg_loss"]))


def test_ppo_training_loop_on_the_paper_task():
    """Paper task end to end: sampled rollout with the value head, GAE, PPO updates of the
    6-action policy; the loss falls on a fixed minibatch and the padding stays zero."""
    require_gpu()
    announce("ppo training loop on the paper task")
    from paper_2512_13359_amd import AuvEnv, PpoLearner
    from paper_2512_13359_amd import _abi as A
    cfg = W.config("c6", n_envs=2048, T=32)
    n, T = cfg["n_envs"], cfg["T"]
    env = AuvEnv(cfg, W.VEHICLE, W.ALLOC)
    env.set_task(W.PAPER_TASK)
    env.reset()
    L = PpoLearner(W.mlp_weights(6, W.PAPER_POLICY_SEED, n_in=12), W.mlp_weights(1, W.VALUE_SEED, n_in=12), lr=1e-3)
    th0 = host(L.pol.theta).copy()
    bufs = env.rollout_buffers(T, record=("obs", "act", "logp", "value", "reward", "done", "last_value"), value=True)
    env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
    adv = torch.empty(T, n, device="cuda")
    ret = torch.empty(T, n, device="cuda")
    A.auv_gae(T, n, bufs["reward"], bufs["value"], bufs["done"], bufs["last_value"], 0.99, 0.95, adv, ret)
    M = T * n
    batch = L.batch(bufs["obs"].reshape(23, M), bufs["act"].reshape(8, M), bufs["logp"].reshape(M), adv.reshape(M),
                    ret.reshape(M))
    fixed = torch.from_numpy(W.ppo_minibatch_idx(M, 8192, seed=0)).cuda()
    L.grad(batch, fixed)
    first = host(L.stats).copy()
    assert abs(first[3]) < 1e-3
    for _ in range(6):
        L.update(batch, fixed)
    L.grad(batch, fixed)
    last = host(L.stats)
    assert np.all(np.isfinite(last)) and last[0] + last[1] < first[0] + first[1]
    th = host(L.pol.theta)
    pad = th0 == 0.0
    pad[:256 * 23] = (np.arange(256 * 23) % 23) >= 12          # W1 columns 12-22
    assert np.all(th[pad & (th0 == 0.0)] == 0.0)


def test_ppo_learns_the_paper_task():
    """End-to-end learning: PPO on the paper task from the seeded networks (1024 envs x one
    512-step episode per iteration, GAE, 4 epochs of 8 minibatches).  The rollouts' mean step
    reward rises steeply within 100 iterations (from about -100 with the initial policy, whose
    large actions and rates are penalised, to a few tenths to units below zero)."""
    require_gpu()
    announce("ppo learns the paper task")
    from paper_2512_13359_amd import AuvEnv, PpoLearner
    from paper_2512_13359_amd import _abi as A
    cfg = W.config("c6", n_envs=1024)
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
    mb = M // 8
    perms = [torch.from_numpy(W.ppo_minibatch_idx(M, M, seed=300 + k)).cuda() for k in range(8)]
    rewards = []
    for it in range(100):
        env.rollout(T, W.MODE_POLICY_SAMPLE, policy={"struct": L.pol.mlp}, value={"struct": L.val.mlp}, bufs=bufs)
        A.auv_gae(T, n, bufs["reward"], bufs["value"], bufs["done"], bufs["last_value"], 0.99, 0.95, adv, ret)
        rewards.append(float(bufs["reward"].mean()))
        for ep in range(4):
            perm = perms[(4 * it + ep) % len(perms)]
            for j in range(8):
                L.update(batch, perm[j * mb:(j + 1) * mb])
    r = np.array(rewards)
    print(f"    mean step reward: it 0 {r[0]:.3f}, it 30 {r[30]:.3f}, it 60 {r[60]:.3f}, it 99 {r[99]:.3f}")
    assert np.isfinite(r).all() and np.isfinite(host(L.stats)).all()
    assert r[0] < -20.0, r[0]
    assert r[-1] > 0.1 * r[0] and r[-1] > -10.0, r[-1]
    assert np.mean(r[-10:]) > np.mean(r[:10]) + 20.0
