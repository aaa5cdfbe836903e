"""Pins of the PPO-update oracle: its gradient against finite differences of
its own loss and against per-term closed forms, the KL against torch's
distribution KL, the clipped surrogate's dead zones, Adam and the norm clip
against torch.optim / torch.nn.utils, the adaptive learning rate, and the
minibatch bookkeeping of the whole update."""
import numpy as np
import pytest
import torch

from oracle import ppo
from paper_2609_09821_amd import synth

P = dict(clip=0.2, value_coef=2.0, entropy_coef=2.5e-4, clipped_value_loss=True,
         max_grad_norm=1.0, beta1=0.9, beta2=0.999, eps=1e-8, desired_kl=0.008,
         lr_min=1e-5, lr_max=1e-2)


def _nets(D=12, H=(16, 8), A=3, bf16=False, seed=0):
    rng = np.random.default_rng(seed)
    actor = synth.make_policy(rng, [D, *H, A], bf16, sigma=0.3)
    critic = synth.make_policy(rng, [D, *H, 1], bf16)
    return actor, critic


def _mb(actor, M=40, seed=1, ratio_noise=0.1):
    rng = np.random.default_rng(seed)
    D = actor["dims"][0]
    A = actor["dims"][-1]
    obs = rng.normal(size=(M, D)).astype(np.float32)
    mean_old = rng.normal(scale=0.3, size=(M, A)).astype(np.float32)
    sig = np.exp(actor["log_std"].astype(np.float64))
    act = (mean_old + sig * rng.normal(size=(M, A))).astype(np.float32)
    logp_old = (-(((act - mean_old) ** 2) / (2 * sig ** 2) + np.log(sig) + 0.5 * ppo.LOG_2PI)
                .sum(axis=1) + rng.normal(scale=ratio_noise, size=M)).astype(np.float32)
    return dict(obs=obs, action=act, mean_old=mean_old, logp_old=logp_old,
                adv=rng.normal(size=M).astype(np.float32),
                ret=rng.normal(size=M).astype(np.float32),
                value_old=rng.normal(size=M).astype(np.float32),
                log_std_old=actor["log_std"].astype(np.float32).copy())


def _loss_at(actor, critic, mb, p, vec):
    a, c = ppo.unflat(vec, actor, critic)
    a = dict(a, W=[w.astype(np.float64) for w in a["W"]])
    return ppo.minibatch(a, c, mb, p, 0.1, 1.3)["loss"]


@pytest.mark.parametrize("clipped", [False, True])
def test_gradient_matches_finite_differences(clipped):
    actor, critic = _nets()
    mb = _mb(actor)
    p = dict(P, clipped_value_loss=clipped)
    r = ppo.minibatch(actor, critic, mb, p, 0.1, 1.3)
    x = ppo.flat_params(actor, critic).astype(np.float64)
    rng = np.random.default_rng(3)
    idx = rng.choice(x.size, size=60, replace=False)
    h = 1e-6
    for i in idx:
        xp, xm = x.copy(), x.copy()
        xp[i] += h
        xm[i] -= h
        fd = (_loss_at(actor, critic, mb, p, xp) - _loss_at(actor, critic, mb, p, xm)) / (2 * h)
        assert abs(fd - r["grad"][i]) <= 1e-5 * max(1.0, abs(fd)), (i, fd, r["grad"][i])


def test_flat_round_trip():
    actor, critic = _nets()
    x = ppo.flat_params(actor, critic)
    a, c = ppo.unflat(x, actor, critic)
    assert np.array_equal(ppo.flat_params(a, c), x)
    n = sum(w.size + b.size for w, b in zip(actor["W"], actor["b"])) + 3 + \
        sum(w.size + b.size for w, b in zip(critic["W"], critic["b"]))
    assert x.size == n


def _segments(actor, critic):
    """name -> slice of the flat vector."""
    out, o = {}, 0
    for l, (W, b) in enumerate(zip(actor["W"], actor["b"])):
        out["aW%d" % l] = slice(o, o + W.size); o += W.size
        out["ab%d" % l] = slice(o, o + b.size); o += b.size
    out["log_std"] = slice(o, o + actor["log_std"].size); o += actor["log_std"].size
    for l, (W, b) in enumerate(zip(critic["W"], critic["b"])):
        out["cW%d" % l] = slice(o, o + W.size); o += W.size
        out["cb%d" % l] = slice(o, o + b.size); o += b.size
    return out


def test_last_layer_gradients_closed_form():
    # one-layer actor and critic: the gradient of the output layer is the
    # per-sample output gradient times the input, summed
    actor, critic = _nets(H=())
    mb = _mb(actor, ratio_noise=0.0)
    p = dict(P, clipped_value_loss=False, entropy_coef=0.0)
    am, asd = 0.2, 0.9
    r = ppo.minibatch(actor, critic, mb, p, am, asd)
    seg = _segments(actor, critic)
    X = mb["obs"].astype(np.float64)
    M = X.shape[0]
    W, b = actor["W"][0].astype(np.float64), actor["b"][0].astype(np.float64)
    mu = X @ W.T + b
    sig = np.exp(actor["log_std"].astype(np.float64))
    act = mb["action"].astype(np.float64)
    logp = -(((act - mu) ** 2) / (2 * sig ** 2) + np.log(sig) + 0.5 * ppo.LOG_2PI).sum(axis=1)
    ratio = np.exp(logp - mb["logp_old"])
    A = (mb["adv"].astype(np.float64) - am) / (asd + 1e-8)
    active = np.where(A >= 0, ratio < 1 + p["clip"], ratio > 1 - p["clip"])
    dlogp = np.where(active, -A * ratio, 0.0) / M
    dmu = dlogp[:, None] * (act - mu) / sig ** 2
    np.testing.assert_allclose(r["grad"][seg["aW0"]], (dmu.T @ X).ravel(), rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(r["grad"][seg["ab0"]], dmu.sum(axis=0), rtol=1e-9, atol=1e-12)
    dls = (dlogp[:, None] * ((act - mu) ** 2 / sig ** 2 - 1.0)).sum(axis=0)
    np.testing.assert_allclose(r["grad"][seg["log_std"]], dls, rtol=1e-9, atol=1e-12)
    Wc, bc = critic["W"][0].astype(np.float64), critic["b"][0].astype(np.float64)
    V = (X @ Wc.T + bc)[:, 0]
    dV = 2.0 * p["value_coef"] * (V - mb["ret"].astype(np.float64)) / M
    np.testing.assert_allclose(r["grad"][seg["cW0"]], (dV @ X), rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(r["grad"][seg["cb0"]], [dV.sum()], rtol=1e-9)


def test_entropy_term_and_kl():
    actor, critic = _nets()
    mb = _mb(actor)
    r0 = ppo.minibatch(actor, critic, mb, dict(P, entropy_coef=0.0), 0.0, 1.0)
    r1 = ppo.minibatch(actor, critic, mb, dict(P, entropy_coef=0.5), 0.0, 1.0)
    seg = _segments(actor, critic)
    np.testing.assert_allclose(r1["grad"][seg["log_std"]] - r0["grad"][seg["log_std"]], -0.5,
                               rtol=1e-9)
    sig = np.exp(actor["log_std"].astype(np.float64))
    np.testing.assert_allclose(r0["entropy"], (np.log(sig) + 0.5 * (1 + ppo.LOG_2PI)).sum())
    # KL against torch's Normal KL, summed over actions and averaged over samples
    a = dict(actor, W=[w.astype(np.float64) for w in actor["W"]])
    mu = ppo._mlp(torch.tensor(mb["obs"], dtype=torch.float64),
                  [torch.tensor(w) for w in a["W"]],
                  [torch.tensor(b, dtype=torch.float64) for b in actor["b"]], False)
    old = torch.distributions.Normal(torch.tensor(mb["mean_old"], dtype=torch.float64),
                                     torch.exp(torch.tensor(mb["log_std_old"], dtype=torch.float64)))
    new = torch.distributions.Normal(mu, torch.exp(torch.tensor(actor["log_std"], dtype=torch.float64)))
    kl = torch.distributions.kl_divergence(old, new).sum(dim=1).mean().item()
    np.testing.assert_allclose(r0["kl"], kl, rtol=1e-10)


def test_clipped_samples_have_no_policy_gradient():
    actor, critic = _nets(H=())
    mb = _mb(actor, ratio_noise=0.0)
    # push every ratio to e^5, far above 1 + eps, and make every advantage positive
    mu = ppo._mlp(torch.tensor(mb["obs"], dtype=torch.float64),
                  [torch.tensor(w, dtype=torch.float64) for w in actor["W"]],
                  [torch.tensor(b, dtype=torch.float64) for b in actor["b"]], False).numpy()
    sig = np.exp(actor["log_std"].astype(np.float64))
    act = mb["action"].astype(np.float64)
    logp = -(((act - mu) ** 2) / (2 * sig ** 2) + np.log(sig) + 0.5 * ppo.LOG_2PI).sum(axis=1)
    mb["logp_old"] = (logp - 5.0).astype(np.float32)
    mb["adv"] = np.abs(mb["adv"]) + 0.5
    p = dict(P, entropy_coef=0.0)
    r = ppo.minibatch(actor, critic, mb, p, 0.0, 1.0)
    seg = _segments(actor, critic)
    assert np.all(r["grad"][seg["aW0"]] == 0) and np.all(r["grad"][seg["log_std"]] == 0)
    assert r["clipfrac"] == 1.0
    # negative advantages with ratios above 1 + eps are not clipped
    mb["adv"] = -mb["adv"]
    r = ppo.minibatch(actor, critic, mb, p, 0.0, 1.0)
    assert np.any(r["grad"][seg["aW0"]] != 0)


def test_adam_and_norm_clip_match_torch():
    rng = np.random.default_rng(9)
    x0 = rng.normal(size=50)
    grads = [rng.normal(scale=s, size=50) for s in (3.0, 0.01, 0.5)]
    p = dict(P, max_grad_norm=1.0)
    t = torch.tensor(x0.copy(), requires_grad=True)
    opt = torch.optim.Adam([t], lr=1e-3, betas=(p["beta1"], p["beta2"]), eps=p["eps"])
    x, m, v = x0.copy(), np.zeros(50), np.zeros(50)
    for k, g in enumerate(grads):
        opt.zero_grad()
        t.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_([t], p["max_grad_norm"])
        opt.step()
        x, m, v = ppo.adam_step(x, g, m, v, k + 1, 1e-3, p)
        np.testing.assert_allclose(x, t.detach().numpy(), rtol=1e-10, atol=1e-13)


def test_adaptive_learning_rate():
    p = P
    d = p["desired_kl"]
    assert ppo.adapt_lr(1e-3, 2.5 * d, p) == pytest.approx(1e-3 / 1.5)
    assert ppo.adapt_lr(1e-3, 0.4 * d, p) == pytest.approx(1.5e-3)
    assert ppo.adapt_lr(1e-3, d, p) == 1e-3
    assert ppo.adapt_lr(1e-3, 1.9 * d, p) == 1e-3 and ppo.adapt_lr(1e-3, 0.6 * d, p) == 1e-3
    assert ppo.adapt_lr(1e-3, 0.0, p) == 1e-3
    assert ppo.adapt_lr(1.2e-5, 10 * d, p) == p["lr_min"]
    assert ppo.adapt_lr(9e-3, 0.1 * d, p) == p["lr_max"]
    assert ppo.adapt_lr(1e-3, 10 * d, dict(p, desired_kl=0.0)) == 1e-3


def _rollout_data(actor, critic, T=3, N=128, seed=4):
    rng = np.random.default_rng(seed)
    D, A = actor["dims"][0], actor["dims"][-1]
    obs = rng.normal(size=(T, D, N)).astype(np.float32)
    mean = rng.normal(scale=0.3, size=(T, N, A)).astype(np.float32)
    act = (mean + 0.3 * rng.normal(size=(T, N, A))).astype(np.float32)
    return dict(obs=obs, action=act, mean=mean,
                logp=rng.normal(size=(T, N)).astype(np.float32) - 3.0,
                adv=rng.normal(size=(T, N)).astype(np.float32),
                ret=rng.normal(size=(T, N)).astype(np.float32),
                value=rng.normal(size=(T + 1, N)).astype(np.float32))


def test_update_bookkeeping():
    actor, critic = _nets()
    data = _rollout_data(actor, critic)
    n_chunks = 3 * 128 // 64
    perm = np.stack([np.random.default_rng(e).permutation(n_chunks) for e in range(2)])
    p = dict(P, epochs=2, minibatches=2)
    # zero learning rate and no adaptation: nothing moves
    a, c, lr, recs = ppo.update(actor, critic, data, perm, dict(p, desired_kl=0.0), 0.0)
    assert np.array_equal(ppo.flat_params(a, c), ppo.flat_params(actor, critic))
    assert len(recs) == 4 and lr == 0.0
    # one epoch, one minibatch: the update is one minibatch step on all samples
    p1 = dict(p, epochs=1, minibatches=1, desired_kl=0.0)
    a, c, lr, recs = ppo.update(actor, critic, data, perm[:1], p1, 1e-3)
    ts = np.repeat(perm[0] // 2, 64)
    es = np.repeat((perm[0] % 2) * 64, 64) + np.tile(np.arange(64), n_chunks)
    mb = dict(obs=data["obs"][ts, :, es], action=data["action"][ts, es],
              mean_old=data["mean"][ts, es], logp_old=data["logp"][ts, es],
              adv=data["adv"][ts, es], ret=data["ret"][ts, es], value_old=data["value"][ts, es],
              log_std_old=actor["log_std"])
    adv = data["adv"].astype(np.float64)
    r = ppo.minibatch(actor, critic, mb, p1, adv.mean(), adv.std(ddof=1))
    x = ppo.flat_params(actor, critic).astype(np.float64)
    x1, _, _ = ppo.adam_step(x, r["grad"], np.zeros_like(x), np.zeros_like(x), 1, 1e-3, p1)
    np.testing.assert_array_equal(ppo.flat_params(a, c), x1.astype(np.float32))


def test_bf16_network_gradient_passes_the_roundings():
    # bf16 rounding points change values by ~2^-9 relative: the gradient stays
    # close to the float32 network's (first layers least: a rare ReLU that
    # flips moves their sums by a few per cent), and is not cut at the roundings
    actor, critic = _nets(D=48, H=(256, 128), A=6, bf16=False, seed=5)
    mb = _mb(actor, M=400, seed=6)
    r32 = ppo.minibatch(actor, critic, mb, P, 0.0, 1.0)
    r16 = ppo.minibatch(dict(actor, bf16=True), dict(critic, bf16=True), mb, P, 0.0, 1.0)
    seg = _segments(actor, critic)
    for k, tol in (("aW0", 0.15), ("aW1", 0.05), ("aW2", 0.05), ("cW0", 0.15), ("cW1", 0.1),
                   ("cW2", 0.05), ("log_std", 0.05)):
        g32, g16 = r32["grad"][seg[k]], r16["grad"][seg[k]]
        assert np.linalg.norm(g16 - g32) <= tol * np.linalg.norm(g32), k
    assert not np.array_equal(r32["grad"], r16["grad"])


def _staged(actor, critic, mb, p, am, asd):
    """The minibatch gradient composed from the staged oracle functions on the
    oracle's own forward: layer_forward per layer (bf16 rounding points as the
    policy forward), output_grads at the resulting mean and value, backward
    through each network."""
    bf16 = bool(actor["bf16"])
    r16 = (lambda a: ppo._bf16(torch.tensor(np.asarray(a, np.float64))).numpy()) if bf16 else \
        (lambda a: np.asarray(a, np.float64))

    def forward(net):
        x = r16(mb["obs"])
        layers = []
        for l, (W, b) in enumerate(zip(net["W"], net["b"])):
            Wr = r16(W)
            layers.append((Wr, x))
            z = ppo.layer_forward(Wr, b, x)
            x = r16(np.maximum(z, 0.0)) if l + 1 < len(net["W"]) else z
        return layers, x

    al, mu = forward(actor)
    cl, V = forward(critic)
    o = ppo.output_grads(mu, V[:, 0], actor["log_std"], mb, p, am, asd)
    g = []
    for dW, db, _ in ppo.backward(al, o["dmu"]):
        g += [dW.ravel(), db]
    g.append(o["dlog_std"])
    for dW, db, _ in ppo.backward(cl, o["dV"][:, None]):
        g += [dW.ravel(), db]
    return np.concatenate(g), o, mu


@pytest.mark.parametrize("bf16", [False, True])
def test_staged_gradient_equals_the_minibatch_gradient(bf16):
    # two routes to the same derivative: torch autograd through the whole
    # minibatch, and the chain rule written out stage by stage (forward per
    # layer, loss gradient at the output, backward through each network);
    # bf16 networks: straight-through at every rounding point in both
    actor, critic = _nets(D=24, H=(32, 16), A=5, bf16=bf16, seed=11)
    mb = _mb(actor, M=64, seed=12)
    p = dict(P, clipped_value_loss=True)
    r = ppo.minibatch(actor, critic, mb, p, 0.1, 1.3)
    g, o, mu = _staged(actor, critic, mb, p, 0.1, 1.3)
    np.testing.assert_allclose(g, r["grad"], rtol=1e-10, atol=1e-13)
    assert o["loss"] == pytest.approx(r["loss"], rel=1e-12)
    # the surrogate reaches log_std through each sample's log-likelihood:
    # d logp_s / d log_std_a = (a - mu)^2 / sigma^2 - 1, plus the entropy term
    sig = np.exp(actor["log_std"].astype(np.float64))
    dl = (o["dlogp"][:, None] * ((mb["action"] - mu) ** 2 / sig ** 2 - 1.0)).sum(axis=0)
    np.testing.assert_allclose(dl - p["entropy_coef"], o["dlog_std"], rtol=1e-10, atol=1e-14)


def test_backward_of_a_two_layer_network_by_hand():
    # y = W1 relu(W0 x + b0) + b1 on two samples, the output gradient given:
    # the gradients written out element by element
    W0 = np.array([[1.0, -2.0], [0.5, 0.25], [-1.0, 1.0]])
    W1 = np.array([[2.0, -1.0, 3.0]])
    x = np.array([[1.0, 0.5], [-2.0, 1.0]])
    b0 = np.array([0.1, 0.0, -0.2])
    h = np.maximum(x @ W0.T + b0, 0.0)      # [[0.1, 0.625, 0.0], [0.0, 0.0, 2.8]]
    g = np.array([[0.5], [-1.0]])
    (dW0, db0, g0), (dW1, db1, g1) = ppo.backward([(W0, x), (W1, h)], g)
    np.testing.assert_allclose(dW1, [[0.5 * 0.1, 0.5 * 0.625, -1.0 * 2.8]])
    np.testing.assert_allclose(db1, [-0.5])
    # layer-0 gradient: W1^T g where h > 0: sample 0 units 0, 1; sample 1 unit 2
    np.testing.assert_allclose(g0, [[1.0, -0.5, 0.0], [0.0, 0.0, -3.0]])
    np.testing.assert_allclose(dW0, [[1.0, 0.5], [-0.5, -0.25], [6.0, -3.0]])
    np.testing.assert_allclose(db0, [1.0, -0.5, -3.0])


@pytest.mark.parametrize("bf16", [False, True])
def test_forward_is_the_policy_forward(bf16):
    # the update's forward equals the rollout's (the C oracle's policy mean)
    import oracle
    actor, _ = _nets(D=20, H=(32, 16), A=5, bf16=bf16, seed=8)
    obs = np.random.default_rng(2).normal(size=(20, 30)).astype(np.float32)
    mean, _, _ = oracle.policy(actor, 0, obs, np.zeros(30, np.uint32))
    mu = ppo._mlp(torch.tensor(obs.T, dtype=torch.float64),
                  [torch.tensor(w, dtype=torch.float64) for w in actor["W"]],
                  [torch.tensor(b, dtype=torch.float64) for b in actor["b"]], bf16).numpy()
    np.testing.assert_allclose(mu, mean, rtol=1e-5, atol=1e-6 if not bf16 else 2e-3)


def test_clipped_value_loss_by_hand():
    actor, critic = _nets(H=())
    mb = _mb(actor, M=4)
    X = mb["obs"].astype(np.float64)
    V = (X @ critic["W"][0].astype(np.float64).T + critic["b"][0])[:, 0]
    eps = P["clip"]
    # V moved 3 eps above V_old; the return far above V: the clipped
    # prediction V_old + eps is further from it and is the one penalised
    mb["value_old"] = (V - 3 * eps).astype(np.float32)
    mb["ret"] = (V + 10.0).astype(np.float32)
    p = dict(P, entropy_coef=0.0)
    r = ppo.minibatch(actor, critic, mb, p, 0.0, 1.0)
    Vc = mb["value_old"].astype(np.float64) + eps
    np.testing.assert_allclose(r["l_v"], np.mean((Vc - mb["ret"]) ** 2), rtol=1e-6)
    seg = _segments(actor, critic)
    assert np.all(r["grad"][seg["cW0"]] == 0) and np.all(r["grad"][seg["cb0"]] == 0)
    # the return below V: the unclipped error is the larger one
    mb["ret"] = (V - 10.0).astype(np.float32)
    r = ppo.minibatch(actor, critic, mb, p, 0.0, 1.0)
    np.testing.assert_allclose(r["l_v"], np.mean((V - mb["ret"]) ** 2), rtol=1e-6)
    np.testing.assert_allclose(r["grad"][seg["cb0"]],
                               [np.sum(2 * p["value_coef"] * (V - mb["ret"]) / 4)], rtol=1e-6)
