"""Oracle of the PPO update (the training loop's update_policy(storage), Fig. 3).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper runs PPO (Sec. 6.1) with the hyperparameters of its configuration
table (Appendix): ratio clip, value-loss coefficient, entropy coefficient,
learning rate with a KL threshold, learning epochs.  It does not restate the
objective; this is Schulman et al.'s clipped surrogate (Proximal Policy
Optimization Algorithms, 2017) in the actor-critic form common to the
frameworks the paper compares against:

  A_hat = (A - mean(A)) / (std(A) + 1e-8)   over the whole rollout (unbiased std)
  logp  = sum_a -( (a - mu)^2 / (2 sigma^2) + log sigma + log(2 pi)/2 )
  ratio = exp(logp - logp_old)
  L_pi  = mean( max(-A_hat ratio, -A_hat clip(ratio, 1 - eps, 1 + eps)) )
  L_V   = mean( max((V - R)^2, (V_old + clip(V - V_old, -eps, eps) - R)^2) )
          (clipped form; unclipped: mean((V - R)^2))
  H     = sum_a (log sigma_a + (1 + log 2 pi) / 2)
  loss  = L_pi + c_V L_V - c_H H
  KL    = mean sum_a ( log(sigma / sigma_old)
                       + (sigma_old^2 + (mu_old - mu)^2) / (2 sigma^2) - 1/2 )

Gradients come from torch autograd in float64 on the CPU.  For bf16 networks
the forward rounds the input, the hidden activations and the weights to bf16
at the same points as the policy forward, and the gradient passes those
roundings unchanged (straight-through: the float32 master weights are what
is trained); the backward rounds the gradient with respect to each layer's
pre-activation to bf16 (the actor's output layer included, the critic's
scalar output not), which is where a bf16 backward stores it.  One Adam step per minibatch (bias-corrected; the gradient of
all parameters clipped to a global norm first); with a KL threshold d the
learning rate is first divided by 1.5 (not below lr_min) when the
minibatch's KL exceeds 2d and multiplied by 1.5 (not above lr_max) when it is
below d/2.
"""
import numpy as np
import torch

LOG_2PI = float(np.log(2.0 * np.pi))


def _bf16(x):
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def _r16(x):
    """Round to bf16 (nearest even) in value, identity in gradient."""
    return x + (_bf16(x) - x).detach()


class _G16(torch.autograd.Function):
    """Identity in value; the gradient passing back is rounded to bf16."""

    @staticmethod
    def forward(ctx, x):
        return x.view_as(x)

    @staticmethod
    def backward(ctx, g):
        return _bf16(g)


def _mlp(x, Ws, bs, bf16, round_out_grad=True):
    """bf16: the input, the weights and the hidden activations are rounded to
    bf16 in the forward, and the gradient with respect to every layer's
    pre-activation is rounded to bf16 in the backward (the output layer's only
    with round_out_grad), where the GPU stores them as GEMM operands."""
    r = _r16 if bf16 else (lambda t: t)
    h = r(x)
    L = len(Ws)
    for l in range(L):
        h = h @ r(Ws[l]).T + bs[l]
        if bf16 and (l < L - 1 or round_out_grad):
            h = _G16.apply(h)
        if l < L - 1:
            h = r(torch.relu(h))
    return h


def flat_params(actor, critic):
    """The parameter vector (float32 masters): actor W_0, b_0, ..., log_std,
    then critic W_0, b_0, ... (row-major weights [out][in])."""
    parts = []
    for W, b in zip(actor["W"], actor["b"]):
        parts += [np.asarray(W, np.float32).ravel(), np.asarray(b, np.float32).ravel()]
    parts.append(np.asarray(actor["log_std"], np.float32).ravel())
    for W, b in zip(critic["W"], critic["b"]):
        parts += [np.asarray(W, np.float32).ravel(), np.asarray(b, np.float32).ravel()]
    return np.concatenate(parts)


def unflat(vec, actor, critic):
    """Inverse of flat_params: (actor, critic) dicts with the vector's values."""
    vec = np.asarray(vec)
    o = 0
    a = dict(actor, W=[], b=[])
    for W, b in zip(actor["W"], actor["b"]):
        a["W"].append(vec[o:o + W.size].reshape(W.shape)); o += W.size
        a["b"].append(vec[o:o + b.size].reshape(b.shape)); o += b.size
    a["log_std"] = vec[o:o + actor["log_std"].size]; o += actor["log_std"].size
    c = dict(critic, W=[], b=[])
    for W, b in zip(critic["W"], critic["b"]):
        c["W"].append(vec[o:o + W.size].reshape(W.shape)); o += W.size
        c["b"].append(vec[o:o + b.size].reshape(b.shape)); o += b.size
    assert o == vec.size
    return a, c


def minibatch(actor, critic, mb, p, adv_mean, adv_std):
    """Loss terms and the float64 gradient (flat_params order) of one minibatch.

    mb: dict of float arrays over the minibatch's samples: obs [M][D],
    action, mean_old [M][A], logp_old, adv, ret, value_old [M]; log_std_old [A].
    p: dict clip, value_coef, entropy_coef, clipped_value_loss."""
    bf16 = bool(actor["bf16"])
    t = lambda a: torch.tensor(np.asarray(a, np.float64), dtype=torch.float64)
    aW = [t(W).requires_grad_() for W in actor["W"]]
    ab = [t(b).requires_grad_() for b in actor["b"]]
    ls = t(actor["log_std"]).requires_grad_()
    cW = [t(W).requires_grad_() for W in critic["W"]]
    cb = [t(b).requires_grad_() for b in critic["b"]]
    obs = t(mb["obs"])
    mu = _mlp(obs, aW, ab, bf16)
    V = _mlp(obs, cW, cb, bf16, round_out_grad=False)[:, 0]
    act = t(mb["action"])
    sig = torch.exp(ls)
    logp = -(((act - mu) ** 2) / (2.0 * sig ** 2) + ls + 0.5 * LOG_2PI).sum(dim=1)
    ratio = torch.exp(logp - t(mb["logp_old"]))
    A = (t(mb["adv"]) - adv_mean) / (adv_std + 1e-8)
    eps = p["clip"]
    l_pi = torch.maximum(-A * ratio, -A * torch.clamp(ratio, 1.0 - eps, 1.0 + eps)).mean()
    R = t(mb["ret"])
    if p["clipped_value_loss"]:
        Vo = t(mb["value_old"])
        Vc = Vo + torch.clamp(V - Vo, -eps, eps)
        l_v = torch.maximum((V - R) ** 2, (Vc - R) ** 2).mean()
    else:
        l_v = ((V - R) ** 2).mean()
    ent = (ls + 0.5 * (1.0 + LOG_2PI)).sum()
    loss = l_pi + p["value_coef"] * l_v - p["entropy_coef"] * ent
    loss.backward()
    ls_old = t(mb["log_std_old"])
    with torch.no_grad():
        so, sn = torch.exp(ls_old), sig
        kl = (ls - ls_old + (so ** 2 + (t(mb["mean_old"]) - mu) ** 2) / (2.0 * sn ** 2)
              - 0.5).sum(dim=1).mean()
        clipfrac = ((ratio - 1.0).abs() > eps).double().mean()
    g = []
    for W, b in zip(aW, ab):
        g += [W.grad.numpy().ravel(), b.grad.numpy().ravel()]
    g.append(ls.grad.numpy().ravel())
    for W, b in zip(cW, cb):
        g += [W.grad.numpy().ravel(), b.grad.numpy().ravel()]
    return dict(loss=loss.item(), l_pi=l_pi.item(), l_v=l_v.item(), entropy=ent.item(),
                kl=float(kl), clipfrac=float(clipfrac), grad=np.concatenate(g))


def adam_step(params, grad, m, v, step, lr, p):
    """One Adam step on float64 copies (clip to the global norm first).
    Returns the new (params, m, v) as float64 arrays; step counts from 1."""
    g = np.asarray(grad, np.float64)
    if p["max_grad_norm"] > 0:
        norm = np.sqrt(np.sum(g * g))
        coef = p["max_grad_norm"] / (norm + 1e-6)
        if coef < 1.0:
            g = g * coef
    b1, b2 = p["beta1"], p["beta2"]
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * g * g
    mh = m / (1.0 - b1 ** step)
    vh = v / (1.0 - b2 ** step)
    return params - lr * mh / (np.sqrt(vh) + p["eps"]), m, v


def adapt_lr(lr, kl, p):
    d = p["desired_kl"]
    if d <= 0:
        return lr
    if kl > 2.0 * d:
        return max(p["lr_min"], lr / 1.5)
    if 0.0 < kl < 0.5 * d:
        return min(p["lr_max"], lr * 1.5)
    return lr


def gather(data, chunks, log_std_old, chunk=64):
    """The minibatch of the given 64-env chunk ids (chunk q = step
    q // (N / chunk), envs chunk * (q % (N / chunk)) onwards), in chunk order."""
    N = np.asarray(data["obs"]).shape[2]
    cpt = N // chunk
    grp = np.asarray(chunks)
    ts = np.repeat(grp // cpt, chunk)
    es = np.repeat((grp % cpt) * chunk, chunk) + np.tile(np.arange(chunk), len(grp))
    return dict(obs=np.asarray(data["obs"])[ts, :, es].astype(np.float32),
                action=data["action"][ts, es], mean_old=data["mean"][ts, es],
                logp_old=data["logp"][ts, es], adv=data["adv"][ts, es], ret=data["ret"][ts, es],
                value_old=data["value"][ts, es], log_std_old=log_std_old)


def adv_stats(adv):
    """Mean and unbiased standard deviation of the rollout's advantages."""
    a = np.asarray(adv, np.float64)
    m = a.mean()
    return m, np.sqrt(((a - m) ** 2).sum() / (a.size - 1))


def update(actor, critic, data, perm, p, lr, chunk=64):
    """The whole update: for every epoch the chunks of perm[epoch] (chunk q =
    step q // (N / chunk), envs chunk * (q % (N / chunk)) onwards) are split
    into p["minibatches"] consecutive groups; each group is one minibatch,
    one adaptive-LR decision and one Adam step.

    data: obs [T][D][N], action / mean [T][N][A], logp / adv / ret [T][N],
    value [T(+1)][N].  Returns (actor, critic, lr, per-minibatch records)."""
    adv_mean, adv_std = adv_stats(data["adv"])
    log_std_old = np.asarray(actor["log_std"], np.float32).copy()
    x = flat_params(actor, critic).astype(np.float64)
    m = np.zeros_like(x)
    v = np.zeros_like(x)
    step = 0
    recs = []
    for ep in range(p["epochs"]):
        q = np.asarray(perm[ep])
        groups = np.array_split(q, p["minibatches"])
        for grp in groups:
            mb = gather(data, grp, log_std_old, chunk)
            a, c = unflat(x.astype(np.float32), actor, critic)
            r = minibatch(a, c, mb, p, adv_mean, adv_std)
            lr = adapt_lr(lr, r["kl"], p)
            step += 1
            x, m, v = adam_step(x, r["grad"], m, v, step, lr, p)
            x = x.astype(np.float32).astype(np.float64)      # the masters are float32
            r["lr"] = lr
            recs.append(r)
    a, c = unflat(x.astype(np.float32), actor, critic)
    return a, c, lr, recs
