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
is trained).  The backward itself is exact float64: how an implementation
stores its intermediate gradients is not part of the method.  One Adam step
per minibatch (bias-corrected; the gradient of all parameters clipped to a
global norm first); with a KL threshold d the learning rate is first divided
by 1.5 (not below lr_min) when the minibatch's KL exceeds 2d and multiplied
by 1.5 (not above lr_max) when it is below d/2.

Besides the whole minibatch, the stages of the gradient are available one by
one, so that an implementation can be compared stage by stage on its own
intermediate values: `layer_forward` (one layer's pre-activation),
`output_grads` (the loss and its gradient with respect to the policy mean,
the value and log_std, given a mean and a value) and `backward` (the chain
rule of an MLP from the gradient at its output).
"""
import numpy as np
import torch

LOG_2PI = float(np.log(2.0 * np.pi))


def _bf16(x):
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def _r16(x):
    """Round to bf16 (nearest even) in value, identity in gradient."""
    return x + (_bf16(x) - x).detach()


def _mlp(x, Ws, bs, bf16):
    """bf16: the input, the weights and the hidden activations are rounded to
    bf16 in the forward (straight-through in the backward)."""
    r = _r16 if bf16 else (lambda t: t)
    h = r(x)
    L = len(Ws)
    for l in range(L):
        h = h @ r(Ws[l]).T + bs[l]
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


def _t(a):
    return torch.tensor(np.asarray(a, np.float64), dtype=torch.float64)


def _loss(mu, V, ls, mb, p, adv_mean, adv_std):
    """The loss terms of a minibatch from the policy mean mu [M][A], the value
    V [M] and log_std [A] (float64 tensors)."""
    act = _t(mb["action"])
    sig = torch.exp(ls)
    logp = -(((act - mu) ** 2) / (2.0 * sig ** 2) + ls + 0.5 * LOG_2PI).sum(dim=1)
    ratio = torch.exp(logp - _t(mb["logp_old"]))
    A = (_t(mb["adv"]) - adv_mean) / (adv_std + 1e-8)
    eps = p["clip"]
    l_pi = torch.maximum(-A * ratio, -A * torch.clamp(ratio, 1.0 - eps, 1.0 + eps)).mean()
    R = _t(mb["ret"])
    if p["clipped_value_loss"]:
        Vo = _t(mb["value_old"])
        Vc = Vo + torch.clamp(V - Vo, -eps, eps)
        l_v = torch.maximum((V - R) ** 2, (Vc - R) ** 2).mean()
    else:
        l_v = ((V - R) ** 2).mean()
    ent = (ls + 0.5 * (1.0 + LOG_2PI)).sum()
    loss = l_pi + p["value_coef"] * l_v - p["entropy_coef"] * ent
    with torch.no_grad():
        so, sn = torch.exp(_t(mb["log_std_old"])), sig
        kl = (ls - _t(mb["log_std_old"]) + (so ** 2 + (_t(mb["mean_old"]) - mu) ** 2) / (2.0 * sn ** 2)
              - 0.5).sum(dim=1).mean()
        clipfrac = ((ratio - 1.0).abs() > eps).double().mean()
    return dict(loss=loss, l_pi=l_pi, l_v=l_v, entropy=ent, kl=kl, clipfrac=clipfrac, ratio=ratio,
                logp=logp)


def minibatch(actor, critic, mb, p, adv_mean, adv_std):
    """Loss terms and the float64 gradient (flat_params order) of one minibatch.

    mb: dict of float arrays over the minibatch's samples: obs [M][D],
    action, mean_old [M][A], logp_old, adv, ret, value_old [M]; log_std_old [A].
    p: dict clip, value_coef, entropy_coef, clipped_value_loss."""
    bf16 = bool(actor["bf16"])
    aW = [_t(W).requires_grad_() for W in actor["W"]]
    ab = [_t(b).requires_grad_() for b in actor["b"]]
    ls = _t(actor["log_std"]).requires_grad_()
    cW = [_t(W).requires_grad_() for W in critic["W"]]
    cb = [_t(b).requires_grad_() for b in critic["b"]]
    obs = _t(mb["obs"])
    mu = _mlp(obs, aW, ab, bf16)
    V = _mlp(obs, cW, cb, bf16)[:, 0]
    r = _loss(mu, V, ls, mb, p, adv_mean, adv_std)
    r["loss"].backward()
    g = []
    for W, b in zip(aW, ab):
        g += [W.grad.numpy().ravel(), b.grad.numpy().ravel()]
    g.append(ls.grad.numpy().ravel())
    for W, b in zip(cW, cb):
        g += [W.grad.numpy().ravel(), b.grad.numpy().ravel()]
    return dict(loss=r["loss"].item(), l_pi=r["l_pi"].item(), l_v=r["l_v"].item(),
                entropy=r["entropy"].item(), kl=float(r["kl"]), clipfrac=float(r["clipfrac"]),
                grad=np.concatenate(g))


def layer_forward(W, b, x):
    """Pre-activation z = x W^T + b of one layer in float64, from the values
    given (for a bf16 network: the bf16 weights and the bf16 input)."""
    return np.asarray(x, np.float64) @ np.asarray(W, np.float64).T + np.asarray(b, np.float64)


def output_grads(mu, V, log_std, mb, p, adv_mean, adv_std):
    """The loss of a minibatch and its float64 gradient with respect to the
    policy mean mu [M][A], the value V [M] and log_std [A], given mu and V
    (e.g. the forward of another implementation).  Also returns each sample's
    ratio and the gradient with respect to each sample's log-likelihood
    (through which the surrogate reaches the mean and log_std)."""
    mu_t = _t(mu).requires_grad_()
    V_t = _t(V).requires_grad_()
    ls = _t(log_std).requires_grad_()
    r = _loss(mu_t, V_t, ls, mb, p, adv_mean, adv_std)
    r["logp"].retain_grad()
    r["loss"].backward()
    return dict(loss=r["loss"].item(), l_pi=r["l_pi"].item(), l_v=r["l_v"].item(),
                kl=float(r["kl"]), clipfrac=float(r["clipfrac"]),
                dmu=mu_t.grad.numpy(), dV=V_t.grad.numpy(), dlog_std=ls.grad.numpy(),
                ratio=r["ratio"].detach().numpy(), dlogp=r["logp"].grad.numpy())


def backward(layers, g_out):
    """The chain rule through an MLP with ReLU hidden layers, in float64.

    layers: [(W_l, x_l)] for l = 0..L-1, W_l [out][in] the weights the forward
    used and x_l [M][in] the input of layer l (for l > 0 the ReLU output of
    layer l - 1, so the ReLU passes the gradient where x_l > 0); g_out [M][out]:
    the gradient of the loss with respect to the last layer's output.
    Returns [(dW_l, db_l, g_l)] with g_l the gradient with respect to layer l's
    pre-activation."""
    out = [None] * len(layers)
    g = np.asarray(g_out, np.float64)
    for l in range(len(layers) - 1, -1, -1):
        W, x = (np.asarray(a, np.float64) for a in layers[l])
        out[l] = (g.T @ x, g.sum(axis=0), g)
        if l > 0:
            g = (g @ W) * (x > 0)
    return out


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
