"""TEST INFRASTRUCTURE: the fp64 oracle of one PPO update of the actor/critic.

The paper trains its actor and critic with PPO (Section 6.1, after Schulman et al., "Proximal
Policy Optimization Algorithms", 2017): Algorithm 1 samples a mini-batch from the replay buffer,
trains the actor with the policy gradient of Eq. 5 (in PPO's clipped form) and the critic with the
MSE of the advantage Y (Eq. 6); Table 5 gives the weights 0.5 (value MSE) and 0.01 (entropy) and the
learning rates 3e-4 (actor) and 1e-3 (critic).

Readings where the paper is silent:
  - network: the shared trunk s -> h1 -> h2 (ReLU) with a linear actor head (the per-type
    segments of harl_policy_select) and a linear value head; parameters in PyTorch nn.Linear
    layout, packed W1, b1, W2, b2, Wa, ba, wv, bv;
  - log-probability of a joint action: the sum over modification types of the segment's
    log-softmax at the chosen action; entropy: the sum of the segments' entropies;
  - loss = -mean(min(ratio A, clip(ratio, 1 - eps, 1 + eps) A)) + w_v mean((V(s) - R)^2)
    - w_e mean(entropy), ratio = exp(logp - logp_old), eps = 0.2 (PPO's default; the paper gives
    none); R = r + gamma V(s') is the critic's target, held fixed (minimising the squared
    advantage of Eq. 6);
  - derivatives at the kinks follow the reference framework's conventions: min passes the
    gradient to the unclipped term when the two are equal, clip passes it for
    1 - eps <= ratio <= 1 + eps, ReLU's derivative at 0 is 0;
  - Adam (beta 0.9 / 0.999, eps 1e-8, bias-corrected), the actor's learning rate for the trunk and
    the actor head, the critic's for the value head.

Only tests/ and bench.py's cpu_baseline leg use this module.
"""
from __future__ import annotations

import numpy as np

PARAM_ORDER = ("w1", "b1", "w2", "b2", "wa", "ba", "wv", "bv")


def param_shapes(s: int, h1: int, h2: int, a: int) -> dict:
    return dict(w1=(h1, s), b1=(h1,), w2=(h2, h1), b2=(h2,), wa=(a, h2), ba=(a,), wv=(1, h2), bv=(1,))


def pack(params: dict) -> np.ndarray:
    return np.concatenate([np.asarray(params[k], np.float64).ravel() for k in PARAM_ORDER])


def unpack(flat, s: int, h1: int, h2: int, a: int) -> dict:
    out, o = {}, 0
    for k in PARAM_ORDER:
        shp = param_shapes(s, h1, h2, a)[k]
        n = int(np.prod(shp))
        out[k] = np.asarray(flat[o:o + n], np.float64).reshape(shp)
        o += n
    return out


def forward(p: dict, X) -> dict:
    """Trunk and heads in fp64 over the given values."""
    X = np.asarray(X, np.float64)
    z1 = X @ p["w1"].T + p["b1"]
    h1 = np.maximum(z1, 0.0)
    z2 = h1 @ p["w2"].T + p["b2"]
    h2 = np.maximum(z2, 0.0)
    logits = h2 @ p["wa"].T + p["ba"]
    v = (h2 @ p["wv"].T)[:, 0] + p["bv"][0]
    return dict(z1=z1, h1=h1, z2=z2, h2=h2, logits=logits, v=v)


def _segment_stats(logits, segs):
    """Per row and segment: log-softmax (full row layout) and entropy."""
    logsm = np.empty_like(logits)
    ent = np.zeros((logits.shape[0], len(segs) - 1))
    for s in range(len(segs) - 1):
        lo, hi = segs[s], segs[s + 1]
        z = logits[:, lo:hi]
        m = z.max(axis=1, keepdims=True)
        lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
        logsm[:, lo:hi] = z - lse
        ent[:, s] = -(np.exp(logsm[:, lo:hi]) * logsm[:, lo:hi]).sum(axis=1)
    return logsm, ent


def loss(p: dict, batch: dict, segs, clip_eps=0.2, w_v=0.5, w_e=0.01) -> dict:
    """The PPO objective of one mini-batch: total and its three terms (fp64)."""
    f = forward(p, batch["states"])
    M = f["logits"].shape[0]
    logsm, ent = _segment_stats(f["logits"], segs)
    act = np.asarray(batch["actions"])
    logp = logsm[np.arange(M)[:, None], act].sum(axis=1)
    ratio = np.exp(logp - np.asarray(batch["logp_old"], np.float64))
    adv = np.asarray(batch["adv"], np.float64)
    s1 = ratio * adv
    s2 = np.clip(ratio, 1 - clip_eps, 1 + clip_eps) * adv
    l_clip = -np.mean(np.minimum(s1, s2))
    l_v = np.mean((f["v"] - np.asarray(batch["ret"], np.float64)) ** 2)
    l_e = np.mean(ent.sum(axis=1))
    return dict(total=l_clip + w_v * l_v - w_e * l_e, clip=l_clip, value=l_v, entropy=l_e, fwd=f, logsm=logsm,
                ent=ent, ratio=ratio, logp=logp, s1=s1, s2=s2)


def grads(p: dict, batch: dict, segs, clip_eps=0.2, w_v=0.5, w_e=0.01, scales: bool = False) -> tuple:
    """Analytic gradient of the PPO objective with respect to every parameter (fp64), and the loss.
    With `scales`, L["scale"] holds for every gradient entry the sum of the absolute values of
    the terms it sums (the basis of a scale-relative tolerance)."""
    L = loss(p, batch, segs, clip_eps, w_v, w_e)
    f = L["fwd"]
    M = f["logits"].shape[0]
    act = np.asarray(batch["actions"])
    adv = np.asarray(batch["adv"], np.float64)
    ratio = L["ratio"]
    # d loss / d logp: the min takes the unclipped term when s1 <= s2; clip passes inside [lo, hi]
    inside = (ratio >= 1 - clip_eps) & (ratio <= 1 + clip_eps)
    active = np.where(L["s1"] <= L["s2"], 1.0, inside.astype(np.float64))
    g_logp = -(adv * ratio * active) / M
    probs = np.exp(L["logsm"])
    dlogits = np.zeros_like(f["logits"])
    for s in range(len(segs) - 1):
        lo, hi = segs[s], segs[s + 1]
        ps = probs[:, lo:hi]
        onehot = np.zeros_like(ps)
        onehot[np.arange(M), act[:, s] - lo] = 1.0
        # d logp / d z = onehot - p ; d entropy / d z = -p (log p + H)
        dent = -ps * (L["logsm"][:, lo:hi] + L["ent"][:, s:s + 1])
        dlogits[:, lo:hi] = g_logp[:, None] * (onehot - ps) - (w_e / M) * dent
    dv = w_v * 2.0 * (f["v"] - np.asarray(batch["ret"], np.float64)) / M
    X = np.asarray(batch["states"], np.float64)
    g = {}
    g["wa"] = dlogits.T @ f["h2"]
    g["ba"] = dlogits.sum(axis=0)
    g["wv"] = (dv @ f["h2"])[None, :]
    g["bv"] = np.array([dv.sum()])
    dh2 = dlogits @ p["wa"] + dv[:, None] * p["wv"][0][None, :]
    dz2 = dh2 * (f["z2"] > 0)
    g["w2"] = dz2.T @ f["h1"]
    g["b2"] = dz2.sum(axis=0)
    dh1 = dz2 @ p["w2"]
    dz1 = dh1 * (f["z1"] > 0)
    g["w1"] = dz1.T @ X
    g["b1"] = dz1.sum(axis=0)
    if scales:
        L["scale"] = _grad_scales(p, X, f, L, g_logp, dlogits, dv, dz2, dz1, segs, w_v, w_e)
    return g, L


def _grad_scales(p, X, f, L, g_logp, dlogits, dv, dz2, dz1, segs, w_v, w_e) -> dict:
    """A running error scale T(q) for every quantity q of the update: q's formula evaluated on the
    absolute values of its factors and the scales of its inner quantities, carried from the inputs
    through the forward pass, the objective's gradient at the logits and backpropagation.  An
    fp32 evaluation of q errs by a small multiple of 2^-24 T(q)."""
    A = np.abs
    M = X.shape[0]
    m1, m2 = (f["z1"] > 0), (f["z2"] > 0)
    t_h1 = (A(X) @ A(p["w1"]).T + A(p["b1"])) * m1
    t_h2 = (t_h1 @ A(p["w2"]).T + A(p["b2"])) * m2
    t_z = t_h2 @ A(p["wa"]).T + A(p["ba"])
    t_v = (t_h2 @ A(p["wv"]).T)[:, 0] + A(p["bv"][0])
    probs = np.exp(L["logsm"])
    t_dl = np.zeros_like(dlogits)
    for s in range(len(segs) - 1):
        lo, hi = segs[s], segs[s + 1]
        ps, ls = probs[:, lo:hi], A(L["logsm"][:, lo:hi])
        H = L["ent"][:, s:s + 1]
        own = A(g_logp)[:, None] * (1.0 + ps) + (w_e / M) * ps * (ls + H)
        # sensitivity to the logits' errors (through the softmax and the ratio of every type)
        sens = (A(g_logp)[:, None] * (len(segs) - 1) + w_e / M) * (1.0 + ls + H) * t_z.max(axis=1, keepdims=True)
        t_dl[:, lo:hi] = own + sens
    t_dv = A(dv) + w_v * 2.0 / M * (t_v + A(f["v"]))
    t_dz2 = (t_dl @ A(p["wa"]) + t_dv[:, None] * A(p["wv"][0])[None, :]) * m2
    t_dz1 = (t_dz2 @ A(p["w2"])) * m1
    return dict(wa=t_dl.T @ A(f["h2"]) + A(dlogits).T @ t_h2, ba=t_dl.sum(axis=0),
                wv=(t_dv @ A(f["h2"]) + A(dv) @ t_h2)[None, :], bv=np.array([t_dv.sum()]),
                w2=t_dz2.T @ A(f["h1"]) + A(dz2).T @ t_h1, b2=t_dz2.sum(axis=0),
                w1=t_dz1.T @ A(X), b1=t_dz1.sum(axis=0))


def adam(flat_p, flat_g, m, v, step: int, lr, beta1=0.9, beta2=0.999, eps=1e-8):
    """One bias-corrected Adam step (fp64); lr may be a per-parameter array.  Returns new
    (params, m, v)."""
    m = beta1 * m + (1 - beta1) * flat_g
    v = beta2 * v + (1 - beta2) * flat_g * flat_g
    mhat = m / (1 - beta1 ** step)
    vhat = v / (1 - beta2 ** step)
    return flat_p - lr * mhat / (np.sqrt(vhat) + eps), m, v


def lr_vector(s: int, h1: int, h2: int, a: int, lr_actor=3e-4, lr_critic=1e-3) -> np.ndarray:
    """The actor's rate for the trunk and the actor head, the critic's for the value head."""
    parts = []
    for k in PARAM_ORDER:
        n = int(np.prod(param_shapes(s, h1, h2, a)[k]))
        parts.append(np.full(n, lr_critic if k in ("wv", "bv") else lr_actor))
    return np.concatenate(parts)


def update(flat_p, m, v, step: int, batch: dict, segs, dims, clip_eps=0.2, w_v=0.5, w_e=0.01, lr_actor=3e-4,
           lr_critic=1e-3) -> dict:
    """One PPO update: gradients of the mini-batch objective, then Adam."""
    s, h1, h2, a = dims
    p = unpack(flat_p, s, h1, h2, a)
    g, L = grads(p, batch, segs, clip_eps, w_v, w_e)
    flat_g = pack(g)
    newp, m2, v2 = adam(np.asarray(flat_p, np.float64), flat_g, m, v, step, lr_vector(s, h1, h2, a, lr_actor, lr_critic))
    return dict(params=newp, m=m2, v=v2, grad=flat_g, loss=np.array([L["total"], L["clip"], L["value"], L["entropy"]]))
