"""GPU parity of harl_ppo_update (one PPO update of the actor/critic: Algorithm 1's training step,
Eq. 5 in PPO's clipped form, the critic's MSE of Eq. 6's advantage; Section 6.1; Table 5) against
the fp64 oracle (oracle/ppo.py).

Bars: loss terms within 1e-4 relative; every gradient entry within 1e-5 of its running error scale
(the oracle's T: the entry's formula on absolute values, carried through the forward pass, the
objective's gradient and backpropagation -- an fp32 evaluation errs by a small multiple of 2^-24 T); the Adam moments and
parameters equal, within fp32 rounding, to the oracle's Adam applied to the GPU's own gradient
(Adam divides by |gradient|, so a gradient entry near 0 makes the step's sign, not the bars above,
decide the parameter); repeated updates bit-identical."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import ppo
from synth import gen_policy, gen_states, get_config
from tests.gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

SEGS = [0, 17, 20, 23, 26]


def _setup(M, dims=(64, 256, 256, 26), segs=SEGS, seed=0, spread=0.3):
    s, h1, h2, a = dims
    cfg = get_config("standard").with_(pol_s=s, pol_h1=h1, pol_h2=h2, pol_a=a, n_prog=M)
    pol = gen_policy(cfg)
    params = dict(w1=pol["w1"], b1=pol["b1"], w2=pol["w2"], b2=pol["b2"], wa=pol["wa"], ba=pol["ba"],
                  wv=np.asarray(pol["wv"]).reshape(1, h2), bv=np.asarray(pol["bv"]).reshape(1))
    flat = ppo.pack(params).astype(np.float32)
    X = gen_states(cfg).astype(np.float32)
    rng = np.random.default_rng(seed)
    acts = np.stack([rng.integers(segs[i], segs[i + 1], M) for i in range(len(segs) - 1)], axis=1).astype(np.int32)
    p64 = ppo.unpack(flat.astype(np.float64), *dims)
    L = ppo.loss(p64, dict(states=X, actions=acts, logp_old=np.zeros(M), adv=np.zeros(M), ret=np.zeros(M)), segs)
    batch = dict(states=X, actions=acts,
                 logp_old=(L["logp"] + rng.uniform(-spread, spread, M)).astype(np.float32),
                 adv=rng.standard_normal(M).astype(np.float32),
                 ret=(L["fwd"]["v"] + rng.standard_normal(M)).astype(np.float32))
    return flat, batch


def _gpu_update(flat, batch, dims, segs, steps=1, m=None, v=None):
    import torch
    from paper_2211_11172_amd import harl
    s, h1, h2, a = dims
    cfg = harl.ppo_config(s, h1, h2, a, segs)
    n = harl.harl_ppo_param_count(cfg)
    assert n == flat.size
    M = batch["states"].shape[0]
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    P = d(flat.copy())
    Mm = d(np.zeros(n, np.float32) if m is None else m.astype(np.float32))
    Vv = d(np.zeros(n, np.float32) if v is None else v.astype(np.float32))
    grad = torch.full((n,), np.nan, device="cuda")
    loss = torch.full((4,), np.nan, device="cuda")
    wsb = harl.harl_ppo_workspace_size(cfg, M)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    args = [d(batch[k]) for k in ("states", "actions", "logp_old", "adv", "ret")]
    out = []
    for step in range(1, steps + 1):
        harl.harl_ppo_update(cfg, P, Mm, Vv, step, *args, M, grad, loss, ws, wsb)
        torch.cuda.synchronize()
        out.append(dict(params=P.cpu().numpy().copy(), m=Mm.cpu().numpy().copy(), v=Vv.cpu().numpy().copy(),
                        grad=grad.cpu().numpy().copy(), loss=loss.cpu().numpy().copy()))
    return out


def _check_step(flat_before, m0, v0, step, batch, got, dims, segs):
    p64 = ppo.unpack(flat_before.astype(np.float64), *dims)
    g, L = ppo.grads(p64, dict(batch), segs, scales=True)
    want_loss = np.array([L["total"], L["clip"], L["value"], L["entropy"]])
    np.testing.assert_allclose(got["loss"], want_loss, rtol=1e-4, atol=1e-6)
    gg = ppo.unpack(got["grad"].astype(np.float64), *dims)
    worst = 0.0
    for k in ppo.PARAM_ORDER:
        err = np.abs(gg[k] - g[k])
        tol = 1e-5 * L["scale"][k] + 1e-12
        worst = max(worst, float((err / tol).max()))
        assert (err <= tol).all(), "%s: %d entries beyond tolerance (max err/tol %.3g)" % (k, int((err > tol).sum()),
                                                                                            float((err / tol).max()))
    log("ppo gradient: max err/tol %.3g" % worst)
    # Adam on the GPU's own gradient, with the hyper-parameters at the fp32 values the ABI takes
    f32 = lambda x: float(np.float32(x))
    lr = ppo.lr_vector(*dims, lr_actor=f32(3e-4), lr_critic=f32(1e-3))
    newp, m1, v1 = ppo.adam(flat_before.astype(np.float64), got["grad"].astype(np.float64), m0, v0, step, lr,
                            beta1=f32(0.9), beta2=f32(0.999), eps=f32(1e-8))
    g64 = got["grad"].astype(np.float64)
    assert np.all(np.abs(got["m"] - m1) <= 1e-6 * (0.9 * np.abs(m0) + 0.1 * np.abs(g64)) + 1e-30)
    np.testing.assert_allclose(got["v"], v1, rtol=1e-5, atol=1e-30)
    assert np.all(np.abs(got["params"] - newp) <= 1e-6 * np.abs(newp) + 1e-3 * lr)
    return m1, v1


@pytest.mark.parametrize("M", [1, 70, 1000, 4096, 20000, 65536])  # 20,000+: two-stage loss, up to 128 split pieces
def test_ppo_update_matches_oracle(M):
    require_gpu()
    dims = (64, 256, 256, 26)
    flat, batch = _setup(M, dims)
    log("ppo update parity: M=%d dims=%s" % (M, dims))
    out = _gpu_update(flat, batch, dims, SEGS, steps=2)
    _check_step(flat, np.zeros(flat.size), np.zeros(flat.size), 1, batch, out[0], dims, SEGS)
    # the second step from the GPU's own first-step state (bias correction of step 2)
    _check_step(out[0]["params"], out[0]["m"].astype(np.float64), out[0]["v"].astype(np.float64), 2, batch, out[1],
                dims, SEGS)


def test_ppo_update_odd_shapes_and_segments():
    require_gpu()
    dims = (13, 70, 45, 9)
    segs = [0, 1, 5, 9]
    flat, batch = _setup(333, dims, segs, seed=4, spread=1.0)
    out = _gpu_update(flat, batch, dims, segs, steps=1)
    _check_step(flat, np.zeros(flat.size), np.zeros(flat.size), 1, batch, out[0], dims, segs)


def test_ppo_update_is_deterministic():
    require_gpu()
    dims = (64, 256, 256, 26)
    flat, batch = _setup(2048, dims, seed=9)
    a = _gpu_update(flat, batch, dims, SEGS, steps=2)
    b = _gpu_update(flat, batch, dims, SEGS, steps=2)
    for x, y in zip(a, b):
        for k in ("params", "grad", "loss", "m", "v"):
            np.testing.assert_array_equal(x[k], y[k])
