"""Pins of the PPO-update oracle (oracle/ppo.py) against things other than itself: central finite
differences of its own objective for every parameter, closed forms of the objective, the clipped
region's zero gradient, and Adam's first steps written out by hand."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import ppo

DIMS = (5, 7, 6, 7)          # s, h1, h2, a
SEGS = [0, 4, 7]


def _net(rng, dims=DIMS, scale=0.7):
    s, h1, h2, a = dims
    return {k: rng.standard_normal(shp) * scale for k, shp in ppo.param_shapes(s, h1, h2, a).items()}


def _batch(rng, p, M=9, segs=SEGS, ratio_spread=0.1):
    X = rng.standard_normal((M, DIMS[0]))
    f = ppo.forward(p, X)
    acts = np.stack([rng.integers(segs[i], segs[i + 1], M) for i in range(len(segs) - 1)], axis=1)
    L = ppo.loss(p, dict(states=X, actions=acts, logp_old=np.zeros(M), adv=np.zeros(M), ret=np.zeros(M)), segs)
    logp_old = L["logp"] + rng.uniform(-ratio_spread, ratio_spread, M)
    return dict(states=X, actions=acts, logp_old=logp_old, adv=rng.standard_normal(M), ret=f["v"] + rng.standard_normal(M))


@pytest.mark.parametrize("seed,spread", [(0, 0.1), (1, 0.6), (2, 1.5)])
def test_gradients_match_central_differences(seed, spread):
    rng = np.random.default_rng(seed)
    p = _net(rng)
    b = _batch(rng, p, ratio_spread=spread)
    g, L = ppo.grads(p, b, SEGS)
    f = L["fwd"]
    # stay away from the kinks: no pre-activation near 0, no ratio near the clip edges
    assert np.abs(f["z1"]).min() > 1e-4 and np.abs(f["z2"]).min() > 1e-4
    assert np.abs(np.abs(L["ratio"] - 1) - 0.2).min() > 1e-4
    h = 1e-6
    for k in ppo.PARAM_ORDER:
        num = np.zeros_like(p[k])
        it = np.nditer(p[k], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            q = {kk: vv.copy() for kk, vv in p.items()}
            q[k][idx] += h
            up = ppo.loss(q, b, SEGS)["total"]
            q[k][idx] -= 2 * h
            dn = ppo.loss(q, b, SEGS)["total"]
            num[idx] = (up - dn) / (2 * h)
        np.testing.assert_allclose(g[k], num, rtol=1e-5, atol=1e-9, err_msg=k)


def test_objective_closed_forms():
    # zero weights: logits = 0 -> uniform segments; value = bv
    s, h1, h2, a = DIMS
    p = {k: np.zeros(shp) for k, shp in ppo.param_shapes(s, h1, h2, a).items()}
    p["bv"][0] = 0.5
    M = 6
    logp_u = -np.log(4) - np.log(3)
    b = dict(states=np.ones((M, s)), actions=np.tile([1, 5], (M, 1)), logp_old=np.full(M, logp_u),
             adv=np.arange(M, dtype=np.float64) - 2, ret=np.full(M, 2.5))
    L = ppo.loss(p, b, SEGS)
    np.testing.assert_allclose(L["ratio"], 1.0)
    assert L["clip"] == pytest.approx(-np.mean(b["adv"]))
    assert L["value"] == pytest.approx(4.0)                      # (0.5 - 2.5)^2
    assert L["entropy"] == pytest.approx(np.log(4) + np.log(3))
    assert L["total"] == pytest.approx(-0.5 + 0.5 * 4.0 - 0.01 * (np.log(4) + np.log(3)))


def test_clipped_rows_carry_no_policy_gradient():
    rng = np.random.default_rng(7)
    p = _net(rng)
    b = _batch(rng, p)
    L = ppo.loss(p, b, SEGS)
    # ratio = 2 with a positive advantage: min(2A, 1.2A) is the constant clipped term
    b2 = dict(b, logp_old=L["logp"] - np.log(2.0), adv=np.abs(b["adv"]) + 0.1)
    g, _ = ppo.grads(p, b2, SEGS, w_v=0.0, w_e=0.0)
    for k in ppo.PARAM_ORDER:
        assert np.all(g[k] == 0.0), k
    # with a negative advantage the unclipped term 2A is the minimum: the gradient flows
    b3 = dict(b2, adv=-b2["adv"])
    g, _ = ppo.grads(p, b3, SEGS, w_v=0.0, w_e=0.0)
    assert np.abs(g["wa"]).max() > 1e-6
    # the value head only sees the value loss, the trunk and actor head only the policy terms
    g, _ = ppo.grads(p, b, SEGS, w_v=0.0)
    assert np.all(g["wv"] == 0.0) and np.all(g["bv"] == 0.0)


def test_adam_first_steps_by_hand():
    p = np.array([1.0, -2.0, 0.5])
    g1 = np.array([0.1, -0.4, 0.0])
    m0 = np.zeros(3)
    p1, m1, v1 = ppo.adam(p, g1, m0, m0, 1, 1e-3)
    # step 1: mhat = g, vhat = g^2, so the step is lr * g / (|g| + eps)
    np.testing.assert_allclose(p1, p - 1e-3 * g1 / (np.abs(g1) + 1e-8), rtol=0, atol=1e-15)
    g2 = np.array([0.3, 0.2, 1.0])
    p2, m2, v2 = ppo.adam(p1, g2, m1, v1, 2, 1e-3)
    m_ref = 0.9 * 0.1 * g1 + 0.1 * g2
    v_ref = 0.999 * 0.001 * g1 ** 2 + 0.001 * g2 ** 2
    step = 1e-3 * (m_ref / 0.19) / (np.sqrt(v_ref / (1 - 0.999 ** 2)) + 1e-8)
    np.testing.assert_allclose(m2, m_ref, rtol=1e-15)
    np.testing.assert_allclose(p2, p1 - step, rtol=1e-13)


def test_learning_rates_per_head():
    lr = ppo.lr_vector(*DIMS)
    s, h1, h2, a = DIMS
    n_actor = h1 * s + h1 + h2 * h1 + h2 + a * h2 + a
    assert lr.size == n_actor + h2 + 1
    assert np.all(lr[:n_actor] == 3e-4) and np.all(lr[n_actor:] == 1e-3)


def test_pack_round_trip():
    rng = np.random.default_rng(3)
    p = _net(rng)
    q = ppo.unpack(ppo.pack(p), *DIMS)
    for k in ppo.PARAM_ORDER:
        np.testing.assert_array_equal(p[k], q[k])
