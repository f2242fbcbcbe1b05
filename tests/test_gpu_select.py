"""GPU parity of harl_policy_select (one action per modification type, Section 4.3 and Appendix
A.1; sampled as in PPO rollouts, Section 6.1) against the oracle.

Bars: greedy actions bit-exact on the same fp32 logits; sampled actions equal to the oracle's on the
same logits (the noise and the decision are fp64 on both sides, so only two candidates within a
few ulps of fp64 log of each other could differ); probabilities within 1e-6 absolute and
log-probabilities within 1e-5 (1 + |logp|) of the fp64 oracle."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_policy, gen_states, get_config
from tests.gpu_util import gpu_policy, log, require_gpu

pytestmark = pytest.mark.gpu

SEGS_26 = [0, 17, 20, 23, 26]   # num_iters = 4: 4 x 4 + 1 tile-size actions, then 3 types of 3


def gpu_select(z, segs, sample=False, seed=0, counter=0):
    import torch
    from paper_2211_11172_amd import harl
    B, a = z.shape
    n_seg = len(segs) - 1
    zd = torch.from_numpy(np.ascontiguousarray(z, np.float32)).cuda()
    act = torch.full((max(B, 1), n_seg), -5, dtype=torch.int32, device="cuda")
    lp = torch.full((max(B, 1), n_seg), np.nan, dtype=torch.float32, device="cuda")
    pr = torch.full((max(B, 1), a), np.nan, dtype=torch.float32, device="cuda")
    harl.harl_policy_select(zd, B, a, segs, harl.HARL_SELECT_SAMPLE if sample else 0, seed, counter, act, lp, pr)
    torch.cuda.synchronize()
    return act.cpu().numpy()[:B], lp.cpu().numpy()[:B], pr.cpu().numpy()[:B]


def _check(z, segs, sample, seed=0, counter=0):
    got_a, got_lp, got_p = gpu_select(z, segs, sample, seed, counter)
    want = oracle.policy_select(z, np.array(segs, np.int32), sample=sample, seed=seed, counter=counter)
    np.testing.assert_array_equal(got_a, want["action"])
    finite = np.isfinite(want["probs"])
    np.testing.assert_allclose(got_p[finite], want["probs"][finite], rtol=0, atol=1e-6)
    ok = np.isfinite(want["logp"])
    err = np.abs(got_lp[ok] - want["logp"][ok])
    assert np.all(err <= 1e-5 * (1 + np.abs(want["logp"][ok]))), float(err.max())
    return got_a


@pytest.mark.parametrize("sample", [False, True])
@pytest.mark.parametrize("B", [1, 63, 64, 4096, 65537])
def test_select_random_logits(B, sample):
    require_gpu()
    rng = np.random.default_rng(B)
    z = (rng.standard_normal((B, 26)) * 2).astype(np.float32)
    log("policy select parity: B=%d sample=%s" % (B, sample))
    _check(z, SEGS_26, sample, seed=0xDEADBEEF12345, counter=B)


def test_select_ties_nan_inf_greedy_and_sampled():
    require_gpu()
    rng = np.random.default_rng(3)
    z = rng.integers(-2, 2, (3000, 26)).astype(np.float32)
    z[::5, 2] = np.nan
    z[7, 17:20] = -np.inf
    z[8, 20:23] = np.nan
    z[9, 0:17] = np.inf
    a = _check(z, SEGS_26, False)
    assert a[7, 1] == 17 and a[8, 2] == 20 and a[9, 0] == 0
    _check(z, SEGS_26, True, seed=5, counter=9)


@pytest.mark.parametrize("segs", [[0, 1], [0, 3], [0, 127], [0, 1, 2, 3, 64, 127], list(range(0, 33))])
def test_select_segment_layouts(segs):
    require_gpu()
    a = segs[-1]
    rng = np.random.default_rng(a)
    z = rng.standard_normal((777, a)).astype(np.float32)
    for sample in (False, True):
        _check(z, segs, sample, seed=a, counter=1 << 33)


def test_select_on_policy_logits_and_counter_streams():
    """A rollout step: the actor's logits from harl_policy_step (fp32 standard policy with a
    26-action head), then per-type actions -- greedy, and sampled at two counters."""
    require_gpu()
    cfg = get_config("standard").with_(pol_a=26)
    pol = gen_policy(cfg)
    st = gen_states(cfg)
    out = gpu_policy(pol, st, probs=False, logits=True)
    z = out["logits"]
    _check(z, SEGS_26, False)
    a0 = _check(z, SEGS_26, True, seed=42, counter=0)
    a1 = _check(z, SEGS_26, True, seed=42, counter=1)
    assert (a0 != a1).mean() > 0.2
    # the empirical distribution of many draws of one state follows its segment softmax
    zz = np.repeat(z[:1], 50000, axis=0)
    got, _, probs = gpu_select(zz, SEGS_26, True, seed=99, counter=7)
    for s in range(4):
        lo, hi = SEGS_26[s], SEGS_26[s + 1]
        freq = np.bincount(got[:, s] - lo, minlength=hi - lo) / got.shape[0]
        p = probs[0, lo:hi].astype(np.float64)
        assert np.all(np.abs(freq - p) < 5 * np.sqrt(p * (1 - p) / got.shape[0]) + 1e-4)
