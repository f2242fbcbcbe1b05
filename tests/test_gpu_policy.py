"""GPU parity of harl_policy_step (actor pi_theta(M|S) and critic V(S), Algorithm 1, Eq. 6)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_policy, gen_states, get_config, mini_config
from tests.gpu_util import assert_close_scaled, gpu_policy, log, require_gpu

pytestmark = pytest.mark.gpu


def _check(cfg, B=None):
    require_gpu()
    pol = gen_policy(cfg)
    st = gen_states(cfg, n=B)
    log("policy parity: %s dtype=%s %d-%d-%d->%d B=%d exact=%s" % (
        cfg.name, cfg.pol_dtype, cfg.pol_s, cfg.pol_h1, cfg.pol_h2, cfg.pol_a, st.shape[0], cfg.exact))
    want = oracle.policy_step(pol, st)
    got = gpu_policy(pol, st)
    lg = got["logits"]
    # the GPU action is the lowest-index argmax of the GPU's own logits, bit-exactly
    np.testing.assert_array_equal(got["action"], np.argmax(lg, axis=1))
    if cfg.exact:
        np.testing.assert_array_equal(lg, want["logits"].astype(np.float32))
        np.testing.assert_array_equal(got["value"], want["value"].astype(np.float32))
        np.testing.assert_array_equal(got["action"], want["action"])
        return got, want
    rtol = 2e-2 if cfg.pol_dtype == "bf16" else 1e-5
    assert_close_scaled(lg, want["logits"], want["logit_scale"], rtol, "logits")
    assert_close_scaled(got["value"], want["value"], want["value_scale"], rtol, "value")
    ptol = 2e-2 if cfg.pol_dtype == "bf16" else 1e-5
    assert np.abs(got["probs"] - want["probs"]).max() <= ptol
    # end-to-end argmax: may differ only where the oracle's top two lie within the tolerance band
    diff = np.nonzero(got["action"] != want["action"])[0]
    for i in diff:
        a, b = got["action"][i], want["action"][i]
        band = rtol * (want["logit_scale"][i, a] + want["logit_scale"][i, b])
        assert want["logits"][i, b] - want["logits"][i, a] <= band, "argmax flip beyond the near-tie band"
    log("  argmax near-tie flips: %d of %d" % (diff.size, st.shape[0]))
    return got, want


def test_tiny_fp32():
    _check(get_config("tiny"))


def test_tiny_fp32_exact():
    _check(get_config("tiny", exact=True))


def test_policy_heavy_bf16_exact_small_batch():
    _check(get_config("policy_heavy", exact=True), B=200)


def test_policy_heavy_bf16_small_batch():
    _check(get_config("policy_heavy"), B=333)


def test_bf16_large_batch_path():
    # from 16,384 states bf16 policies run on the large-batch kernel (k_policy_x32: 128 states per
    # workgroup, 32x32x16 MFMA tiles, weights streamed into LDS in chunks); 37 states in a ragged
    # last workgroup
    _check(get_config("policy_heavy", exact=True), B=16384 + 37)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_odd_sizes(dtype):
    cfg = mini_config(pol_dtype=dtype, pol_s=19, pol_h1=50, pol_h2=70, pol_a=13, n_prog=45)
    _check(cfg)
    _check(cfg.with_(exact=True))


def test_single_action_and_wide_head():
    _check(mini_config(pol_a=1, n_prog=20))
    _check(mini_config(pol_a=100, pol_h2=64, n_prog=40))


# Batches of 16384 states and more of a bf16 policy take the 128-states-per-workgroup kernel
# (h1 kept in registers, weights streamed through LDS): its shape limits and ragged edges.
_LARGE = 16384


@pytest.mark.parametrize("exact", [True, False])
def test_large_batch_odd_shapes(exact):
    # h1 <= 512 variant, h2 not a multiple of 32, 41 head rows, a ragged last workgroup
    cfg = mini_config(pol_dtype="bf16", pol_s=64, pol_h1=300, pol_h2=100, pol_a=40, exact=exact)
    _check(cfg, B=_LARGE + 77)


@pytest.mark.parametrize("a", [95, 127])
def test_large_batch_wide_heads(a):
    # 95 actions + value fill the large-batch kernel's 3 head tiles of 32 rows; 127 are beyond its
    # limit and take the general kernel.  h1 of 1000 units (1024-unit variant)
    cfg = mini_config(pol_dtype="bf16", pol_s=128, pol_h1=1000, pol_h2=70, pol_a=a, exact=True)
    _check(cfg, B=_LARGE + 3)


@pytest.mark.parametrize("exact", [True, False])
def test_large_fp32_batch(exact):
    # fp32 batches of 16384 states and more share weight fragments between two state groups
    cfg = mini_config(pol_s=64, pol_h1=256, pol_h2=200, pol_a=24, exact=exact)
    _check(cfg, B=_LARGE + 45)


def test_large_batch_policy_heavy_values():
    # the policy-heavy network with its own (non-integer) weights and states
    _check(get_config("policy_heavy"), B=_LARGE + 129)


@pytest.mark.parametrize("dtype,a,B", [
    ("f32", 6, 333),              # 16 head rows: four states per wave pass
    ("f32", 40, 333),             # 48 rows, five head tiles: one state per pass, a second 64-row chunk
    ("f32", 63, 333),             # 64 rows: the value in the last row of the first chunk
    ("bf16", 40, 200),            # the same on the bf16 general kernel
    ("f32", 60, _LARGE + 45),     # 32-state workgroups with five head tiles
    ("f32", 10, _LARGE + 45),     # 32-state workgroups, four states per pass
])
def test_epilogue_widths(dtype, a, B):
    # the general kernel's epilogue takes 64 / W states per wave pass, W = 16, 32 or 64 lanes per
    # state: every width, with one and two row chunks, on 16- and 32-state workgroups
    for exact in (True, False):
        _check(mini_config(pol_dtype=dtype, pol_s=64, pol_h1=256, pol_h2=200, pol_a=a, exact=exact), B=B)
