"""The seeded input generator: determinism and the distributions the workloads call for."""
from __future__ import annotations

import numpy as np
import pytest

from synth import CONFIGS, gen_batch, gen_ensemble, gen_policy, gen_states, get_config, mini_config
from synth.configs import CONFIG_ORDER
from synth.gen import bf16_bits_from_f32, digest, f32_from_bf16_bits, gen_features, gen_prog_ptr


def test_same_seed_same_bytes_and_streams_independent():
    cfg = get_config("tiny")
    a, b = gen_batch(cfg), gen_batch(cfg)
    assert digest(a["features"], a["prog_ptr"], a["states"]) == digest(b["features"], b["prog_ptr"], b["states"])
    e1, e2 = gen_ensemble(cfg), gen_ensemble(cfg)
    assert digest(*[e1[k] for k in ("feature", "threshold", "leaf_value")]) == \
        digest(*[e2[k] for k in ("feature", "threshold", "leaf_value")])
    # other batches and the exact variant draw different values
    c = gen_batch(cfg.with_(n_batches=2), batch=1)
    assert digest(c["prog_ptr"]) != digest(a["prog_ptr"])
    assert digest(gen_batch(cfg.with_(exact=True))["states"]) != digest(a["states"])


def test_feature_distribution():
    cfg = get_config("tiny").with_(p_nan=0.1)
    X = gen_features(cfg, 20000)
    nan = np.isnan(X)
    zero = X == 0
    assert abs(nan.mean() - 0.1) < 0.005 and abs(zero.mean() - 0.4) < 0.005
    v = X[~nan & ~zero]
    assert v.min() >= np.float32(1e-3) * (1 - 1e-6) and v.max() <= np.float32(1e3)
    # log-uniform: log10 of the non-zero values is ~U[-3, 3)
    lg = np.log10(v.astype(np.float64))
    assert abs(lg.mean()) < 0.05 and abs(lg.std() - 6 / np.sqrt(12)) < 0.05


def test_padding_is_nan_and_ld():
    cfg = mini_config()
    b = gen_batch(cfg, ld_pad=13)
    assert b["ld"] == b["n_rows"] + 13
    assert np.isnan(b["features"][:, b["n_rows"]:]).all()


def test_statement_counts():
    for name in CONFIG_ORDER[:3]:
        cfg = CONFIGS[name]
        ptr = gen_prog_ptr(cfg)
        c = np.diff(ptr)
        assert ptr[0] == 0 and c.min() >= 1 and c.max() <= cfg.s_max
        assert c.min() == 1 and c.max() == cfg.s_max       # both ends reached at these sizes
        assert abs(c.mean() - (1 + cfg.s_max) / 2) < 0.1 * cfg.s_max


def test_ensemble_shape_and_thresholds():
    cfg = get_config("tiny")
    e = gen_ensemble(cfg)
    T, D = cfg.n_trees, cfg.depth
    M = 2 ** (D + 1) - 1
    assert e["feature"].size == T * M
    internal = e["feature"] >= 0
    assert internal.sum() == T * (2 ** D - 1)
    assert (e["feature"][internal] < cfg.n_features).all()
    # about 40% of thresholds are 0.0 (calibration values are 40% zeros); others in [1e-3, 1e3)
    thr = e["threshold"][internal]
    assert 0.3 < (thr == 0).mean() < 0.5
    assert (thr[thr != 0] >= np.float32(1e-3) * (1 - 1e-6)).all()
    leaves = e["leaf_value"][~internal]
    assert abs(leaves.std() - 0.1) < 0.01
    ex = gen_ensemble(cfg.with_(exact=True))
    lv = ex["leaf_value"][ex["feature"] < 0].astype(np.float64) * 4096
    assert (lv == np.round(lv)).all() and np.abs(lv).max() <= 64


def test_policy_shapes_and_init():
    cfg = get_config("policy_heavy")
    p = gen_policy(cfg)
    assert p["w1"].dtype == np.uint16 and p["w1"].shape == (1024, 128)
    assert p["wa"].shape == (64, 1024) and p["wv"].shape == (1, 1024)
    w2 = f32_from_bf16_bits(p["w2"])
    a = np.sqrt(6 / 2048)
    assert np.abs(w2).max() <= a * 1.01 and abs(w2.std() - a / np.sqrt(3)) < 0.01 * a
    assert np.abs(p["b2"]).max() <= 1 / np.sqrt(1024)
    st = gen_states(cfg, n=4096)
    assert st.dtype == np.uint16 and st.shape == (4096, 128)
    f = f32_from_bf16_bits(st)
    assert abs(f.mean()) < 0.02 and abs(f.std() - 1) < 0.02


def test_bf16_store_round_trip():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 0.0, np.inf], np.float32)
    y = f32_from_bf16_bits(bf16_bits_from_f32(x))
    assert y.tolist() == [1.0, 1.0, 1 + 2 ** -6, -2.5, 0.0, np.inf]


@pytest.mark.parametrize("name", CONFIG_ORDER)
def test_named_configs(name):
    cfg = get_config(name)
    assert cfg.n_features == 164 and cfg.top_k <= cfg.n_candidates
    assert get_config(name + "-exact").exact
