"""GPU parity of harl_score_round (cost-model scores C(S'), Algorithm 1) against the oracle."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_batch, gen_ensemble, get_config, mini_config
from tests.gpu_util import assert_close_scaled, gpu_score, log, require_gpu
from tests.test_oracle_pins import _irregular_ensemble

pytestmark = pytest.mark.gpu


def _check(cfg, ens=None, b=None, exact=None, ld_pad=0):
    require_gpu()
    ens = gen_ensemble(cfg) if ens is None else ens
    b = gen_batch(cfg, ld_pad=ld_pad) if b is None else b
    log("score parity: %s trees=%d depth=%d rows=%d progs=%d nan=%.2f" % (
        cfg.name, int(ens["n_trees"]), cfg.depth, b["n_rows"], len(b["prog_ptr"]) - 1, cfg.p_nan))
    want = oracle.score_round(ens, b["features"], b["prog_ptr"])
    ps, ss = gpu_score(ens, b["features"], b["prog_ptr"])
    exact = cfg.exact if exact is None else exact
    if exact:
        np.testing.assert_array_equal(ps, want["prog32"])
        np.testing.assert_array_equal(ss, want["stmt32"])
    else:
        assert_close_scaled(ps, want["prog"], want["scale"], 1e-5, "program scores")
        # statement scale: sum of |leaf| over trees of that row (bounded by its program's scale)
        row_prog = np.repeat(np.arange(len(b["prog_ptr"]) - 1), np.diff(b["prog_ptr"]))
        assert_close_scaled(ss, want["stmt"], want["scale"][row_prog], 1e-5, "statement scores")
    return ps, want


def test_tiny_config():
    _check(get_config("tiny"))


def test_tiny_exact_bitwise():
    _check(get_config("tiny", exact=True))


@pytest.mark.parametrize("depth", [1, 2, 5, 7, 9, 11])
def test_depths_ragged_with_missing(depth):
    cfg = mini_config(depth=depth, n_trees=37, n_features=20, n_prog=157, s_max=7, p_nan=0.15)
    _check(cfg)


@pytest.mark.parametrize("depth", [6, 8, 10])
def test_depths_exact_many_tiles(depth):
    cfg = get_config("tiny", exact=True).with_(depth=depth, n_trees=29, n_prog=700, p_nan=0.1, name="exact-d%d" % depth)
    _check(cfg)


@pytest.mark.parametrize("groups", [2, 4, 8])
def test_tree_groups_exact(groups, monkeypatch):
    # the ensemble split into tree groups walked by different XCDs (the split large ensembles get
    # so that each group stays L2-resident), forced here on a small ensemble with a ragged tree
    # count; exact leaves make every grouping bit-identical to the oracle
    monkeypatch.setenv("HARL_SCORE_TREE_GROUPS", str(groups))
    cfg = get_config("tiny", exact=True).with_(depth=8, n_trees=45, n_prog=900, p_nan=0.1, name="groups%d" % groups)
    _check(cfg)


@pytest.mark.parametrize("trees_depth", [(16, 1), (4, 4), (2, 8), (1, 5)])
def test_shallow_ensembles_many_tiles(trees_depth):
    """Few, shallow trees over many row tiles: every slice spans many tiles (the ingest-bound
    shape); 164 features, 10 % missing values."""
    n_trees, depth = trees_depth
    cfg = get_config("tiny").with_(n_trees=n_trees, depth=depth, n_prog=2500, s_max=16, p_nan=0.1,
                                   name="shallow-%dx%d" % trees_depth)
    _check(cfg)


def test_standard_config_exact():
    _check(get_config("standard", exact=True))


def test_irregular_trees():
    rng = np.random.default_rng(9)
    cfg = mini_config(p_nan=0.1, n_features=12, n_prog=300, s_max=9)
    b = gen_batch(cfg)
    pool = np.unique(b["features"][~np.isnan(b["features"])])
    ens = _irregular_ensemble(rng, n_trees=23, n_features=12, max_depth=7, thr_pool=pool)
    _check(cfg, ens=ens, b=b)


def test_padded_ld_and_base_score():
    cfg = mini_config(depth=4, n_trees=9, n_prog=90)
    ens = gen_ensemble(cfg)
    ens["base_score"] = 0.375
    _check(cfg, ens=ens, ld_pad=20)     # features [F][n_rows+20]: padding columns hold NaN


def test_empty_programs_and_zero_rows():
    require_gpu()
    cfg = mini_config(depth=3, n_trees=5)
    ens = gen_ensemble(cfg)
    ens["base_score"] = 0.25
    b = gen_batch(cfg)
    ptr = np.array([0, 0, 3, 3, 5, 5], np.int32)
    X = np.ascontiguousarray(b["features"][:, :8])
    ps, _ = gpu_score(ens, X, ptr)
    want = oracle.score_round(ens, X, ptr)
    assert_close_scaled(ps, want["prog"], want["scale"], 1e-5, "empty programs")
    assert ps[0] == np.float32(0.25) and ps[2] == np.float32(0.25) and ps[4] == np.float32(0.25)
    X0 = np.zeros((cfg.n_features, 4), np.float32)
    ps, _ = gpu_score(ens, X0, np.zeros(4, np.int32), want_stmt=False)
    assert (ps == np.float32(0.25)).all()


def test_threshold_ties_planted():
    cfg = mini_config(depth=6, n_trees=16, n_features=10, n_prog=120)
    ens = gen_ensemble(cfg)
    b = gen_batch(cfg)
    X = b["features"].copy()
    rng = np.random.default_rng(1)
    internal = np.nonzero(ens["feature"] >= 0)[0]
    for r in range(b["n_rows"]):
        for n in rng.choice(internal, 5, replace=False):
            th = ens["threshold"][n]
            X[ens["feature"][n], r] = rng.choice([th, np.nextafter(th, np.float32(-np.inf)), np.float32(-0.0)])
    b["features"] = X
    _check(cfg.with_(exact=True), ens={**ens, "leaf_value": (np.round(ens["leaf_value"] * 4096) / 4096).astype(np.float32)}, b=b)


def test_deterministic_repeat():
    require_gpu()
    cfg = get_config("tiny")
    ens, b = gen_ensemble(cfg), gen_batch(cfg)
    a1, s1 = gpu_score(ens, b["features"], b["prog_ptr"])
    a2, s2 = gpu_score(ens, b["features"], b["prog_ptr"])
    assert a1.tobytes() == a2.tobytes() and s1.tobytes() == s2.tobytes()
