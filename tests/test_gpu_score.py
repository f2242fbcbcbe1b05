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


# ---- the binned path (ensembles of depth 9 or 10, and of depth 8 on rounds of at least 2^17
# statement rows; <= 256 features, <= 65,534 distinct thresholds per feature) and the fp32 walks
# that remain for the others ----
def _exact_leaves(ens):
    return {**ens, "leaf_value": (np.round(ens["leaf_value"] * 4096) / 4096).astype(np.float32)}


@pytest.mark.parametrize("depth,n_prog", [(9, 611), (10, 611), (10, 37), (9, 5)])
def test_binned_depths_exact(depth, n_prog):
    """The binned walk at both of its depths, 15 % missing values, a ragged last tile and rounds of
    fewer rows than one tile: bit-exact against the oracle."""
    cfg = get_config("tiny", exact=True).with_(depth=depth, n_trees=23, n_prog=n_prog, s_max=9, p_nan=0.15,
                                               name="binned-d%d-p%d" % (depth, n_prog))
    _check(cfg)


@pytest.mark.parametrize("n_prog,groups", [(611, 0), (5, 0), (900, 2), (900, 4)])
def test_binned_depth8_exact(n_prog, groups, monkeypatch):
    """Depth 8 on the binned walk (its slots are half a prefetch wide), forced below the row count
    from which it is taken by default, with tree groups: bit-exact against the oracle."""
    monkeypatch.setenv("HARL_SCORE_BINNED_MIN_ROWS", "0")
    if groups:
        monkeypatch.setenv("HARL_SCORE_TREE_GROUPS", str(groups))
    cfg = get_config("tiny", exact=True).with_(depth=8, n_trees=31, n_prog=n_prog, s_max=9, p_nan=0.15,
                                               name="binned-d8-p%d-g%d" % (n_prog, groups))
    _check(cfg)


@pytest.mark.parametrize("above", [True, False])
def test_depth8_route_by_round_size_exact(above, monkeypatch):
    """A depth-8 ensemble takes the binned walk from a row count on and the fp32 walk below it; both
    routes, on the same ensemble and batch, are bit-exact against the oracle."""
    cfg = get_config("tiny", exact=True).with_(depth=8, n_trees=29, n_prog=300, s_max=9, p_nan=0.1,
                                               name="route-d8")
    n_rows = gen_batch(cfg)["n_rows"]
    monkeypatch.setenv("HARL_SCORE_BINNED_MIN_ROWS", str(n_rows if above else n_rows + 1))
    _check(cfg)


def test_depth8_workspace_serves_smaller_rounds_exact(monkeypatch):
    """A workspace sized for a round that takes the binned walk serves a smaller round of the same
    depth-8 ensemble on the fp32 walk (and the other way round): both calls, on one workspace of the
    larger round's size, are bit-exact against the oracle."""
    require_gpu()
    import torch
    from paper_2211_11172_amd import harl
    cfg = get_config("tiny", exact=True).with_(depth=8, n_trees=27, n_prog=600, s_max=9, p_nan=0.1,
                                               name="ws-d8")
    ens, b = gen_ensemble(cfg), gen_batch(cfg)
    ptr_all = b["prog_ptr"]
    small = 150                                           # programs of the smaller round
    n_small, n_big = int(ptr_all[small]), int(ptr_all[-1])
    monkeypatch.setenv("HARL_SCORE_BINNED_MIN_ROWS", str(n_small + 1))   # big: binned, small: fp32
    E = harl.harl_ensemble_create(ens)
    try:
        ws_small = harl.harl_score_round_workspace_size(E, n_small, small)
        wsb = harl.harl_score_round_workspace_size(E, n_big, len(ptr_all) - 1)
        assert wsb >= ws_small
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        for n_prog in (len(ptr_all) - 1, small):
            ptr = ptr_all[: n_prog + 1]
            n_rows = int(ptr[-1])
            X = np.ascontiguousarray(b["features"][:, :n_rows])
            want = oracle.score_round(ens, X, ptr)
            Xd = torch.from_numpy(X).cuda()
            ptr_d = torch.from_numpy(np.ascontiguousarray(ptr, np.int32)).cuda()
            ps = torch.full((n_prog,), np.nan, dtype=torch.float32, device="cuda")
            harl.harl_score_round(E, Xd, X.shape[1], n_rows, ptr_d, n_prog, ps, None, ws, wsb)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(ps.cpu().numpy(), want["prog32"])
    finally:
        E.close()


def test_binned_depth8_irregular_trees(monkeypatch):
    """Early leaves (dummy splits below them) at depth 8 on the binned walk."""
    monkeypatch.setenv("HARL_SCORE_BINNED_MIN_ROWS", "0")
    rng = np.random.default_rng(29)
    cfg = mini_config(p_nan=0.1, n_features=12, n_prog=400, s_max=9)
    b = gen_batch(cfg)
    pool = np.unique(b["features"][~np.isnan(b["features"])])
    ens = _irregular_ensemble(rng, n_trees=21, n_features=12, max_depth=8, thr_pool=pool)

    def depth(n):
        return 0 if ens["feature"][n] < 0 else 1 + max(depth(ens["left"][n]), depth(ens["right"][n]))
    assert max(depth(r) for r in ens["root"]) == 8
    _check(cfg, ens=_exact_leaves(ens), b=b, exact=True)


@pytest.mark.parametrize("groups", [2, 4, 8])
def test_binned_tree_groups_exact(groups, monkeypatch):
    monkeypatch.setenv("HARL_SCORE_TREE_GROUPS", str(groups))
    cfg = get_config("tiny", exact=True).with_(depth=10, n_trees=45, n_prog=900, p_nan=0.1,
                                               name="binned-groups%d" % groups)
    _check(cfg)


def test_binned_irregular_trees():
    """Trees with early leaves (packed with dummy splits below them), depth 10."""
    rng = np.random.default_rng(19)
    cfg = mini_config(p_nan=0.1, n_features=12, n_prog=400, s_max=9)
    b = gen_batch(cfg)
    pool = np.unique(b["features"][~np.isnan(b["features"])])
    ens = _irregular_ensemble(rng, n_trees=19, n_features=12, max_depth=10, thr_pool=pool)

    def depth(n):
        return 0 if ens["feature"][n] < 0 else 1 + max(depth(ens["left"][n]), depth(ens["right"][n]))
    assert max(depth(r) for r in ens["root"]) == 10
    _check(cfg, ens=_exact_leaves(ens), b=b, exact=True)


def test_binned_special_thresholds_and_values():
    """Thresholds NaN, +-inf, -0.0, +0.0 and denormals; feature values equal to thresholds, their
    fp32 neighbours, +-inf, +-0 and NaN: the codes order every value exactly as the fp32 compare."""
    rng = np.random.default_rng(5)
    cfg = get_config("tiny", exact=True).with_(depth=9, n_trees=40, n_prog=400, s_max=8, p_nan=0.1,
                                               n_features=24, name="binned-special")
    ens = gen_ensemble(cfg)
    internal = np.nonzero(ens["feature"] >= 0)[0]
    special = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, 1e-45, -1e-45, 1e-40], np.float32)
    pick = rng.choice(internal, size=internal.size // 4, replace=False)
    ens["threshold"] = ens["threshold"].copy()
    ens["threshold"][pick] = rng.choice(special, size=pick.size)
    b = gen_batch(cfg)
    X = b["features"].copy()
    n = b["n_rows"]
    vals = np.concatenate([special, np.nextafter(special[1:], np.float32(0))]).astype(np.float32)
    for r in range(0, n, 2):
        for nd in rng.choice(internal, 6, replace=False):
            f, th = ens["feature"][nd], np.float32(ens["threshold"][nd])
            X[f, r] = rng.choice([th, np.nextafter(th, np.float32(-np.inf)), np.nextafter(th, np.float32(np.inf)),
                                  rng.choice(vals)])
    b["features"] = X
    _check(cfg, ens=_exact_leaves(ens), b=b)


@pytest.mark.parametrize("n_features", [193, 256])
def test_binned_wide_tiles_staged_directly(n_features):
    """Tiles of more than 192 features are staged without the register prefetch; 256 is the widest
    binned ensemble."""
    cfg = get_config("tiny", exact=True).with_(depth=10, n_trees=37, n_prog=500, s_max=12, p_nan=0.1,
                                               n_features=n_features, name="binned-f%d" % n_features)
    _check(cfg)


@pytest.mark.parametrize("aligned", [True, False])
def test_binned_whole_tile_passes_exact(aligned):
    """More than 16 whole tiles of rows: the bin kernel's unchecked passes (16 tiles each, features
    read one pass ahead) and its bounds-checked rest, with 16-byte feature loads when the leading
    dimension is a multiple of 4 floats and element loads when it is not."""
    cfg = get_config("tiny", exact=True).with_(depth=10, n_trees=23, n_prog=3000, s_max=9, p_nan=0.1,
                                               name="binned-passes-%s" % ("vec" if aligned else "scalar"))
    n_rows = gen_batch(cfg)["n_rows"]
    assert n_rows > 3 * 16 * 256 and n_rows % 256 != 0
    pad = (-n_rows) % 4 if aligned else (1 if (n_rows + 1) % 4 else 2)
    b = gen_batch(cfg, ld_pad=pad)
    assert (b["ld"] % 4 == 0) == aligned
    _check(cfg, b=b)


def test_binned_probe_counts_and_global_search():
    """Features searched with different probe counts (the bin kernel is specialised for the most
    common one, the others take its general loop), a feature with one distinct threshold, one that
    no node splits on, and one with more thresholds than the LDS table holds (searched in global
    memory)."""
    rng = np.random.default_rng(23)
    cfg = get_config("tiny", exact=True).with_(depth=10, n_trees=60, n_prog=700, s_max=8, p_nan=0.1,
                                               n_features=8, name="binned-probes")
    ens = gen_ensemble(cfg)
    b = gen_batch(cfg)
    internal = np.nonzero(ens["feature"] >= 0)[0]
    feat = ens["feature"].copy()
    thr = ens["threshold"].copy()
    feat[feat == 7] = 6                                   # feature 7: no split
    on0 = internal[feat[internal] == 0]
    many = np.unique(np.float32(10.0) ** rng.uniform(-3, 3, size=4 * on0.size).astype(np.float32))
    on0 = np.concatenate([on0, internal[feat[internal] == 5][: 22000 - on0.size]])
    feat[on0] = 0                                         # feature 0: > 10,240 distinct thresholds
    thr[on0] = rng.permutation(many)[: on0.size]
    thr[internal[feat[internal] == 1]] = np.float32(0.5)  # feature 1: one threshold
    on2 = internal[feat[internal] == 2]
    thr[on2] = rng.choice(np.float32(10.0) ** np.linspace(-2, 2, 40).astype(np.float32), size=on2.size)
    ens = _exact_leaves({**ens, "feature": feat, "threshold": thr})
    assert np.unique(thr[internal[feat[internal] == 0]]).size > 10240
    _check(cfg, ens=ens, b=b)


@pytest.mark.parametrize("depth", [8, 10])
def test_fp32_walk_wide_ensembles(depth):
    """More than 256 features: the fp32 walk (16-bit feature codes) scores the round."""
    cfg = get_config("tiny", exact=True).with_(depth=depth, n_trees=21, n_prog=300, s_max=8, p_nan=0.1,
                                               n_features=300, name="fp32-wide-d%d" % depth)
    _check(cfg)


def test_fp32_walk_many_distinct_thresholds():
    """One feature split at more than 65,534 distinct thresholds does not fit 16-bit codes: the fp32
    walk scores the round, bit-exact."""
    rng = np.random.default_rng(11)
    cfg = get_config("tiny", exact=True).with_(depth=10, n_trees=70, n_prog=200, s_max=6, p_nan=0.1,
                                               n_features=8, name="fp32-many-thr")
    ens = gen_ensemble(cfg)
    internal = np.nonzero(ens["feature"] >= 0)[0]
    ens["feature"] = ens["feature"].copy()
    ens["threshold"] = ens["threshold"].copy()
    ens["feature"][internal] = 0
    thr = np.unique(np.float32(10.0) ** rng.uniform(-3, 3, size=internal.size * 2).astype(np.float32))
    assert thr.size > 65534
    ens["threshold"][internal] = rng.permutation(thr)[:internal.size]
    assert np.unique(ens["threshold"][internal]).size > 65534
    _check(cfg, ens=ens)
