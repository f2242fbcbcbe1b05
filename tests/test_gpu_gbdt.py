"""GPU parity of the cost-model refit (Algorithm 1: the cost model is trained on the measured
top-K; Section 6.1 and Appendix A.1: XGBoost with Ansor's settings) against the oracle.

Bar: bit-exact.  Binning is integer work; the tree is a sequence of decisions taken on exact
64-bit integer sums and on fp64 gains evaluated by the same expressions in the same order on both
sides (contraction off), and leaves and margins are single roundings of identical fp64 / fp32
operations, so every node field, every leaf value and every margin must match bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_measured, get_config, mini_config
from tests.gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

FIELDS = ("feature", "threshold", "left", "right", "default_left", "leaf_value")


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_groups(bins_rows, F, ld_rows):
    """Row-major bins [N][>= F] (the oracle's layout) -> the library's planes [ceil(F/8)][ld_rows][8]
    (a relayout only)."""
    N = bins_rows.shape[0]
    n_fg = (F + 7) // 8
    padded = np.zeros((N, n_fg * 8), np.uint8)
    padded[:, :F] = bins_rows[:, :F]
    out = np.zeros((n_fg, ld_rows, 8), np.uint8)
    out[:, :N, :] = padded.reshape(N, n_fg, 8).transpose(1, 0, 2)
    return out


def from_groups(planes, F, N):
    n_fg = planes.shape[0]
    return planes[:, :N, :].transpose(1, 0, 2).reshape(N, n_fg * 8)[:, :F]


def gpu_bin(X, n_rows, cuts, n_cuts, ld_rows):
    """harl_gbdt_bin; returns the planes [ceil(F/8)][ld_rows][8]."""
    import torch
    from paper_2211_11172_amd import harl
    F = X.shape[0]
    n_fg = (F + 7) // 8
    bins = torch.full((n_fg, max(ld_rows, 1), 8), 0xAB, dtype=torch.uint8, device="cuda")
    harl.harl_gbdt_bin(_dev(X), X.shape[1], F, n_rows, _dev(cuts), cuts.shape[1], _dev(n_cuts), bins, ld_rows)
    torch.cuda.synchronize()
    return bins.cpu().numpy()


def gpu_rounds(bins, F, cuts, n_cuts, prog_ptr, label, weight, margin, rounds=1, **kw):
    """Run `rounds` boosting rounds back to back on the device (margins carried on the device);
    returns the list of trees (numpy node arrays) and the final margins."""
    import torch
    from paper_2211_11172_amd import harl
    prm = harl.gbdt_params(**kw)
    N = bins.shape[0]
    ld = N + 3  # ragged plane stride
    P = len(prog_ptr) - 1
    n_nodes = (1 << (prm.max_depth + 1)) - 1
    d_bins = _dev(to_groups(bins, F, ld))
    d_margin = _dev(np.asarray(margin, np.float32)) if N else torch.zeros(1, dtype=torch.float32, device="cuda")
    d_label = _dev(np.asarray(label, np.float32)) if P else torch.zeros(1, device="cuda")
    d_weight = _dev(np.asarray(weight, np.float32)) if P else torch.zeros(1, device="cuda")
    wsb = harl.harl_gbdt_round_workspace_size(prm, F, N, P)
    assert wsb > 0
    ws = torch.full((wsb,), 0x5A, dtype=torch.uint8, device="cuda")  # stale contents must not matter
    trees = []
    for _ in range(rounds):
        out = dict(feature=torch.full((n_nodes,), 77, dtype=torch.int32, device="cuda"),
                   threshold=torch.full((n_nodes,), np.nan, dtype=torch.float32, device="cuda"),
                   left=torch.full((n_nodes,), 77, dtype=torch.int32, device="cuda"),
                   right=torch.full((n_nodes,), 77, dtype=torch.int32, device="cuda"),
                   default_left=torch.full((n_nodes,), 7, dtype=torch.uint8, device="cuda"),
                   leaf_value=torch.full((n_nodes,), np.nan, dtype=torch.float32, device="cuda"))
        harl.harl_gbdt_round(prm, d_bins, ld, F, N, _dev(cuts), cuts.shape[1], _dev(n_cuts), _dev(prog_ptr), P,
                             d_label, d_weight, d_margin, out["feature"], out["threshold"], out["left"], out["right"],
                             out["default_left"], out["leaf_value"], ws, wsb)
        torch.cuda.synchronize()
        trees.append({k: v.cpu().numpy() for k, v in out.items()})
    return trees, d_margin.cpu().numpy()[:N]


def oracle_rounds(bins, F, cuts, n_cuts, prog_ptr, label, weight, margin, rounds=1, **kw):
    trees, m = [], np.asarray(margin, np.float32)
    for _ in range(rounds):
        r = oracle.gbdt_round(bins, F, cuts, n_cuts, prog_ptr, label, weight, m, **kw)
        m = r["margin"]
        trees.append(r)
    return trees, m


def assert_trees_equal(got, want, what):
    for i, (g, w) in enumerate(zip(got, want)):
        for f in FIELDS:
            gv, wv = np.asarray(g[f]), np.asarray(w[f])
            if gv.dtype == np.float32:
                gv, wv = gv.view(np.uint32), wv.astype(np.float32).view(np.uint32)
            bad = np.nonzero(gv != wv)[0]
            assert bad.size == 0, "%s round %d: %s differs at nodes %s (gpu %s, oracle %s)" % (
                what, i, f, bad[:6], np.asarray(g[f])[bad[:6]], np.asarray(w[f])[bad[:6]])


def _case(cfg, n_cuts=254, p_nan=None):
    if p_nan is not None:
        cfg = cfg.with_(p_nan=p_nan)
    return gen_measured(cfg, n_cuts=n_cuts)


def _ld(F):
    return (F + 7) // 8 * 8


@pytest.mark.parametrize("F,n_cuts,p_nan", [(164, 254, 0.1), (13, 7, 0.3), (1, 3, 0.0), (24, 254, 0.0)])
def test_bins_bit_exact(F, n_cuts, p_nan):
    require_gpu()
    cfg = mini_config(n_prog=700, s_max=9, n_features=F)
    m = _case(cfg, n_cuts, p_nan)
    X = m["features"]
    # values equal to cut points, infinities and a ragged padded ld
    X[:, ::11] = np.where(m["n_cuts"][:, None] > 0, m["cuts"][:, :1], X[:, ::11])
    X[:, 5] = np.inf
    X[:, 6] = -np.inf
    Xp = np.full((F, m["n_rows"] + 5), np.nan, np.float32)
    Xp[:, :m["n_rows"]] = X
    ldr = m["n_rows"] + 9
    log("gbdt bin parity: F=%d n_cuts=%d rows=%d" % (F, n_cuts, m["n_rows"]))
    planes = gpu_bin(Xp, m["n_rows"], m["cuts"], m["n_cuts"], ldr)
    want = oracle.gbdt_bin(Xp, m["n_rows"], m["cuts"], m["n_cuts"], _ld(F))
    np.testing.assert_array_equal(from_groups(planes, F, m["n_rows"]), want[:, :F])
    n_fg = planes.shape[0]
    tail = planes[:, :m["n_rows"], :].transpose(1, 0, 2).reshape(m["n_rows"], n_fg * 8)[:, F:]
    assert (tail == 0).all(), "bytes of features past F must be 0"
    assert (planes[:, m["n_rows"]:, :] == 0xAB).all(), "rows past n_rows must not be written"


@pytest.mark.parametrize("name,n_prog,s_max,F,depth,p_nan,rounds", [
    ("one-chunk nodes", 300, 8, 20, 6, 0.0, 3),
    ("multi-chunk root, NaN", 1500, 8, 37, 6, 0.2, 2),
    ("depth 10, 164 features", 1200, 16, 164, 10, 0.1, 2),
    ("depth 1", 800, 4, 9, 1, 0.0, 2),
    ("depth 12", 2500, 6, 16, 12, 0.05, 1),
])
def test_rounds_bit_exact(name, n_prog, s_max, F, depth, p_nan, rounds):
    require_gpu()
    cfg = mini_config(n_prog=n_prog, s_max=s_max, n_features=F, p_nan=p_nan, seed=depth)
    m = _case(cfg, 254)
    ld = _ld(F)
    bins = oracle.gbdt_bin(m["features"], m["n_rows"], m["cuts"], m["n_cuts"], ld)
    m0 = np.zeros(m["n_rows"], np.float32)
    kw = dict(max_depth=depth, gamma=0.0 if depth > 6 else 0.001, reg_lambda=1.0, eta=0.3)
    log("gbdt round parity: %s rows=%d F=%d depth=%d rounds=%d" % (name, m["n_rows"], F, depth, rounds))
    got, gm = gpu_rounds(bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, rounds, **kw)
    want, wm = oracle_rounds(bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, rounds, **kw)
    assert sum(int((w["feature"] >= 0).sum()) for w in want) >= rounds, "degenerate case: no splits"
    assert_trees_equal(got, want, name)
    np.testing.assert_array_equal(gm.view(np.uint32), wm.view(np.uint32))


def test_standard_measured_set_bit_exact():
    """4,096 measured programs of U{1..32} statements (66,923 rows), 164 features, 254 cut points,
    Ansor's settings (depth 10, eta 0.2, gamma 0.001): two rounds."""
    require_gpu()
    m = _case(get_config("standard"), 254)
    bins = oracle.gbdt_bin(m["features"], m["n_rows"], m["cuts"], m["n_cuts"], 168)
    m0 = np.zeros(m["n_rows"], np.float32)
    log("gbdt round parity: standard measured set rows=%d" % m["n_rows"])
    got, gm = gpu_rounds(bins, 164, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 2)
    want, wm = oracle_rounds(bins, 164, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 2,
                             **oracle.GBDT_DEFAULTS)
    assert_trees_equal(got, want, "standard")
    np.testing.assert_array_equal(gm.view(np.uint32), wm.view(np.uint32))


@pytest.mark.parametrize("case", ["no rows", "one program", "constant features", "zero weights", "heavy mcw",
                                  "huge gamma", "all missing", "empty programs", "extreme scales", "base score"])
def test_degenerate_cases_bit_exact(case):
    require_gpu()
    cfg = mini_config(n_prog=200, s_max=5, n_features=11, p_nan=0.1)
    m = _case(cfg, 31)
    X, ptr, label, weight = m["features"], m["prog_ptr"], m["label"], m["weight"]
    kw = dict(max_depth=5, gamma=0.0)
    if case == "no rows":
        ptr = np.zeros(4, np.int32)
        X = X[:, :0]
        label, weight = label[:3], weight[:3]
    elif case == "one program":
        ptr = np.array([0, 40], np.int32)
        X = X[:, :40]
        label, weight = label[:1], weight[:1]
    elif case == "constant features":
        X = np.full_like(X, 0.5)
    elif case == "zero weights":
        weight = np.zeros_like(weight)
    elif case == "heavy mcw":
        kw["min_child_weight"] = float(weight.sum()) * 3
    elif case == "huge gamma":
        kw["gamma"] = 1e30
    elif case == "all missing":
        X = np.full_like(X, np.nan)
    elif case == "extreme scales":  # fixed-point exponents far from 0
        label = (label * np.float32(1e15)).astype(np.float32)
        weight = (weight * np.float32(1e-12)).astype(np.float32)
        kw["gamma"] = 0.0
        kw["reg_lambda"] = 1e-20  # on the hessians' scale, so that splits still gain
    elif case == "base score":
        kw["base_score"] = -0.75
    elif case == "empty programs":
        counts = np.diff(ptr)
        counts[::3] = 0
        ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        X = X[:, :int(ptr[-1])]
    n_rows = int(ptr[-1])
    bins = oracle.gbdt_bin(X, n_rows, m["cuts"], m["n_cuts"], 16)
    m0 = np.linspace(-1, 1, n_rows).astype(np.float32)
    log("gbdt degenerate case: %s rows=%d" % (case, n_rows))
    got, gm = gpu_rounds(bins, 11, m["cuts"], m["n_cuts"], ptr, label, weight, m0, 1, **kw)
    want, wm = oracle_rounds(bins, 11, m["cuts"], m["n_cuts"], ptr, label, weight, m0, 1, **kw)
    assert_trees_equal(got, want, case)
    np.testing.assert_array_equal(gm.view(np.uint32), wm.view(np.uint32))


def test_throughput_measured_set_full_size():
    """65,536 measured programs (2,134,518 rows), the benchmark's launch configuration (Ansor's
    settings, depth 10): bins bit-exact on every row; a depth-1 and the depth-10 round bit-exact
    against the oracle (every node field, leaf value and margin); the depth-10 round's margin change on 4,096 sampled rows
    equal to the leaf the scoring oracle reaches by routing the raw features through the GPU's tree
    (thresholds, default directions and leaves agree with the bins the tree was grown on)."""
    require_gpu()
    import torch
    m = _case(get_config("throughput"), 254)
    N, F = m["n_rows"], 164
    log("gbdt full size: %d rows; oracle binning" % N)
    want_bins = oracle.gbdt_bin_np(m["features"], N, m["cuts"], m["n_cuts"], 168)
    planes = gpu_bin(m["features"], N, m["cuts"], m["n_cuts"], N)
    np.testing.assert_array_equal(from_groups(planes, F, N), want_bins[:, :F])
    del planes
    m0 = np.zeros(N, np.float32)
    log("gbdt full size: depth-1 round")
    got, gm = gpu_rounds(want_bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 1,
                         max_depth=1)
    want, wm = oracle_rounds(want_bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 1,
                             **dict(oracle.GBDT_DEFAULTS, max_depth=1))
    assert_trees_equal(got, want, "full size depth 1")
    np.testing.assert_array_equal(gm.view(np.uint32), wm.view(np.uint32))
    log("gbdt full size: depth-10 round")
    got, gm = gpu_rounds(want_bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 1)
    tree = got[0]
    assert (tree["feature"] >= 0).sum() >= 8
    log("gbdt full size: the oracle's depth-10 round on all rows")
    want, wm = oracle_rounds(want_bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"], m0, 1,
                             **oracle.GBDT_DEFAULTS)
    assert_trees_equal(got, want, "full size depth 10")
    np.testing.assert_array_equal(gm.view(np.uint32), wm.view(np.uint32))
    rows = np.sort(np.random.default_rng(5).choice(N, 4096, replace=False))
    ens = dict(n_trees=1, n_features=F, root=np.zeros(1, np.int32), feature=tree["feature"],
               threshold=tree["threshold"], left=tree["left"], right=tree["right"],
               default_left=tree["default_left"], leaf_value=tree["leaf_value"], base_score=0.0)
    sc = oracle.score_round(ens, np.ascontiguousarray(m["features"][:, rows]),
                            np.arange(rows.size + 1, dtype=np.int32))
    np.testing.assert_array_equal(gm[rows], sc["stmt32"])
    torch.cuda.empty_cache()


def test_refit_tree_scores_through_the_scoring_path():
    """The GPU's refit tree, packed by harl_ensemble_create and evaluated by harl_score_round (an
    independent kernel path) on the same statement rows, gives every row exactly the margin change
    of the round (single tree, margins starting at 0) and every program the sum of its rows: the tree
    arrays are a valid ensemble and thresholds, default directions and leaves agree with the bins."""
    require_gpu()
    from tests.gpu_util import gpu_score
    m = _case(get_config("standard"), 254)
    N, F = m["n_rows"], 164
    bins = oracle.gbdt_bin_np(m["features"], N, m["cuts"], m["n_cuts"], 168)
    got, gm = gpu_rounds(bins, F, m["cuts"], m["n_cuts"], m["prog_ptr"], m["label"], m["weight"],
                         np.zeros(N, np.float32), 1, gamma=0.0)
    tree = got[0]
    assert (tree["feature"] >= 0).sum() >= 20
    ens = dict(n_trees=1, n_features=F, n_nodes=tree["feature"].size, root=np.zeros(1, np.int32),
               feature=tree["feature"], threshold=tree["threshold"], left=tree["left"], right=tree["right"],
               default_left=tree["default_left"], leaf_value=tree["leaf_value"], base_score=0.0)
    log("refit tree through harl_score_round: %d rows, %d splits" % (N, int((tree["feature"] >= 0).sum())))
    prog, stmt = gpu_score(ens, m["features"], m["prog_ptr"])
    np.testing.assert_array_equal(stmt, gm)
    want_prog = np.array([gm[m["prog_ptr"][p]:m["prog_ptr"][p + 1]].astype(np.float64).sum()
                          for p in range(len(m["prog_ptr"]) - 1)])
    np.testing.assert_allclose(prog, want_prog, rtol=1e-6, atol=1e-7)
