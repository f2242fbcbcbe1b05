"""Pins of the CPU oracle against things other than itself (brute force, closed forms, invariants,
library routines).  Paper anchors: the cost model C scores every new schedule (Algorithm 1; the
cost model is XGBoost, Section 6.1, Appendix A.1); the actor and critic act on the states
(Algorithm 1; Section 4.3, Eq. 6); the top-K of the heap H are the K best predicted scores
(Algorithm 1; Section 4.3, Top-K Selection Phase); each step of a schedule track is rewarded with
the relative change of its score (Algorithm 1) and judged by the advantage of Eq. 6, and the
adaptive-stopping search drops the tracks of lowest advantage (Section 5); the actor picks the best
modification of each type (Section 4.3, Appendix A.1), sampled during PPO rollouts (Section 6.1)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_batch, gen_ensemble, gen_policy, gen_states, mini_config, get_config
from synth.gen import bf16_bits_from_f32, f32_from_bf16_bits
from tests import brute


# ----------------------------------------------------------------------------------------------
# tree routing and sums
# ----------------------------------------------------------------------------------------------
def _irregular_ensemble(rng, n_trees, n_features, max_depth, thr_pool):
    """Random non-complete trees in the explicit node format (children ids, leaves feature -1)."""
    feature, threshold, left, right, dl, leaf, root = [], [], [], [], [], [], []

    def build(depth):
        nid = len(feature)
        feature.append(-1); threshold.append(0.0); left.append(-1); right.append(-1)
        dl.append(0); leaf.append(0.0)
        if depth < max_depth and (depth == 0 or rng.random() < 0.7):
            feature[nid] = int(rng.integers(0, n_features))
            threshold[nid] = float(rng.choice(thr_pool))
            dl[nid] = int(rng.random() < 0.5)
            left[nid] = build(depth + 1)
            right[nid] = build(depth + 1)
        else:
            leaf[nid] = float(np.float32(rng.normal(0, 0.1)))
        return nid

    for _ in range(n_trees):
        root.append(build(0))
    return dict(n_trees=n_trees, n_features=n_features, max_depth=max_depth,
                root=np.array(root, np.int32), feature=np.array(feature, np.int32),
                threshold=np.array(threshold, np.float32), left=np.array(left, np.int32),
                right=np.array(right, np.int32), default_left=np.array(dl, np.uint8),
                leaf_value=np.array(leaf, np.float32), base_score=0.0)


def _plant_threshold_rows(X, ens, n_rows, rng):
    """Overwrite some feature values with exact thresholds and their fp32 neighbours so that
    x == thr and x just below thr occur for many splits."""
    internal = np.nonzero(ens["feature"] >= 0)[0]
    for r in range(0, n_rows, 3):
        for n in rng.choice(internal, size=min(6, internal.size), replace=False):
            f, th = ens["feature"][n], np.float32(ens["threshold"][n])
            X[f, r] = rng.choice([th, np.nextafter(th, np.float32(-np.inf)), np.nextafter(th, np.float32(np.inf))])


@pytest.mark.parametrize("p_nan", [0.0, 0.2])
@pytest.mark.parametrize("depth", [1, 3, 4])
def test_tree_sums_match_path_predicates(p_nan, depth):
    cfg = mini_config(depth=depth, p_nan=p_nan, n_trees=4, n_features=8, n_prog=60, s_max=6)
    ens = gen_ensemble(cfg)
    b = gen_batch(cfg)
    X, n = b["features"].copy(), b["n_rows"]
    _plant_threshold_rows(X, ens, n, np.random.default_rng(7))
    got = oracle.score_round(ens, X, b["prog_ptr"])
    want, n_true = brute.brute_stmt_scores(ens, X, n)
    assert (n_true == 1).all(), "every (row, tree) must satisfy exactly one leaf predicate"
    np.testing.assert_allclose(got["stmt"], want, rtol=0, atol=1e-12)


def test_irregular_trees_match_path_predicates():
    rng = np.random.default_rng(3)
    cfg = mini_config(p_nan=0.15, n_features=6, n_prog=50)
    b = gen_batch(cfg)
    X, n = b["features"].copy(), b["n_rows"]
    pool = np.unique(X[~np.isnan(X)])
    ens = _irregular_ensemble(rng, n_trees=5, n_features=6, max_depth=5, thr_pool=pool)
    got = oracle.score_round(ens, X, b["prog_ptr"])
    want, n_true = brute.brute_stmt_scores(ens, X, n)
    assert (n_true == 1).all()
    np.testing.assert_allclose(got["stmt"], want, rtol=0, atol=1e-12)


def _stump(feature, thr, dl, lv, rv, n_features):
    return dict(n_trees=1, n_features=n_features, max_depth=1, root=np.array([0], np.int32),
                feature=np.array([feature, -1, -1], np.int32),
                threshold=np.array([thr, 0, 0], np.float32),
                left=np.array([1, -1, -1], np.int32), right=np.array([2, -1, -1], np.int32),
                default_left=np.array([dl, 0, 0], np.uint8),
                leaf_value=np.array([0, lv, rv], np.float32), base_score=0.0)


@pytest.mark.parametrize("thr", [np.float32(0.0), np.float32(1.5), np.float32(-2.25), np.float32(3.0e-3)])
@pytest.mark.parametrize("dl", [0, 1])
def test_threshold_ties_and_missing(thr, dl):
    """x == thr goes right; the fp32 value just below goes left; -0 equals +0; NaN follows the
    default direction; +-inf go to the sides their order says."""
    L, R = 1.0, 2.0
    below = np.nextafter(thr, np.float32(-np.inf))
    above = np.nextafter(thr, np.float32(np.inf))
    vals = [thr, below, above, np.float32(np.nan), np.float32(-np.inf), np.float32(np.inf)]
    want = [R, L, R, L if dl else R, L, R]
    if thr == 0:
        vals.append(np.float32(-0.0)); want.append(R)
    X = np.array([vals], dtype=np.float32)
    ens = _stump(0, thr, dl, L, R, 1)
    ptr = np.arange(len(vals) + 1, dtype=np.int32)
    got = oracle.score_round(ens, X, ptr)
    np.testing.assert_array_equal(got["prog"], np.array(want))


def test_all_missing_row_follows_default_bits():
    """A row of NaN reaches, in every complete tree, the leaf spelled by the default bits along
    the default path: leaf number = the bits read as a binary number (1 = right)."""
    cfg = mini_config(depth=5, n_trees=6, n_features=8)
    ens = gen_ensemble(cfg)
    X = np.full((8, 1), np.nan, dtype=np.float32)
    got = oracle.score_round(ens, X, np.array([0, 1], np.int32))
    D, M = cfg.depth, 2 ** (cfg.depth + 1) - 1
    total = 0.0
    for t in range(cfg.n_trees):
        n, bits = 0, 0
        for _ in range(D):
            go_right = 0 if ens["default_left"][t * M + n] else 1
            bits = 2 * bits + go_right
            n = 2 * n + 1 + go_right
        total += float(ens["leaf_value"][t * M + (2 ** D - 1) + bits])
    assert got["prog"][0] == pytest.approx(total, abs=1e-12)


def test_leafless_root_and_constant_leaves_closed_form():
    """Constant leaves c = 2**-4: every statement scores T*c, every program n_stmt*T*c, exactly."""
    cfg = mini_config(depth=4, n_trees=7, n_prog=40, s_max=9)
    ens = gen_ensemble(cfg)
    ens["leaf_value"] = np.where(ens["feature"] < 0, np.float32(2.0 ** -4), np.float32(0)).astype(np.float32)
    b = gen_batch(cfg)
    got = oracle.score_round(ens, b["features"], b["prog_ptr"])
    n_stmt = np.diff(b["prog_ptr"]).astype(np.float64)
    np.testing.assert_array_equal(got["prog"], n_stmt * cfg.n_trees * 2.0 ** -4)
    np.testing.assert_array_equal(got["stmt"], np.full(b["n_rows"], cfg.n_trees * 2.0 ** -4))


def test_program_sum_invariants_exact_variant():
    """Dyadic leaves: every partial sum is exact in fp32; prog = sum of stmt exactly; a
    one-statement program equals its statement; permuting statements changes nothing; fp32 sums
    in forward and reverse order agree bit for bit with the fp64 oracle."""
    cfg = get_config("tiny", exact=True).with_(n_prog=96)
    ens = gen_ensemble(cfg)
    b = gen_batch(cfg)
    got = oracle.score_round(ens, b["features"], b["prog_ptr"])
    ptr = b["prog_ptr"]
    for p in range(cfg.n_prog):
        rows = got["stmt"][ptr[p]:ptr[p + 1]]
        assert got["prog"][p] == rows.sum()
        fwd = np.float32(0)
        for v in rows.astype(np.float32):
            fwd = np.float32(fwd + v)
        rev = np.float32(0)
        for v in rows.astype(np.float32)[::-1]:
            rev = np.float32(rev + v)
        assert fwd == rev == np.float32(got["prog"][p])
        if ptr[p + 1] - ptr[p] == 1:
            assert got["prog"][p] == got["stmt"][ptr[p]]
    # permute statements inside each program
    rng = np.random.default_rng(5)
    perm = np.concatenate([ptr[p] + rng.permutation(ptr[p + 1] - ptr[p]) for p in range(cfg.n_prog)])
    got2 = oracle.score_round(ens, b["features"][:, perm], ptr)
    np.testing.assert_array_equal(got2["prog"], got["prog"])


def test_scale_bounds_score():
    cfg = mini_config(depth=4, n_trees=5, p_nan=0.1)
    ens, b = gen_ensemble(cfg), gen_batch(cfg)
    got = oracle.score_round(ens, b["features"], b["prog_ptr"])
    assert (np.abs(got["prog"]) <= got["scale"] + 1e-12).all()
    assert (got["scale"] > 0).all()


def test_base_score_and_empty_programs():
    cfg = mini_config(depth=2, n_trees=3)
    ens, b = gen_ensemble(cfg), gen_batch(cfg)
    ens["base_score"] = 0.5
    ptr = np.array([0, 0, 2, 2, 3], np.int32)      # programs 0 and 2 have no statements
    got = oracle.score_round(ens, b["features"], ptr, n_rows=3)
    assert got["prog"][0] == 0.5 and got["prog"][2] == 0.5
    want, _ = brute.brute_stmt_scores(ens, b["features"], 3)
    assert got["prog"][1] == pytest.approx(0.5 + want[0] + want[1], abs=1e-12)


def test_malformed_inputs_rejected():
    cfg = mini_config()
    ens, b = gen_ensemble(cfg), gen_batch(cfg)
    bad_ptr = b["prog_ptr"].copy()
    bad_ptr[3] = bad_ptr[4] + 1
    with pytest.raises(ValueError):
        oracle.score_round(ens, b["features"], bad_ptr, n_rows=b["n_rows"])
    cyc = dict(ens)
    cyc["left"] = ens["left"].copy()
    cyc["left"][0] = 0                                  # a cycle
    cyc["default_left"] = np.ones_like(ens["default_left"])
    X = np.full_like(b["features"], np.nan)
    with pytest.raises(ValueError):
        oracle.score_round(cyc, X, b["prog_ptr"])


# ----------------------------------------------------------------------------------------------
# actor / critic
# ----------------------------------------------------------------------------------------------
def test_bf16_rounding_rule():
    """Ties go to even; the oracle's rounding agrees with an independent bit-level rounding and,
    on fp32 inputs, with the input generator's fp32 -> bf16 rounding."""
    assert oracle.round_bf16(1 + 2 ** -8) == 1.0                       # tie, even is 1.0
    assert oracle.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6           # tie, rounds up to even
    assert oracle.round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7    # just above the tie
    assert oracle.round_bf16(-(1 + 2 ** -8)) == -1.0
    assert oracle.round_bf16(2.0 ** -130) == 2.0 ** -130                 # bf16 subnormal, exact
    rng = np.random.default_rng(11)
    v = rng.standard_normal(4000) * np.exp(rng.uniform(-20, 20, 4000))
    ties = np.array([1 + 2 ** -8, 3 + 2 ** -6, 0.75 + 2 ** -10, 100.0 + 0.25])
    v = np.concatenate([v, ties, -ties])
    ours = np.array([oracle.round_bf16(x) for x in v])
    np.testing.assert_array_equal(ours, brute.bf16_round_bits(v))
    f32 = v.astype(np.float32)
    gen = f32_from_bf16_bits(bf16_bits_from_f32(f32)).astype(np.float64)
    np.testing.assert_array_equal(np.array([oracle.round_bf16(float(x)) for x in f32]), gen)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_matches_numpy_matmul(dtype):
    cfg = mini_config(pol_dtype=dtype, pol_s=24, pol_h1=40, pol_h2=36, pol_a=9, n_prog=70)
    pol, st = gen_policy(cfg), gen_states(cfg)
    got = oracle.policy_step(pol, st)
    ref = brute.numpy_policy(pol, st)
    np.testing.assert_allclose(got["logits"], ref["logits"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["value"], ref["value"], rtol=0, atol=1e-12)
    gap = np.sort(ref["logits"], axis=1)
    clear = (gap[:, -1] - gap[:, -2]) > 1e-9
    np.testing.assert_array_equal(got["action"][clear], ref["action"][clear])
    assert (np.abs(got["logits"]) <= got["logit_scale"] + 1e-12).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_policy_exact_integer_variant(dtype):
    """Integer states/weights/biases: every activation is an integer of magnitude <= 85, exact in
    bf16 and fp32; compare with pure-Python integer arithmetic; ties resolve to the lowest index."""
    cfg = mini_config(pol_dtype=dtype, pol_s=16, pol_h1=32, pol_h2=32, pol_a=10, n_prog=50, exact=True)
    pol, st = gen_policy(cfg), gen_states(cfg)
    got = oracle.policy_step(pol, st)
    W1, W2, Wa, Wv = (brute.decode(pol[k], dtype).astype(int).tolist() for k in ("w1", "w2", "wa", "wv"))
    b1, b2, ba, bv = (np.asarray(pol[k]).astype(int).tolist() for k in ("b1", "b2", "ba", "bv"))
    S = brute.decode(st, dtype).astype(int).tolist()
    n_ties = 0
    for i, s in enumerate(S):
        h1 = [max(0, sum(w * x for w, x in zip(row, s)) + b) for row, b in zip(W1, b1)]
        h2 = [max(0, sum(w * x for w, x in zip(row, h1)) + b) for row, b in zip(W2, b2)]
        z = [sum(w * x for w, x in zip(row, h2)) + b for row, b in zip(Wa, ba)]
        v = sum(w * x for w, x in zip(Wv[0], h2)) + bv[0]
        assert max(map(abs, h1 + h2 + z)) <= 85
        assert got["logits"][i].tolist() == z
        assert got["value"][i] == v
        assert got["action"][i] == z.index(max(z))
        n_ties += z.count(max(z)) > 1
    assert n_ties > 0, "the exact variant should exercise the lowest-index tie rule"


def test_policy_positive_weights_collapse_to_one_linear_map():
    """With non-negative states, weights and biases the ReLUs are identities, so the logits equal
    (Wa W2 W1) s + Wa W2 b1 + Wa b2 + ba, with the matrices multiplied first."""
    cfg = mini_config(pol_s=12, pol_h1=20, pol_h2=18, pol_a=7, n_prog=30)
    pol = gen_policy(cfg)
    for k in ("w1", "w2", "wa", "wv", "b1", "b2", "ba", "bv"):
        pol[k] = np.abs(pol[k]).astype(np.float32)
    st = np.abs(gen_states(cfg))
    got = oracle.policy_step(pol, st)
    W1, W2, Wa, Wv = (pol[k].astype(np.float64) for k in ("w1", "w2", "wa", "wv"))
    b1, b2, ba, bv = (pol[k].astype(np.float64) for k in ("b1", "b2", "ba", "bv"))
    M = Wa @ W2 @ W1
    c = Wa @ W2 @ b1 + Wa @ b2 + ba
    want = st.astype(np.float64) @ M.T + c
    np.testing.assert_allclose(got["logits"], want, rtol=1e-12, atol=1e-12)
    mv = Wv @ W2 @ W1
    cv = Wv @ W2 @ b1 + Wv @ b2 + bv
    np.testing.assert_allclose(got["value"], (st.astype(np.float64) @ mv.T + cv)[:, 0], rtol=1e-12)


def test_softmax_invariants():
    cfg = mini_config(pol_a=17, n_prog=64)
    got = oracle.policy_step(gen_policy(cfg), gen_states(cfg))
    np.testing.assert_allclose(got["probs"].sum(axis=1), 1.0, atol=1e-12)
    assert (got["probs"] > 0).all()
    best = got["probs"][np.arange(64), got["action"]]
    assert (best >= got["probs"].max(axis=1) - 1e-15).all()
    # softmax is invariant to adding a constant to every logit: compare ratios
    z = got["logits"]
    r = got["probs"][:, 1:] / got["probs"][:, :1]
    np.testing.assert_allclose(r, np.exp(z[:, 1:] - z[:, :1]), rtol=1e-10)


# ----------------------------------------------------------------------------------------------
# top-K and the running heap
# ----------------------------------------------------------------------------------------------
def test_topk_matches_lexsort():
    rng = np.random.default_rng(1)
    s = rng.standard_normal(3000).astype(np.float32)
    s[rng.integers(0, 3000, 400)] = np.float32(0.5)           # many exact ties
    s[::97] = -0.0
    s[::89] = 0.0
    for k in (1, 7, 128, 3000):
        got = oracle.topk(s, k, index_base=1000)
        want = brute.lexsort_topk(s, k, index_base=1000)
        np.testing.assert_array_equal(got[1], want[1])
        np.testing.assert_array_equal(got[0], want[0])


def test_topk_special_cases():
    assert oracle.topk(np.zeros(10, np.float32), 4)[1].tolist() == [0, 1, 2, 3]
    s = np.array([-0.0, 0.0, -0.0, 0.0], np.float32)
    assert oracle.topk(s, 4)[1].tolist() == [0, 1, 2, 3]
    s = np.array([1.0, np.nan, 3.0, -np.inf, 3.0], np.float32)
    assert oracle.topk(s, 5)[1].tolist() == [2, 4, 0, 3, 1]
    rng = np.random.default_rng(2)
    s = rng.integers(0, 5, 200).astype(np.float32)
    assert oracle.topk(s, 1)[1][0] == int(np.argmax(s))        # k = 1: lowest-index argmax
    with pytest.raises(ValueError):
        oracle.topk(s, 201)


def test_merge_equals_topk_of_union_in_any_order():
    rng = np.random.default_rng(4)
    k, nb, n = 50, 6, 300
    batches = [rng.integers(-20, 20, n).astype(np.float32) / 4 for _ in range(nb)]
    allv = np.concatenate(batches)
    want = oracle.topk(allv, k)
    np.testing.assert_array_equal(want[1], brute.lexsort_topk(allv, k)[1])
    for order in (range(nb), reversed(range(nb)), rng.permutation(nb)):
        rs, ri = oracle.reset(k)
        for bidx in order:
            rs, ri = oracle.merge(rs, ri, batches[bidx], bidx * n)
        np.testing.assert_array_equal(ri, want[1])
        np.testing.assert_array_equal(rs, want[0])
    # save after 3 batches, resume from the copy: identical
    rs, ri = oracle.reset(k)
    for bidx in range(3):
        rs, ri = oracle.merge(rs, ri, batches[bidx], bidx * n)
    saved = (rs.copy(), ri.copy())
    for bidx in range(3, nb):
        saved = oracle.merge(saved[0], saved[1], batches[bidx], bidx * n)
    np.testing.assert_array_equal(saved[1], want[1])


def test_merge_fewer_candidates_than_k_keeps_sentinels():
    rs, ri = oracle.reset(8)
    rs, ri = oracle.merge(rs, ri, np.array([3.0, -np.inf, 1.0], np.float32), 10)
    assert ri[:3].tolist() == [10, 12, 11]
    assert (ri[3:] == oracle.RESET_INDEX).all() and np.isneginf(rs[3:]).all()


# ----------------------------------------------------------------------------------------------
# schedule tracks: reward, advantage, elimination
# ----------------------------------------------------------------------------------------------
def test_reward_advantage_closed_forms():
    # (c_prev, c_next, v_prev, v_next) -> reward, advantage with gamma = 0.75, eps = 0.25
    rows = [
        (2.0, 3.0, 1.0, 2.0, 0.5, 0.5 + 1.5 - 1.0),      # +50 % score, V from 1 to 2
        (-4.0, -2.0, 0.0, 0.0, 0.5, 0.5),                # negative scores: an improvement is positive
        (-2.0, -4.0, 0.5, -1.0, -1.0, -1.0 - 0.75 - 0.5),
        (0.125, 0.375, 0.0, 0.0, 1.0, 1.0),              # |C(s)| below eps: the denominator is eps
        (0.0, -0.5, 0.25, 1.0, -2.0, -2.0 + 0.75 - 0.25),
        (3.0, 3.0, -1.0, 1.0, 0.0, 0.0 + 0.75 + 1.0),    # unchanged score: only the critic terms
    ]
    c0, c1, v0, v1, r, a = (np.array(x, dtype=np.float64) for x in zip(*rows))
    got = oracle.track_advantage(c0, c1, v0, v1, gamma=0.75, eps=0.25)
    np.testing.assert_array_equal(got["reward"], r)
    np.testing.assert_array_equal(got["adv"], a)
    np.testing.assert_array_equal(got["scale"], np.abs(r) + np.abs(0.75 * v1) + np.abs(v0))


def test_reward_sign_and_critic_reductions():
    rng = np.random.default_rng(11)
    n = 5000
    c0 = (rng.standard_normal(n) * 10).astype(np.float32)
    c1 = (c0 + rng.standard_normal(n)).astype(np.float32)
    v0 = rng.standard_normal(n).astype(np.float32)
    v1 = rng.standard_normal(n).astype(np.float32)
    got = oracle.track_advantage(c0, c1, v0, v1, gamma=0.0)
    # the reward has the sign of the score change whatever the sign of the score
    np.testing.assert_array_equal(np.sign(got["reward"]), np.sign(c1.astype(np.float64) - c0))
    # gamma = 0: A = r - V(s); gamma = 1 with an unchanged score: A = V(s') - V(s), exact in fp64
    np.testing.assert_array_equal(got["adv"], got["reward"] - v0)
    same = oracle.track_advantage(c0, c0, v0, v1, gamma=1.0)
    np.testing.assert_array_equal(same["reward"], np.zeros(n))
    np.testing.assert_array_equal(same["adv"], v1.astype(np.float64) - v0)
    # the discount factor of Section 6.1 enters at its fp32 value
    dflt = oracle.track_advantage(c0, c0, np.zeros(n), v1)
    np.testing.assert_array_equal(dflt["adv"], v1.astype(np.float64) * float(np.float32(0.9)))


def _elimination_properties(adv, n_keep, keep):
    """The survivors are the unique set of n_keep tracks such that every survivor ranks ahead of
    every eliminated track: a larger advantage, or an equal one (-0 == +0) at a lower index; NaN
    behind every number."""
    n = adv.size
    keep = np.asarray(keep)
    assert keep.size == n_keep
    assert (np.diff(keep) > 0).all() and (keep >= 0).all() and (keep < n).all()
    kept = np.zeros(n, bool)
    kept[keep] = True
    for i in np.flatnonzero(kept):
        for j in np.flatnonzero(~kept):
            ai, aj = adv[i], adv[j]
            if np.isnan(ai):
                assert np.isnan(aj) and i < j
            elif not np.isnan(aj):
                assert ai > aj or (ai == aj and i < j)


def test_eliminate_ranking_properties_small():
    rng = np.random.default_rng(12)
    pool = np.array([-1.5, -0.0, 0.0, 0.25, 2.0, np.nan, np.inf, -np.inf], np.float32)
    for trial in range(40):
        n = int(rng.integers(1, 12))
        adv = rng.choice(pool, n).astype(np.float32)
        for n_keep in range(n + 1):
            _elimination_properties(adv, n_keep, oracle.track_eliminate(adv, n_keep))


def test_eliminate_special_cases():
    adv = np.array([0.5, -1.0, 3.0, 3.0, np.nan, 0.5, -0.0, 0.0], np.float32)
    assert oracle.track_eliminate(adv, 8).tolist() == list(range(8))
    assert oracle.track_eliminate(adv, 0).tolist() == []
    assert oracle.track_eliminate(adv, 2).tolist() == [2, 3]
    assert oracle.track_eliminate(adv, 3).tolist() == [0, 2, 3]          # tie at 0.5: lower index
    assert oracle.track_eliminate(adv, 6).tolist() == [0, 2, 3, 5, 6, 7]  # -0 ties +0
    assert oracle.track_eliminate(adv, 7).tolist() == [0, 1, 2, 3, 5, 6, 7]  # NaN goes first
    assert oracle.track_eliminate(np.zeros(10, np.float32), 4).tolist() == [0, 1, 2, 3]
    # distinct advantages: permuting the tracks permutes the survivors
    rng = np.random.default_rng(13)
    a = rng.permutation(1000).astype(np.float32)
    perm = rng.permutation(1000)
    base = set(oracle.track_eliminate(a, 300).tolist())
    moved = set(oracle.track_eliminate(a[perm], 300).tolist())
    assert {int(perm[i]) for i in moved} == base
    assert base == set(np.flatnonzero(a >= 700).tolist())
    with pytest.raises(ValueError):
        oracle.track_eliminate(adv, 9)


def test_eliminate_count_rounds_the_dropped_share_down():
    assert [oracle.eliminate_count(n) for n in (1, 2, 3, 64, 65, 127, 4096)] == [1, 1, 2, 32, 33, 64, 2048]
    assert oracle.eliminate_count(100, rho=0.3) == 70


# ----------------------------------------------------------------------------------------------
# per-type action selection and its random numbers
# ----------------------------------------------------------------------------------------------
def test_philox_known_answers():
    # known-answer values of Philox4x32-10 distributed with the generator's reference
    # implementation (Salmon et al., SC'11): (counter, key) -> output
    kat = [
        ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
        ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
        ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
         [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
    ]
    for ctr, key, want in kat:
        assert oracle.philox4x32(ctr, key) == want


_SEGS = np.array([0, 17, 20, 23, 26], np.int32)   # num_iters = 4: 4 x 4 + 1 tile actions, 3 x 3 others


def test_greedy_select_is_per_segment_first_argmax():
    rng = np.random.default_rng(21)
    z = rng.integers(-3, 3, (500, 26)).astype(np.float32)     # many ties
    z[::7, 3] = np.nan
    z[5, 17:20] = -np.inf
    z[6, 20:23] = np.nan
    got = oracle.policy_select(z, _SEGS)
    for s in range(4):
        lo, hi = _SEGS[s], _SEGS[s + 1]
        seg = np.where(np.isnan(z[:, lo:hi]), -np.inf, z[:, lo:hi])
        np.testing.assert_array_equal(got["action"][:, s], lo + np.argmax(seg, axis=1))
    assert got["action"][5, 1] == 17 and got["action"][6, 2] == 20


def test_select_softmax_and_logp_identities():
    rng = np.random.default_rng(22)
    z = (rng.standard_normal((300, 26)) * 3).astype(np.float32)
    for sample in (False, True):
        got = oracle.policy_select(z, _SEGS, sample=sample, seed=7, counter=3)
        for s in range(4):
            lo, hi = _SEGS[s], _SEGS[s + 1]
            np.testing.assert_allclose(got["probs"][:, lo:hi].sum(axis=1), 1.0, atol=1e-12)
            p = got["probs"][np.arange(300), got["action"][:, s]]
            np.testing.assert_allclose(got["logp"][:, s], np.log(p), rtol=0, atol=1e-12)
            ratio = got["probs"][:, lo + 1] / got["probs"][:, lo]
            np.testing.assert_allclose(ratio, np.exp(z[:, lo + 1].astype(np.float64) - z[:, lo]), rtol=1e-12)


def test_sampling_frequencies_follow_the_softmax():
    # Gumbel-max: argmax(z + G) is distributed as softmax(z); 40,000 draws (states) of one row
    z = np.log(np.array([[0.5, 0.3, 0.2, 0.05, 0.6, 0.35]], np.float64)).astype(np.float32)
    segs = np.array([0, 3, 6], np.int32)
    n = 40000
    got = oracle.policy_select(np.repeat(z, n, axis=0), segs, sample=True, seed=0x1234_5678_9ABC, counter=5)
    for s, (lo, hi) in enumerate(((0, 3), (3, 6))):
        p = np.exp(z[0, lo:hi].astype(np.float64))
        p /= p.sum()
        freq = np.bincount(got["action"][:, s] - lo, minlength=hi - lo) / n
        sigma = np.sqrt(p * (1 - p) / n)
        assert np.all(np.abs(freq - p) < 5 * sigma), (freq, p)


def test_sampling_is_a_function_of_seed_counter_state():
    rng = np.random.default_rng(23)
    z = rng.standard_normal((2000, 26)).astype(np.float32)
    a = oracle.policy_select(z, _SEGS, sample=True, seed=11, counter=0)["action"]
    np.testing.assert_array_equal(a, oracle.policy_select(z, _SEGS, sample=True, seed=11, counter=0)["action"])
    for other in (dict(seed=12, counter=0), dict(seed=11, counter=1), dict(seed=11 + (1 << 32), counter=0),
                  dict(seed=11, counter=1 << 32)):
        b = oracle.policy_select(z, _SEGS, sample=True, **other)["action"]
        assert (a != b).mean() > 0.3
    # the noise of state b does not depend on the other states
    sub = oracle.policy_select(z[:1000], _SEGS, sample=True, seed=11, counter=0)["action"]
    np.testing.assert_array_equal(sub, a[:1000])
    # huge logit gaps: sampling agrees with the greedy choice
    zz = z.copy()
    zz[:, 0] += 1000.0
    assert (oracle.policy_select(zz, _SEGS, sample=True, seed=3)["action"][:, 0] == 0).all()
