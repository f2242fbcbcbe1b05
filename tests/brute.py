"""Brute-force and closed-form checkers used to pin the oracle.

Independent of ``oracle/`` and of the HIP path: nothing here walks a tree node by node or sorts
with the oracle's comparator.  Trees are checked by enumerating every root-to-leaf path as an
explicit conjunction of split predicates and evaluating all of them; the MLP with numpy float64
matrix products; rankings with ``numpy.lexsort``.
"""
from __future__ import annotations

import numpy as np


def leaf_paths(ens: dict, t: int):
    """Every root-to-leaf path of tree t as (leaf_node, [(feature, threshold, went_left, default_left)])."""
    feature, left, right = ens["feature"], ens["left"], ens["right"]
    thr, dl = ens["threshold"], ens["default_left"]
    out = []
    stack = [(int(ens["root"][t]), [])]
    while stack:
        n, conds = stack.pop()
        if feature[n] < 0:
            out.append((n, conds))
            continue
        c = (int(feature[n]), np.float32(thr[n]), bool(dl[n]))
        stack.append((int(left[n]), conds + [(c[0], c[1], True, c[2])]))
        stack.append((int(right[n]), conds + [(c[0], c[1], False, c[2])]))
    return out


def edge_holds(x: np.ndarray, thr: np.float32, went_left: bool, default_left: bool) -> np.ndarray:
    """Whether the edge condition holds for each value: a left edge needs x < thr (or x missing
    with default left); a right edge needs x >= thr (or x missing with default right)."""
    miss = np.isnan(x)
    with np.errstate(invalid="ignore"):
        if went_left:
            return (~miss & (x < thr)) | (miss & default_left)
        return (~miss & (x >= thr)) | (miss & (not default_left))


def brute_stmt_scores(ens: dict, X: np.ndarray, n_rows: int):
    """Per-row ensemble sum from explicit path predicates.  Also returns, per (row, tree), how many
    leaf predicates hold (must be exactly one)."""
    T = int(ens["n_trees"])
    total = np.zeros(n_rows, dtype=np.float64)
    n_true = np.zeros((n_rows, T), dtype=np.int64)
    for t in range(T):
        for leaf, conds in leaf_paths(ens, t):
            pred = np.ones(n_rows, dtype=bool)
            for f, th, wl, dl in conds:
                pred &= edge_holds(X[f, :n_rows], th, wl, dl)
            n_true[:, t] += pred
            total += np.where(pred, np.float64(ens["leaf_value"][leaf]), 0.0)
    return total, n_true


def bf16_round_bits(v) -> np.ndarray:
    """Round fp64 values (normal range) to bf16 precision, ties to even, on the fp64 bit pattern:
    bf16 keeps 7 of fp64's 52 stored mantissa bits."""
    v = np.asarray(v, dtype=np.float64)
    b = v.view(np.uint64)
    drop = np.uint64(45)
    half = np.uint64((1 << 44) - 1)
    lsb = (b >> drop) & np.uint64(1)
    r = ((b + half + lsb) >> drop) << drop
    out = r.view(np.float64).copy()
    out[v == 0] = v[v == 0]
    return out


def decode(w, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return (np.asarray(w, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(w, dtype=np.float32).astype(np.float64)


def numpy_policy(pol: dict, states) -> dict:
    """Actor/critic forward with numpy float64 matmul (bf16 policies round h1, h2 to bf16)."""
    dt = pol["dtype"]
    s = decode(states, dt)
    W1, W2, Wa, Wv = (decode(pol[k], dt) for k in ("w1", "w2", "wa", "wv"))
    b1, b2, ba, bv = (np.asarray(pol[k], dtype=np.float64) for k in ("b1", "b2", "ba", "bv"))
    h1 = np.maximum(s @ W1.T + b1, 0.0)
    if dt == "bf16":
        h1 = bf16_round_bits(h1)
    h2 = np.maximum(h1 @ W2.T + b2, 0.0)
    if dt == "bf16":
        h2 = bf16_round_bits(h2)
    z = h2 @ Wa.T + ba
    v = (h2 @ Wv.T + bv)[:, 0]
    return dict(logits=z, value=v, action=np.argmax(z, axis=1).astype(np.int32))


def lexsort_topk(score, k: int, index_base: int = 0):
    """Full ranking by (score desc, index asc) via numpy.lexsort; NaN last; -0 ties +0."""
    s = np.asarray(score, dtype=np.float32).astype(np.float64)
    idx = np.arange(s.size, dtype=np.int64)
    neg = -s
    neg[np.isnan(s)] = np.inf      # NaN after every number, then by index
    nan_last = np.isnan(s).astype(np.int8)
    order = np.lexsort((idx, neg, nan_last))
    return s[order[:k]].astype(np.float32), order[:k] + index_base
