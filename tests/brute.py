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


def brute_gbdt_tree(bins, F, cuts, n_cuts, prog_ptr, label, weight, margin, max_depth, eta, lam, gamma, mcw,
                    base_score=0.0):
    """Depth-wise greedy tree of one boosting round under the pack-sum squared error, from sets of
    rows and exact rational arithmetic: every candidate (feature f, threshold index t, missing
    direction) is scored by summing the rows' gradients directly.  Returns (nodes, margins, gaps):
    nodes maps heap index -> ("split", f, t, default_left) or ("leaf", value as Fraction); gaps
    lists, per split decision, the relative distance between the best and the next distinct gain
    (a decision closer than fp64 rounding cannot be pinned)."""
    from fractions import Fraction as Fr
    P = len(prog_ptr) - 1
    g, h = {}, {}
    for p in range(P):
        s = Fr(base_score)
        for r in range(prog_ptr[p], prog_ptr[p + 1]):
            s += Fr(float(margin[r]))
        for r in range(prog_ptr[p], prog_ptr[p + 1]):
            g[r] = Fr(float(weight[p])) * (s - Fr(float(label[p])))
            h[r] = Fr(float(weight[p]))
    lam, eta, gamma, mcw = Fr(lam), Fr(eta), Fr(gamma), Fr(mcw)
    nodes, gaps = {}, []
    new_margin = np.array(margin, dtype=np.float32, copy=True)

    def score(G, H):
        return G * G / (H + lam)

    def grow(k, depth, rows):
        G = sum((g[r] for r in rows), Fr(0))
        H = sum((h[r] for r in rows), Fr(0))
        cands = []
        if depth < max_depth:
            for f in range(F):
                for t in range(1, int(n_cuts[f]) + 1):
                    for dleft in (1, 0):
                        L = [r for r in rows if (bins[r, f] == 255 and dleft) or (bins[r, f] != 255 and bins[r, f] < t)]
                        GL = sum((g[r] for r in L), Fr(0))
                        HL = sum((h[r] for r in L), Fr(0))
                        if HL < mcw or H - HL < mcw:
                            continue
                        cands.append((score(GL, HL) + score(G - GL, H - HL) - score(G, H), f, t, dleft))
        if cands:
            best = max(c[0] for c in cands)
            first = next(c for c in cands if c[0] == best)
            others = [c[0] for c in cands if c[0] != best]
            if others:
                gaps.append(float((best - max(others)) / max(abs(best), Fr(1, 10**30))))
            if best > gamma:
                gaps.append(float(abs(best - gamma) / max(abs(best), Fr(1, 10**30))))
                _, f, t, dleft = first
                nodes[k] = ("split", f, t, dleft)
                L = [r for r in rows if (bins[r, f] == 255 and dleft) or (bins[r, f] != 255 and bins[r, f] < t)]
                R = [r for r in rows if r not in set(L)]
                grow(2 * k + 1, depth + 1, L)
                grow(2 * k + 2, depth + 1, R)
                return
            gaps.append(float(abs(best - gamma) / max(abs(best), Fr(1, 10**30))))
        w = -(G / (H + lam)) * eta
        nodes[k] = ("leaf", w)
        for r in rows:
            new_margin[r] = np.float32(new_margin[r] + np.float32(float(w)))

    grow(0, 0, list(range(int(prog_ptr[-1]))))
    return nodes, new_margin, gaps
