"""TEST INFRASTRUCTURE: the CPU oracle for one HARL search round.

A ctypes wrapper over ``harl_oracle.c`` (plain C, fp64, optional OpenMP).  It computes, from the
paper's definitions, what the HIP path must reproduce: per-program cost-model scores (GBDT over
statement rows, summed per program), the actor/critic forward with its argmax action, and the
top-K / running-heap selection, and for schedule tracks the reward, the advantage and the
adaptive-stopping elimination, the per-modification-type action selection (greedy or sampled
through a counter-based generator) and one boosting round of the cost model's refit on measured
programs.  Only ``tests/``, the package's ``smoke()`` check and
``bench.py``'s ``cpu_baseline`` leg may import this package; the product path never does.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "harl_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_liboracle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/_liboracle.so`` (plain -O2, no fast-math)."""
    global _lib
    with _lock:
        if force or not os.path.exists(_LIB_PATH):
            tmp = _LIB_PATH + ".tmp%d" % os.getpid()
            subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
            os.replace(tmp, _LIB_PATH)
            _lib = None
    return _LIB_PATH


def _bind(lib):
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_score_round.argtypes = [i32, i32, P, P, P, P, P, P, P, dbl, i32, P, i64, i32,
                                       P, i32, P, P, P, ctypes.c_int]
    lib.oracle_policy_step.argtypes = [ctypes.c_int, i32, i32, i32, i32, P, P, P, P, P, P, P, P,
                                       P, i32, P, P, P, P, P, P, ctypes.c_int]
    lib.oracle_topk.argtypes = [P, i64, i32, i64, P, P]
    lib.oracle_merge.argtypes = [P, P, i32, P, i64, i64]
    lib.oracle_track_advantage.argtypes = [P, P, P, P, i64, dbl, dbl, P, P, P]
    lib.oracle_track_eliminate.argtypes = [P, i64, i64, P]
    lib.oracle_philox4x32.argtypes = [P, P, P]
    lib.oracle_philox4x32.restype = None
    lib.oracle_policy_select.argtypes = [P, i64, i32, P, i32, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, P, P, P]
    lib.oracle_gbdt_bin.argtypes = [P, i64, i32, i64, P, i32, P, i64, P]
    lib.oracle_gbdt_round.argtypes = [P, i64, i32, i64, P, i32, P, P, i64, P, P, dbl, i32, dbl, dbl, dbl, dbl,
                                      P, P, P, P, P, P, P, P]
    lib.oracle_max_threads.argtypes = []
    lib.oracle_round_bf16.argtypes = [dbl]
    lib.oracle_round_bf16.restype = dbl
    for f in (lib.oracle_score_round, lib.oracle_policy_step, lib.oracle_topk,
              lib.oracle_merge, lib.oracle_max_threads, lib.oracle_track_advantage,
              lib.oracle_track_eliminate, lib.oracle_policy_select, lib.oracle_gbdt_bin, lib.oracle_gbdt_round):
        f.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build(force=True)
        with _lock:
            if _lib is None:
                _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


def use_library(path: str | None):
    """Point this wrapper at another build of the oracle source (the tests use this to check that
    their pins reject deliberately broken copies); ``None`` restores the default build."""
    global _lib
    with _lock:
        _lib = None if path is None else _bind(ctypes.CDLL(path))


def round_bf16(v: float) -> float:
    """The oracle's fp64 -> bf16 rounding (nearest, ties to even), returned as a float."""
    return float(_load().oracle_round_bf16(float(v)))


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def score_round(ens: dict, features: np.ndarray, prog_ptr: np.ndarray, n_rows: int | None = None,
                threads: int = 0) -> dict:
    """Cost-model scores of every program (GBDT per statement row, summed per program).

    ``features`` is the feature-major matrix ``[n_features][ld]``.  Returns fp64 ``prog`` and
    ``stmt`` scores, their fp32 roundings ``prog32`` / ``stmt32``, and ``scale`` (sum of |terms|
    per program, the basis of the scale-relative tolerance).
    """
    lib = _load()
    X = _c(features, np.float32)
    ptr = _c(prog_ptr, np.int32)
    n_prog = ptr.size - 1
    n_rows = int(ptr[-1]) if n_rows is None else n_rows
    arrs = dict(root=_c(ens["root"], np.int32), feature=_c(ens["feature"], np.int32),
                threshold=_c(ens["threshold"], np.float32), left=_c(ens["left"], np.int32),
                right=_c(ens["right"], np.int32), default_left=_c(ens["default_left"], np.uint8),
                leaf_value=_c(ens["leaf_value"], np.float32))
    prog = np.zeros(n_prog, dtype=np.float64)
    stmt = np.zeros(n_rows, dtype=np.float64)
    scale = np.zeros(n_prog, dtype=np.float64)
    rc = lib.oracle_score_round(int(ens["n_trees"]), arrs["feature"].size, _p(arrs["root"]),
                                _p(arrs["feature"]), _p(arrs["threshold"]), _p(arrs["left"]),
                                _p(arrs["right"]), _p(arrs["default_left"]), _p(arrs["leaf_value"]),
                                float(ens.get("base_score", 0.0)), int(ens["n_features"]), _p(X),
                                X.shape[1], n_rows, _p(ptr), n_prog, _p(prog), _p(stmt), _p(scale),
                                threads)
    if rc != 0:
        raise ValueError("oracle_score_round failed (%d): malformed input" % rc)
    return dict(prog=prog, stmt=stmt, scale=scale, prog32=prog.astype(np.float32),
                stmt32=stmt.astype(np.float32))


def policy_step(pol: dict, states: np.ndarray, threads: int = 0, want_probs: bool = True) -> dict:
    """Actor/critic forward for every state: action (lowest-index argmax of the logits), value,
    logits, softmax probabilities and per-output tolerance scales (fp64)."""
    lib = _load()
    dt = 1 if pol["dtype"] == "bf16" else 0
    wdt = np.uint16 if dt else np.float32
    S, H1, H2, A = int(pol["s"]), int(pol["h1"]), int(pol["h2"]), int(pol["a"])
    st = _c(states, wdt)
    B = st.shape[0]
    assert st.shape == (B, S)
    w = {k: _c(pol[k], wdt) for k in ("w1", "w2", "wa", "wv")}
    b = {k: _c(pol[k], np.float32) for k in ("b1", "b2", "ba", "bv")}
    action = np.zeros(B, dtype=np.int32)
    value = np.zeros(B, dtype=np.float64)
    logits = np.zeros((B, A), dtype=np.float64)
    probs = np.zeros((B, A), dtype=np.float64) if want_probs else None
    lscale = np.zeros((B, A), dtype=np.float64)
    vscale = np.zeros(B, dtype=np.float64)
    rc = lib.oracle_policy_step(dt, S, H1, H2, A, _p(w["w1"]), _p(b["b1"]), _p(w["w2"]), _p(b["b2"]),
                                _p(w["wa"]), _p(b["ba"]), _p(w["wv"]), _p(b["bv"]), _p(st), B,
                                _p(action), _p(value), _p(logits), _p(probs), _p(lscale), _p(vscale),
                                threads)
    if rc != 0:
        raise ValueError("oracle_policy_step failed (%d)" % rc)
    return dict(action=action, value=value, logits=logits, probs=probs, logit_scale=lscale,
                value_scale=vscale)


def topk(score: np.ndarray, k: int, index_base: int = 0):
    """The k best scores ranked by (score desc, index asc); returns (scores fp32, indices int64)."""
    lib = _load()
    s = _c(score, np.float32)
    out_s = np.zeros(k, dtype=np.float32)
    out_i = np.zeros(k, dtype=np.int64)
    rc = lib.oracle_topk(_p(s), s.size, k, index_base, _p(out_s), _p(out_i))
    if rc != 0:
        raise ValueError("oracle_topk failed (%d)" % rc)
    return out_s, out_i


RESET_SCORE = np.float32(-np.inf)
RESET_INDEX = np.int64(np.iinfo(np.int64).max)


def reset(k: int):
    """An empty running heap of capacity k: every slot (-inf, INT64_MAX)."""
    return np.full(k, RESET_SCORE, dtype=np.float32), np.full(k, RESET_INDEX, dtype=np.int64)


def merge(run_score: np.ndarray, run_index: np.ndarray, score: np.ndarray, index_base: int):
    """running <- top-k(running U {(score[i], index_base + i)}); returns new (scores, indices)."""
    lib = _load()
    rs = np.array(run_score, dtype=np.float32, copy=True)
    ri = np.array(run_index, dtype=np.int64, copy=True)
    s = _c(score, np.float32)
    rc = lib.oracle_merge(_p(rs), _p(ri), rs.size, _p(s), s.size, index_base)
    if rc != 0:
        raise ValueError("oracle_merge failed (%d)" % rc)
    return rs, ri


def track_advantage(c_prev, c_next, v_prev, v_next, gamma: float = 0.9, eps: float = 1e-6) -> dict:
    """Reward (Algorithm 1, denominator max(|C(s)|, eps)) and advantage (Eq. 6) of one step of
    every schedule track, fp64 over the fp32 inputs; ``scale`` = |r| + |gamma V(s')| + |V(s)|.
    ``gamma`` and ``eps`` are taken at their fp32 values (the values the GPU path computes with)."""
    lib = _load()
    a = [_c(x, np.float32) for x in (c_prev, c_next, v_prev, v_next)]
    n = a[0].size
    assert all(x.size == n for x in a)
    reward = np.zeros(n, dtype=np.float64)
    adv = np.zeros(n, dtype=np.float64)
    scale = np.zeros(n, dtype=np.float64)
    rc = lib.oracle_track_advantage(*[_p(x) for x in a], n, float(np.float32(gamma)), float(np.float32(eps)),
                                    _p(reward), _p(adv), _p(scale))
    if rc != 0:
        raise ValueError("oracle_track_advantage failed (%d)" % rc)
    return dict(reward=reward, adv=adv, scale=scale)


def track_eliminate(adv, n_keep: int) -> np.ndarray:
    """Adaptive-stopping elimination (Section 5): the indices of the n_keep tracks ranked first by
    (advantage desc, NaN last, -0 ties +0, lower index first), in ascending order."""
    lib = _load()
    a = _c(adv, np.float32)
    out = np.zeros(max(n_keep, 0), dtype=np.int32)
    rc = lib.oracle_track_eliminate(_p(a), a.size, n_keep, _p(out))
    if rc != 0:
        raise ValueError("oracle_track_eliminate failed (%d)" % rc)
    return out


def eliminate_count(n: int, rho: float = 0.5) -> int:
    """Tracks that survive one elimination of proportion rho (Section 5): the eliminated number
    floor(rho * n) is rounded down."""
    return n - int(np.floor(rho * n))


def philox4x32(counter, key) -> list:
    """Philox4x32-10 of a 4-word counter and a 2-word key (the published generator)."""
    lib = _load()
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib.oracle_philox4x32(_p(c), _p(k), _p(out))
    return [int(x) for x in out]


def policy_select(logits, seg_offsets, sample: bool = False, seed: int = 0, counter: int = 0) -> dict:
    """One action per modification type (segment of the logits row): greedy or Gumbel-max sampled;
    returns action [B][n_seg] int32, logp [B][n_seg] and probs [B][a] (fp64)."""
    lib = _load()
    z = _c(logits, np.float32)
    B, a = z.shape
    off = _c(seg_offsets, np.int32)
    n_seg = off.size - 1
    action = np.zeros((B, n_seg), dtype=np.int32)
    logp = np.zeros((B, n_seg), dtype=np.float64)
    probs = np.zeros((B, a), dtype=np.float64)
    rc = lib.oracle_policy_select(_p(z), B, a, _p(off), n_seg, int(bool(sample)), seed, counter, _p(action),
                                  _p(logp), _p(probs))
    if rc != 0:
        raise ValueError("oracle_policy_select failed (%d)" % rc)
    return dict(action=action, logp=logp, probs=probs)


# Ansor's XGBoost settings for the cost model (eta, max_depth, gamma, min_child_weight) with
# XGBoost's default L2 regularisation lambda = 1.
GBDT_DEFAULTS = dict(max_depth=10, eta=0.2, reg_lambda=1.0, gamma=0.001, min_child_weight=0.0, base_score=0.0)


def gbdt_bin(x_fm, n_rows: int, cuts, n_cuts, ld: int) -> np.ndarray:
    """Bins [n_rows][ld] uint8 of feature-major values x_fm [F][ldx]: the number of cut points of
    the feature that are <= x, 255 for NaN, padding bytes 0."""
    lib = _load()
    x = _c(x_fm, np.float32)
    F, ldx = x.shape
    cu = _c(cuts, np.float32)
    nc = _c(n_cuts, np.int32)
    out = np.zeros((n_rows, ld), dtype=np.uint8)
    rc = lib.oracle_gbdt_bin(_p(x), n_rows, F, ldx, _p(cu), cu.shape[1], _p(nc), ld, _p(out))
    if rc != 0:
        raise ValueError("oracle_gbdt_bin failed (%d)" % rc)
    return out


def gbdt_bin_np(x_fm, n_rows: int, cuts, n_cuts, ld: int) -> np.ndarray:
    """The same bins as ``gbdt_bin`` with numpy's ``searchsorted`` (side="right": the number of cut
    points <= x) as the counting step, for row counts the plain C count is too slow for."""
    x = np.asarray(x_fm, dtype=np.float32)
    F = x.shape[0]
    out = np.zeros((n_rows, ld), dtype=np.uint8)
    for f in range(F):
        v = x[f, :n_rows]
        b = np.searchsorted(np.asarray(cuts[f, :int(n_cuts[f])], np.float32), v, side="right")
        b[np.isnan(v)] = 255
        out[:, f] = b
    return out


def gbdt_round(bins, F: int, cuts, n_cuts, prog_ptr, label, weight, margin, max_depth=10, eta=0.2,
               reg_lambda=1.0, gamma=0.001, min_child_weight=0.0, base_score=0.0) -> dict:
    """One boosting round under the pack-sum squared error; returns the tree (heap-numbered node
    arrays), the updated margins and the fixed-point exponents."""
    lib = _load()
    b = _c(bins, np.uint8)
    N, ld = b.shape
    cu = _c(cuts, np.float32)
    nc = _c(n_cuts, np.int32)
    pp = _c(prog_ptr, np.int32)
    P = pp.size - 1
    y = _c(label, np.float32)
    w = _c(weight, np.float32)
    m = np.array(margin, dtype=np.float32, copy=True)
    n_nodes = (1 << (max_depth + 1)) - 1
    feature = np.zeros(n_nodes, np.int32)
    threshold = np.zeros(n_nodes, np.float32)
    left = np.zeros(n_nodes, np.int32)
    right = np.zeros(n_nodes, np.int32)
    dl = np.zeros(n_nodes, np.uint8)
    leaf = np.zeros(n_nodes, np.float32)
    exps = np.zeros(2, np.int32)
    rc = lib.oracle_gbdt_round(_p(b), N, F, ld, _p(cu), cu.shape[1], _p(nc), _p(pp), P, _p(y), _p(w),
                               float(base_score), int(max_depth), float(eta), float(reg_lambda), float(gamma),
                               float(min_child_weight), _p(m), _p(feature), _p(threshold), _p(left), _p(right),
                               _p(dl), _p(leaf), _p(exps))
    if rc != 0:
        raise ValueError("oracle_gbdt_round failed (%d)" % rc)
    return dict(feature=feature, threshold=threshold, left=left, right=right, default_left=dl, leaf_value=leaf,
                margin=m, exps=exps)
