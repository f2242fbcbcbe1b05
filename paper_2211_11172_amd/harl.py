"""Thin ctypes binding of libharl (include/harl.h): same names, argument marshalling only.

Every computation runs in the HIP kernels behind the C ABI.  Device buffers are passed as torch
tensors (their ``data_ptr()``) or raw integer addresses; streams as torch streams, raw
``hipStream_t`` integers, or ``None`` for torch's current stream.  Loading fails loudly when the
library has not been built (``python -m paper_2211_11172_amd.build``): there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libharl.so")

HARL_OK, HARL_E_INVALID_ARG, HARL_E_UNSUPPORTED, HARL_E_WORKSPACE, HARL_E_HIP, HARL_E_NOMEM = 0, -1, -2, -3, -4, -5
HARL_F32, HARL_BF16 = 0, 1
HARL_TOPK_MAX_K = 2048
HARL_TOPK_MERGE = 1
HARL_SELECT_MAX_SEGMENTS = 32
HARL_SELECT_SAMPLE = 1

# every entry point declared in include/harl.h
EXPORTS = (
    "harl_last_error", "harl_version",
    "harl_ensemble_create", "harl_ensemble_destroy", "harl_ensemble_info",
    "harl_score_round_workspace_size", "harl_score_round",
    "harl_policy_create", "harl_policy_destroy", "harl_policy_step",
    "harl_topk_workspace_size", "harl_topk", "harl_topk_reset", "harl_topk_static",
    "harl_policy_select",
    "harl_ppo_param_count", "harl_ppo_workspace_size", "harl_ppo_update",
    "harl_track_advantage", "harl_track_keep_count", "harl_track_eliminate_workspace_size", "harl_track_eliminate",
    "harl_gbdt_bin", "harl_gbdt_round_workspace_size", "harl_gbdt_round",
)
HARL_GBDT_MAX_DEPTH = 12
HARL_GBDT_MAX_CUTS = 254
HARL_GBDT_MAX_FEATURES = 4096


class PpoConfig(ctypes.Structure):
    _fields_ = [("s", ctypes.c_int32), ("h1", ctypes.c_int32), ("h2", ctypes.c_int32), ("a", ctypes.c_int32),
                ("n_seg", ctypes.c_int32), ("seg_offsets", ctypes.c_int32 * (HARL_SELECT_MAX_SEGMENTS + 1)),
                ("clip_eps", ctypes.c_float), ("w_value", ctypes.c_float), ("w_entropy", ctypes.c_float),
                ("lr_actor", ctypes.c_float), ("lr_critic", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float)]


def ppo_config(s: int, h1: int, h2: int, a: int, segs, clip_eps=0.2, w_value=0.5, w_entropy=0.01, lr_actor=3e-4,
               lr_critic=1e-3, beta1=0.9, beta2=0.999, adam_eps=1e-8) -> PpoConfig:
    c = PpoConfig()
    c.s, c.h1, c.h2, c.a, c.n_seg = s, h1, h2, a, len(segs) - 1
    for i, o in enumerate(segs):
        c.seg_offsets[i] = int(o)
    c.clip_eps, c.w_value, c.w_entropy = clip_eps, w_value, w_entropy
    c.lr_actor, c.lr_critic, c.beta1, c.beta2, c.adam_eps = lr_actor, lr_critic, beta1, beta2, adam_eps
    return c


class GbdtParams(ctypes.Structure):
    _fields_ = [("max_depth", ctypes.c_int32), ("eta", ctypes.c_double), ("reg_lambda", ctypes.c_double),
                ("gamma", ctypes.c_double), ("min_child_weight", ctypes.c_double), ("base_score", ctypes.c_double)]


def gbdt_params(max_depth=10, eta=0.2, reg_lambda=1.0, gamma=0.001, min_child_weight=0.0, base_score=0.0) -> GbdtParams:
    """Boosting hyper-parameters; the defaults are Ansor's cost-model settings with XGBoost's lambda."""
    p = GbdtParams()
    p.max_depth, p.eta, p.reg_lambda, p.gamma, p.min_child_weight, p.base_score = (
        max_depth, eta, reg_lambda, gamma, min_child_weight, base_score)
    return p


class HarlError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__("%s failed (status %d): %s" % (where, status, message))
        self.status = status


class _EnsembleDesc(ctypes.Structure):
    _fields_ = [("n_trees", ctypes.c_int32), ("n_features", ctypes.c_int32), ("n_nodes", ctypes.c_int32),
                ("root", ctypes.c_void_p), ("feature", ctypes.c_void_p), ("threshold", ctypes.c_void_p),
                ("left", ctypes.c_void_p), ("right", ctypes.c_void_p), ("default_left", ctypes.c_void_p),
                ("leaf_value", ctypes.c_void_p), ("base_score", ctypes.c_float)]


class _PolicyDesc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("s", ctypes.c_int32), ("h1", ctypes.c_int32), ("h2", ctypes.c_int32),
                ("a", ctypes.c_int32), ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
                ("b2", ctypes.c_void_p), ("wa", ctypes.c_void_p), ("ba", ctypes.c_void_p), ("wv", ctypes.c_void_p),
                ("bv", ctypes.c_void_p)]


_lock = threading.Lock()
_lib = None


def load():
    """Load libharl.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError("libharl.so is not built (%s); run `python -m paper_2211_11172_amd.build`" % LIB_PATH)
            lib = ctypes.CDLL(LIB_PATH)
            P, i32, i64, sz, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_uint32
            sig = {
                "harl_last_error": ([], ctypes.c_char_p),
                "harl_version": ([], ctypes.c_char_p),
                "harl_ensemble_create": ([P, P, P], ctypes.c_int),
                "harl_ensemble_destroy": ([P], ctypes.c_int),
                "harl_ensemble_info": ([P, P, P, P], ctypes.c_int),
                "harl_score_round_workspace_size": ([P, i32, i32], sz),
                "harl_score_round": ([P, P, i64, i32, P, i32, P, P, P, sz, P], ctypes.c_int),
                "harl_policy_create": ([P, P, P], ctypes.c_int),
                "harl_policy_destroy": ([P], ctypes.c_int),
                "harl_policy_step": ([P, P, i32, P, P, P, P, P], ctypes.c_int),
                "harl_topk_workspace_size": ([i32, i32], sz),
                "harl_topk": ([P, i32, i32, i64, P, P, u32, P, sz, P], ctypes.c_int),
                "harl_topk_reset": ([P, P, i32, P], ctypes.c_int),
                "harl_topk_static": ([P, i32, i32, i64, P, P, u32, P], ctypes.c_int),
                "harl_ppo_param_count": ([P], sz),
                "harl_ppo_workspace_size": ([P, i32], sz),
                "harl_ppo_update": ([P, P, P, P, i32, P, P, P, P, P, i32, P, P, P, sz, P], ctypes.c_int),
                "harl_policy_select": ([P, i32, i32, P, i32, u32, ctypes.c_uint64, ctypes.c_uint64, P, P, P, P],
                                       ctypes.c_int),
                "harl_track_advantage": ([P, P, P, P, i32, ctypes.c_float, ctypes.c_float, P, P, P], ctypes.c_int),
                "harl_track_keep_count": ([i32, ctypes.c_double, P], ctypes.c_int),
                "harl_track_eliminate_workspace_size": ([i32], sz),
                "harl_track_eliminate": ([P, i32, i32, P, P, i64, P, P, sz, P], ctypes.c_int),
                "harl_gbdt_bin": ([P, i64, i32, i32, P, i32, P, P, i64, P], ctypes.c_int),
                "harl_gbdt_round_workspace_size": ([P, i32, i32, i32], sz),
                "harl_gbdt_round": ([P, P, i64, i32, i32, P, i32, P, P, i32, P, P, P, P, P, P, P, P, P, P, sz, P],
                                    ctypes.c_int),
            }
            for name, (args, res) in sig.items():
                f = getattr(lib, name)
                f.argtypes, f.restype = args, res
            _lib = lib
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def harl_last_error() -> str:
    return load().harl_last_error().decode()


def harl_version() -> str:
    return load().harl_version().decode()


def _check(rc: int, where: str):
    if rc != HARL_OK:
        raise HarlError(rc, where, harl_last_error())


# ------------------------------------------------------------------------------------------------
# cost model
# ------------------------------------------------------------------------------------------------
class Ensemble:
    """A library-owned packed GBDT (see harl_ensemble_create)."""

    def __init__(self, handle: int):
        self.handle = handle
        t, d, f = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(load().harl_ensemble_info(handle, ctypes.byref(t), ctypes.byref(d), ctypes.byref(f)), "harl_ensemble_info")
        self.n_trees, self.depth, self.n_features = t.value, d.value, f.value

    def close(self):
        if self.handle:
            _check(load().harl_ensemble_destroy(self.handle), "harl_ensemble_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def harl_ensemble_create(ens: dict, stream=0) -> Ensemble:
    """Pack a host ensemble given as explicit node arrays (keys of harl_ensemble_desc)."""
    arrs = dict(root=np.ascontiguousarray(ens["root"], np.int32), feature=np.ascontiguousarray(ens["feature"], np.int32),
                threshold=np.ascontiguousarray(ens["threshold"], np.float32),
                left=np.ascontiguousarray(ens["left"], np.int32), right=np.ascontiguousarray(ens["right"], np.int32),
                default_left=np.ascontiguousarray(ens["default_left"], np.uint8),
                leaf_value=np.ascontiguousarray(ens["leaf_value"], np.float32))
    d = _EnsembleDesc(int(ens["n_trees"]), int(ens["n_features"]), int(arrs["feature"].size),
                      *[arrs[k].ctypes.data for k in ("root", "feature", "threshold", "left", "right", "default_left",
                                                      "leaf_value")],
                      float(ens.get("base_score", 0.0)))
    h = ctypes.c_void_p()
    _check(load().harl_ensemble_create(ctypes.byref(d), ctypes.byref(h), _stream(stream)), "harl_ensemble_create")
    return Ensemble(h.value)


def harl_score_round_workspace_size(ens: Ensemble, n_rows: int, n_prog: int) -> int:
    return int(load().harl_score_round_workspace_size(ens.handle, n_rows, n_prog))


def harl_score_round(ens: Ensemble, feat, ld: int, n_rows: int, prog_ptr, n_prog: int, prog_score, stmt_score,
                     ws, ws_bytes: int, stream=None):
    _check(load().harl_score_round(ens.handle, _ptr(feat), ld, n_rows, _ptr(prog_ptr), n_prog, _ptr(prog_score),
                                   _ptr(stmt_score), _ptr(ws), ws_bytes, _stream(stream)), "harl_score_round")


# ------------------------------------------------------------------------------------------------
# actor / critic
# ------------------------------------------------------------------------------------------------
class Policy:
    """A library-owned pre-tiled actor/critic (see harl_policy_create)."""

    def __init__(self, handle: int, dtype: int, s: int, h1: int, h2: int, a: int):
        self.handle, self.dtype, self.s, self.h1, self.h2, self.a = handle, dtype, s, h1, h2, a

    def close(self):
        if self.handle:
            _check(load().harl_policy_destroy(self.handle), "harl_policy_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def harl_policy_create(pol: dict, stream=0) -> Policy:
    """Pre-tile host weights: keys dtype ("f32"/"bf16"), s, h1, h2, a, w1, b1, w2, b2, wa, ba, wv, bv."""
    bf = pol["dtype"] == "bf16"
    wdt = np.uint16 if bf else np.float32
    w = {k: np.ascontiguousarray(pol[k], wdt) for k in ("w1", "w2", "wa", "wv")}
    b = {k: np.ascontiguousarray(pol[k], np.float32) for k in ("b1", "b2", "ba", "bv")}
    d = _PolicyDesc(HARL_BF16 if bf else HARL_F32, int(pol["s"]), int(pol["h1"]), int(pol["h2"]), int(pol["a"]),
                    w["w1"].ctypes.data, b["b1"].ctypes.data, w["w2"].ctypes.data, b["b2"].ctypes.data,
                    w["wa"].ctypes.data, b["ba"].ctypes.data, w["wv"].ctypes.data, b["bv"].ctypes.data)
    h = ctypes.c_void_p()
    _check(load().harl_policy_create(ctypes.byref(d), ctypes.byref(h), _stream(stream)), "harl_policy_create")
    return Policy(h.value, d.dtype, d.s, d.h1, d.h2, d.a)


def harl_policy_step(pol: Policy, states, B: int, action, value, probs=None, logits=None, stream=None):
    _check(load().harl_policy_step(pol.handle, _ptr(states), B, _ptr(action), _ptr(value), _ptr(probs), _ptr(logits),
                                   _stream(stream)), "harl_policy_step")


# ------------------------------------------------------------------------------------------------
# top-K and the running heap
# ------------------------------------------------------------------------------------------------
def harl_topk_workspace_size(n: int, k: int) -> int:
    return int(load().harl_topk_workspace_size(n, k))


def harl_topk(score, n: int, k: int, index_base: int, io_score, io_index, flags: int, ws, ws_bytes: int, stream=None):
    _check(load().harl_topk(_ptr(score), n, k, index_base, _ptr(io_score), _ptr(io_index), flags, _ptr(ws), ws_bytes,
                            _stream(stream)), "harl_topk")


def harl_topk_static(score, n: int, k: int, index_base: int, io_score, io_index, flags: int, stream=None):
    _check(load().harl_topk_static(_ptr(score), n, k, index_base, _ptr(io_score), _ptr(io_index), flags,
                                   _stream(stream)), "harl_topk_static")


HARL_TOPK_STATIC_SCRATCH_BYTES = 8 << 20


def harl_topk_reset(io_score, io_index, k: int, stream=None):
    _check(load().harl_topk_reset(_ptr(io_score), _ptr(io_index), k, _stream(stream)), "harl_topk_reset")


def harl_policy_select(logits, B: int, a: int, seg_offsets, flags: int, seed: int, counter: int, action, logp=None,
                       probs=None, stream=None):
    """seg_offsets: host sequence [n_seg + 1] (0 .. a)."""
    off = np.ascontiguousarray(seg_offsets, np.int32)
    _check(load().harl_policy_select(_ptr(logits), B, a, off.ctypes.data, off.size - 1, flags, seed, counter,
                                     _ptr(action), _ptr(logp), _ptr(probs), _stream(stream)), "harl_policy_select")


def harl_ppo_param_count(cfg: PpoConfig) -> int:
    return int(load().harl_ppo_param_count(ctypes.byref(cfg)))


def harl_ppo_workspace_size(cfg: PpoConfig, M: int) -> int:
    return int(load().harl_ppo_workspace_size(ctypes.byref(cfg), M))


def harl_ppo_update(cfg: PpoConfig, params, adam_m, adam_v, step: int, states, actions, logp_old, adv, ret, M: int,
                    grad=None, loss=None, ws=None, ws_bytes: int = 0, stream=None):
    _check(load().harl_ppo_update(ctypes.byref(cfg), _ptr(params), _ptr(adam_m), _ptr(adam_v), step, _ptr(states),
                                  _ptr(actions), _ptr(logp_old), _ptr(adv), _ptr(ret), M, _ptr(grad), _ptr(loss),
                                  _ptr(ws), ws_bytes, _stream(stream)), "harl_ppo_update")


# ------------------------------------------------------------------------------------------------
# schedule tracks
# ------------------------------------------------------------------------------------------------
def harl_track_advantage(c_prev, c_next, v_prev, v_next, n: int, gamma: float, eps: float, reward, adv, stream=None):
    _check(load().harl_track_advantage(_ptr(c_prev), _ptr(c_next), _ptr(v_prev), _ptr(v_next), n, gamma, eps,
                                       _ptr(reward), _ptr(adv), _stream(stream)), "harl_track_advantage")


def harl_track_eliminate_workspace_size(n: int) -> int:
    return int(load().harl_track_eliminate_workspace_size(n))


def harl_track_eliminate(adv, n: int, n_keep: int, keep_index, rows=None, row_bytes: int = 0, rows_out=None, ws=None,
                         ws_bytes: int = 0, stream=None):
    _check(load().harl_track_eliminate(_ptr(adv), n, n_keep, _ptr(keep_index), _ptr(rows), row_bytes, _ptr(rows_out),
                                       _ptr(ws), ws_bytes, _stream(stream)), "harl_track_eliminate")


def harl_track_keep_count(n: int, rho: float = 0.5) -> int:
    out = ctypes.c_int32(0)
    _check(load().harl_track_keep_count(n, ctypes.c_double(rho), ctypes.byref(out)), "harl_track_keep_count")
    return int(out.value)


# ------------------------------------------------------------------------------------------------
# cost-model refit
# ------------------------------------------------------------------------------------------------
def harl_gbdt_bin(feat, ld_feat: int, n_features: int, n_rows: int, cuts, cut_stride: int, n_cuts, bins,
                  ld_bins: int, stream=None):
    _check(load().harl_gbdt_bin(_ptr(feat), ld_feat, n_features, n_rows, _ptr(cuts), cut_stride, _ptr(n_cuts),
                                _ptr(bins), ld_bins, _stream(stream)), "harl_gbdt_bin")


def harl_gbdt_round_workspace_size(prm: GbdtParams, n_features: int, n_rows: int, n_prog: int) -> int:
    return int(load().harl_gbdt_round_workspace_size(ctypes.byref(prm), n_features, n_rows, n_prog))


def harl_gbdt_round(prm: GbdtParams, bins, ld_bins: int, n_features: int, n_rows: int, cuts, cut_stride: int, n_cuts,
                    prog_ptr, n_prog: int, label, weight, margin, feature, threshold, left, right, default_left,
                    leaf_value, ws, ws_bytes: int, stream=None):
    _check(load().harl_gbdt_round(ctypes.byref(prm), _ptr(bins), ld_bins, n_features, n_rows, _ptr(cuts), cut_stride,
                                  _ptr(n_cuts), _ptr(prog_ptr), n_prog, _ptr(label), _ptr(weight), _ptr(margin),
                                  _ptr(feature), _ptr(threshold), _ptr(left), _ptr(right), _ptr(default_left),
                                  _ptr(leaf_value), _ptr(ws), ws_bytes, _stream(stream)), "harl_gbdt_round")
