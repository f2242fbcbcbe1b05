"""The C ABI on a host without a GPU: the library loads, exports every symbol include/harl.h
declares, and rejects bad host-visible arguments before any HIP call (no compute calls)."""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2211_11172_amd import harl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "harl.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(harl_\w+)\s*\(", src)))


def test_exports_every_declared_symbol():
    lib = ctypes.CDLL(harl.LIB_PATH)
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), "libharl.so does not export %s" % n
    assert sorted(harl.EXPORTS) == names


def test_version_and_last_error():
    assert harl.harl_version().startswith("harl")
    assert isinstance(harl.harl_last_error(), str)


def _status(fn, *args):
    return getattr(harl.load(), fn)(*args)


def test_track_keep_count_matches_the_oracle_rule():
    """Host-only arithmetic behind the ABI: n - floor(rho n) tracks survive (Section 5)."""
    import oracle
    for n in (0, 1, 2, 3, 7, 64, 65, 100, 4095, 4096, 65537, 1048653, 2**31 - 1):
        for rho in (0.0, 0.25, 0.3, 0.5, 0.75, 0.999, 1.0):
            assert harl.harl_track_keep_count(n, rho) == oracle.eliminate_count(n, rho), (n, rho)
    out = ctypes.c_int32(0)
    lib = harl.load()
    assert lib.harl_track_keep_count(-1, ctypes.c_double(0.5), ctypes.byref(out)) == harl.HARL_E_INVALID_ARG
    assert lib.harl_track_keep_count(10, ctypes.c_double(1.5), ctypes.byref(out)) == harl.HARL_E_INVALID_ARG
    assert lib.harl_track_keep_count(10, ctypes.c_double(float("nan")), ctypes.byref(out)) == harl.HARL_E_INVALID_ARG
    assert lib.harl_track_keep_count(10, ctypes.c_double(0.5), None) == harl.HARL_E_INVALID_ARG


def test_topk_argument_errors():
    assert _status("harl_topk", None, 10, 11, 0, None, None, 0, None, 0, None) == harl.HARL_E_INVALID_ARG
    assert "k > n" in harl.harl_last_error()
    assert _status("harl_topk", None, 10, 5000, 0, None, None, 1, None, 0, None) == harl.HARL_E_UNSUPPORTED
    assert _status("harl_topk", None, 10, 5, 0, None, None, 4, None, 0, None) == harl.HARL_E_INVALID_ARG
    assert _status("harl_topk", None, 10, 5, -1, None, None, 0, None, 0, None) == harl.HARL_E_INVALID_ARG
    assert _status("harl_topk", None, -1, 5, 0, None, None, 0, None, 0, None) == harl.HARL_E_INVALID_ARG
    # misaligned outputs, null scores and a short workspace are caught before any launch
    assert _status("harl_topk", 0x1000, 10, 5, 0, 0x1001, 0x2000, 0, 0x3000, 1 << 20, None) == harl.HARL_E_INVALID_ARG
    assert _status("harl_topk", None, 10, 5, 0, 0x1000, 0x2000, 0, 0x3000, 1 << 20, None) == harl.HARL_E_INVALID_ARG
    assert _status("harl_topk", 0x1000, 10, 5, 0, 0x1000, 0x2000, 0, 0x3000, 8, None) == harl.HARL_E_WORKSPACE
    assert _status("harl_topk", 0x1000, 10, 5, 0, 0x1000, 0x2000, 0, 0x3001, 1 << 20, None) == harl.HARL_E_INVALID_ARG
    # k == 0 and (MERGE with n == 0) are valid no-ops
    assert _status("harl_topk", None, 0, 0, 0, None, None, 0, None, 0, None) == harl.HARL_OK
    assert _status("harl_topk", None, 0, 4, 0, 0x1000, 0x2000, 1, None, 0, None) == harl.HARL_OK
    assert _status("harl_topk_reset", None, None, 3, None) == harl.HARL_E_INVALID_ARG
    assert _status("harl_topk_reset", None, None, 0, None) == harl.HARL_OK


def test_score_round_argument_errors():
    assert _status("harl_score_round", None, None, 0, 0, None, 1, None, None, None, 0, None) == harl.HARL_E_INVALID_ARG
    assert harl.harl_score_round_workspace_size(type("E", (), {"handle": None})(), 10, 1) == 0


def _ens_dict(**over):
    d = dict(n_trees=1, n_features=2, root=np.array([0], np.int32), feature=np.array([1, -1, -1], np.int32),
             threshold=np.array([0.5, 0, 0], np.float32), left=np.array([1, -1, -1], np.int32),
             right=np.array([2, -1, -1], np.int32), default_left=np.zeros(3, np.uint8),
             leaf_value=np.array([0, 1, 2], np.float32), base_score=0.0)
    d.update(over)
    return d


@pytest.mark.parametrize("over,status", [
    (dict(feature=np.array([5, -1, -1], np.int32)), harl.HARL_E_INVALID_ARG),      # feature >= n_features
    (dict(left=np.array([0, -1, -1], np.int32)), harl.HARL_E_INVALID_ARG),         # a cycle
    (dict(right=np.array([9, -1, -1], np.int32)), harl.HARL_E_INVALID_ARG),        # child out of range
    (dict(root=np.array([3], np.int32)), harl.HARL_E_INVALID_ARG),                 # root out of range
    (dict(n_features=1000), harl.HARL_E_UNSUPPORTED),                              # feature tile too big
    (dict(n_trees=0, root=np.zeros(0, np.int32)), harl.HARL_E_INVALID_ARG),
])
def test_ensemble_validation(over, status):
    with pytest.raises(harl.HarlError) as e:
        harl.harl_ensemble_create(_ens_dict(**over), stream=0)
    assert e.value.status == status


def test_too_deep_tree_unsupported():
    D = 13   # a chain of 13 splits
    n = 2 * D + 1
    feature = np.full(n, -1, np.int32)
    left = np.full(n, -1, np.int32)
    right = np.full(n, -1, np.int32)
    for i in range(D):
        feature[i] = 0
        left[i] = i + 1 if i + 1 < D else D
        right[i] = D + 1 + i
    d = _ens_dict(feature=feature, left=left, right=right, threshold=np.zeros(n, np.float32),
                  default_left=np.zeros(n, np.uint8), leaf_value=np.ones(n, np.float32))
    with pytest.raises(harl.HarlError) as e:
        harl.harl_ensemble_create(d, stream=0)
    assert e.value.status == harl.HARL_E_UNSUPPORTED


@pytest.mark.parametrize("over", [dict(dtype="f32", s=0), dict(dtype="f32", a=128), dict(dtype="f32", h1=5000)])
def test_policy_validation(over):
    p = dict(dtype="f32", s=4, h1=8, h2=8, a=3)
    p.update(over)
    for k, shape in (("w1", (8, 4)), ("w2", (8, 8)), ("wa", (3, 8)), ("wv", (1, 8))):
        p[k] = np.zeros(shape, np.float32)
    for k, m in (("b1", 8), ("b2", 8), ("ba", 3), ("bv", 1)):
        p[k] = np.zeros(m, np.float32)
    with pytest.raises(harl.HarlError) as e:
        harl.harl_policy_create(p, stream=0)
    assert e.value.status == harl.HARL_E_INVALID_ARG


def test_policy_step_argument_errors():
    assert _status("harl_policy_step", None, None, 4, None, None, None, None, None) == harl.HARL_E_INVALID_ARG


def test_track_argument_errors():
    F = ctypes.c_float
    adv = lambda *a: _status("harl_track_advantage", *a)
    assert adv(None, None, None, None, -1, F(0.9), F(1e-6), None, None, None) == harl.HARL_E_INVALID_ARG
    assert adv(None, None, None, None, 0, F(0.9), F(1e-6), None, None, None) == harl.HARL_OK
    assert adv(None, None, None, None, 0, F(0.9), F(0.0), None, None, None) == harl.HARL_E_INVALID_ARG  # eps <= 0
    assert adv(0x1000, 0x1000, 0x1000, None, 4, F(0.9), F(1e-6), None, 0x2000, None) == harl.HARL_E_INVALID_ARG
    assert adv(0x1000, 0x1000, 0x1000, 0x1000, 4, F(0.9), F(1e-6), 0x2002, 0x2000, None) == harl.HARL_E_INVALID_ARG
    el = lambda *a: _status("harl_track_eliminate", *a)
    assert el(None, 10, 11, None, None, 0, None, None, 0, None) == harl.HARL_E_INVALID_ARG       # n_keep > n
    assert el(None, 10, 0, None, None, 0, None, None, 0, None) == harl.HARL_OK                    # no-op
    assert el(0x1000, 10, 4, 0x2000, 0x3000, 16, None, 0x4000, 1 << 20, None) == harl.HARL_E_INVALID_ARG  # rows w/o out
    assert el(0x1000, 10, 4, 0x2000, 0x3000, 0, 0x9000, 0x4000, 1 << 20, None) == harl.HARL_E_INVALID_ARG  # row_bytes 0
    assert el(0x1000, 10, 4, 0x2000, 0x3000, 64, 0x3100, 0x4000, 1 << 20, None) == harl.HARL_E_INVALID_ARG  # overlap
    assert el(0x1000, 10, 4, 0x2000, None, 0, None, 0x4000, 8, None) == harl.HARL_E_WORKSPACE
    assert el(0x1000, 10, 4, 0x2000, None, 0, None, 0x4001, 1 << 20, None) == harl.HARL_E_INVALID_ARG
    assert el(0x1001, 10, 4, 0x2000, None, 0, None, 0x4000, 1 << 20, None) == harl.HARL_E_INVALID_ARG
    assert harl.harl_track_eliminate_workspace_size(-1) == 0
    assert harl.harl_track_eliminate_workspace_size(100000) >= 256 + 25 * 1024


def test_policy_select_argument_errors():
    sel = lambda B, a, off, flags=0, logits=0x1000, action=0x2000: _status(
        "harl_policy_select", logits, B, a, np.ascontiguousarray(off, np.int32).ctypes.data, len(off) - 1, flags, 0, 0,
        action, None, None, None)
    assert sel(4, 26, [0, 17, 20, 23, 27]) == harl.HARL_E_INVALID_ARG        # does not end at a
    assert sel(4, 26, [1, 17, 20, 23, 26]) == harl.HARL_E_INVALID_ARG        # does not start at 0
    assert sel(4, 26, [0, 17, 17, 23, 26]) == harl.HARL_E_INVALID_ARG        # empty segment
    assert sel(4, 26, [0, 17, 20, 23, 26], flags=2) == harl.HARL_E_INVALID_ARG
    assert sel(4, 26, [0, 17, 20, 23, 26], logits=0x1002) == harl.HARL_E_INVALID_ARG
    assert sel(4, 26, [0, 17, 20, 23, 26], action=None) == harl.HARL_E_INVALID_ARG
    assert sel(4, 4097, [0, 4097]) == harl.HARL_E_INVALID_ARG
    assert sel(4, 40, list(range(0, 41, 1))) == harl.HARL_E_INVALID_ARG     # 40 segments > 32
    assert sel(0, 26, [0, 17, 20, 23, 26], logits=None, action=None) == harl.HARL_OK


def test_ppo_argument_errors():
    cfg = harl.ppo_config(64, 256, 256, 26, [0, 17, 20, 23, 26])
    n = harl.harl_ppo_param_count(cfg)
    assert n == 256 * 64 + 256 + 256 * 256 + 256 + 26 * 256 + 26 + 256 + 1
    assert harl.harl_ppo_workspace_size(cfg, 4096) > 4096 * (256 * 4 + 26 * 2) * 4
    bad = harl.ppo_config(64, 256, 256, 26, [0, 17, 20, 23, 27])
    assert harl.harl_ppo_param_count(bad) == 0
    up = lambda c, step=1, M=4, ws=0x5000, wsb=1 << 30, params=0x1000: _status(
        "harl_ppo_update", ctypes.byref(c), params, 0x2000, 0x3000, step, 0x4000, 0x4000, 0x4000, 0x4000, 0x4000, M,
        None, None, ws, wsb, None)
    assert up(bad) == harl.HARL_E_INVALID_ARG
    assert up(cfg, step=0) == harl.HARL_E_INVALID_ARG
    assert up(cfg, M=0) == harl.HARL_OK
    assert up(cfg, params=None) == harl.HARL_E_INVALID_ARG
    assert up(cfg, ws=0x5001) == harl.HARL_E_INVALID_ARG
    assert up(cfg, wsb=64) == harl.HARL_E_WORKSPACE
    lr = harl.ppo_config(64, 256, 256, 26, [0, 26], beta1=1.0)
    assert up(lr) == harl.HARL_E_INVALID_ARG


def test_gbdt_argument_errors():
    prm = harl.gbdt_params()
    assert harl.harl_gbdt_round_workspace_size(prm, 164, 65536, 2048) > 65536 * 40
    for bad in (harl.gbdt_params(max_depth=0), harl.gbdt_params(max_depth=13), harl.gbdt_params(reg_lambda=0.0),
                harl.gbdt_params(gamma=-1.0), harl.gbdt_params(min_child_weight=float("nan"))):
        assert harl.harl_gbdt_round_workspace_size(bad, 164, 100, 10) == 0
    assert harl.harl_gbdt_round_workspace_size(prm, 0, 100, 10) == 0
    b = lambda ldf=100, F=164, N=100, ldb=100, bins=0x1000, stride=16: _status(
        "harl_gbdt_bin", 0x2000, ldf, F, N, 0x3000, stride, 0x4000, bins, ldb, None)
    assert b(ldf=99) == harl.HARL_E_INVALID_ARG
    assert b(ldb=99) == harl.HARL_E_INVALID_ARG  # planes shorter than the rows
    assert b(bins=0x1004) == harl.HARL_E_INVALID_ARG
    assert b(stride=0) == harl.HARL_E_INVALID_ARG
    assert b(N=0) == harl.HARL_OK
    r = lambda p=prm, ldb=100, bins=0x1000, ws=0x5000, wsb=1 << 30, N=100, P=10, label=0x6000: _status(
        "harl_gbdt_round", ctypes.byref(p), bins, ldb, 164, N, 0x3000, 16, 0x4000, 0x7000, P, label, 0x6000, 0x8000,
        0x9000, 0x9000, 0x9000, 0x9000, 0x9000, 0x9000, ws, wsb, None)
    assert r(p=harl.gbdt_params(max_depth=13)) == harl.HARL_E_INVALID_ARG
    assert r(ldb=99) == harl.HARL_E_INVALID_ARG
    assert r(bins=0x1004) == harl.HARL_E_INVALID_ARG
    assert r(label=None) == harl.HARL_E_INVALID_ARG
    assert r(ws=0x5001) == harl.HARL_E_INVALID_ARG
    assert r(wsb=64) == harl.HARL_E_WORKSPACE


def test_header_is_plain_c():
    """include/harl.h compiles on its own as C99 (pedantic) and as C++: a C ABI with no torch or HIP
    types."""
    import shutil
    import subprocess
    hdr = os.path.join(ROOT, "include", "harl.h")
    for cc, args in (("gcc", ["-std=c99", "-pedantic", "-x", "c"]), ("g++", ["-std=c++11", "-x", "c++"])):
        if shutil.which(cc) is None:
            pytest.skip("%s not available" % cc)
        r = subprocess.run([cc, *args, "-Wall", "-Wextra", "-Werror", "-fsyntax-only", hdr], capture_output=True,
                           text=True)
        assert r.returncode == 0, r.stderr
    src = open(hdr).read()
    for banned in ("torch", "hip_runtime", "at::", "c10::"):
        assert banned not in src, banned
