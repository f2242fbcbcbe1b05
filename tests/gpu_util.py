"""Helpers for the GPU parity tests: device round-trips through the C ABI and tolerance checks.

The parity bars: fp32 cost-model scores and fp32 logits/values within 1e-5 of the oracle's
scale (sum of |terms|, fp64); bf16-policy logits/values within 2e-2 of that scale; probabilities
within 2e-2 absolute (bf16) or 1e-5 (fp32); argmax, top-K indices and the exact variants
bit-exact.  Where floating point decides an integer (argmax, ranking), a position may differ from
the oracle only when the two candidates' oracle values lie within their combined tolerance band.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU on this host")


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def assert_close_scaled(got, want, scale, rtol, what):
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - want)
    tol = rtol * np.asarray(scale, dtype=np.float64)
    bad = err > tol
    ratio = float(np.max(err / np.maximum(tol, 1e-300))) if err.size else 0.0
    assert not bad.any(), "%s: %d of %d beyond tolerance (max err/tol %.3g)" % (what, int(bad.sum()), err.size, ratio)
    return ratio


def gpu_score(ens_dict, X, prog_ptr, want_stmt=True, ld=None):
    """Run harl_score_round once; returns (prog_score, stmt_score) as numpy."""
    import torch
    from paper_2211_11172_amd import harl
    E = harl.harl_ensemble_create(ens_dict)
    try:
        n_prog = len(prog_ptr) - 1
        n_rows = int(prog_ptr[-1])
        Xd = torch.from_numpy(np.ascontiguousarray(X, np.float32)).cuda()
        ld = X.shape[1] if ld is None else ld
        ptr = torch.from_numpy(np.ascontiguousarray(prog_ptr, np.int32)).cuda()
        ps = torch.full((max(n_prog, 1),), np.nan, dtype=torch.float32, device="cuda")
        ss = torch.full((max(n_rows, 1),), np.nan, dtype=torch.float32, device="cuda") if want_stmt else None
        wsb = harl.harl_score_round_workspace_size(E, n_rows, n_prog)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        harl.harl_score_round(E, Xd, ld, n_rows, ptr, n_prog, ps, ss, ws, wsb)
        torch.cuda.synchronize()
        return ps.cpu().numpy()[:n_prog], (ss.cpu().numpy()[:n_rows] if want_stmt else None)
    finally:
        E.close()


def gpu_policy(pol_dict, states, probs=True, logits=True):
    import torch
    from paper_2211_11172_amd import harl
    P = harl.harl_policy_create(pol_dict)
    try:
        B = states.shape[0]
        if states.dtype == np.uint16:
            st = torch.from_numpy(np.ascontiguousarray(states).view(np.int16)).cuda()
        else:
            st = torch.from_numpy(np.ascontiguousarray(states, np.float32)).cuda()
        a = int(pol_dict["a"])
        act = torch.full((max(B, 1),), -7, dtype=torch.int32, device="cuda")
        val = torch.full((max(B, 1),), np.nan, dtype=torch.float32, device="cuda")
        pr = torch.full((max(B, 1), a), np.nan, dtype=torch.float32, device="cuda") if probs else None
        lg = torch.full((max(B, 1), a), np.nan, dtype=torch.float32, device="cuda") if logits else None
        harl.harl_policy_step(P, st, B, act, val, pr, lg)
        torch.cuda.synchronize()
        out = dict(action=act.cpu().numpy()[:B], value=val.cpu().numpy()[:B])
        out["probs"] = pr.cpu().numpy()[:B] if probs else None
        out["logits"] = lg.cpu().numpy()[:B] if logits else None
        return out
    finally:
        P.close()


def gpu_topk(scores, k, index_base=0, running=None):
    """harl_topk on a score array; with `running` (scores, indices) the call merges into it."""
    import torch
    from paper_2211_11172_amd import harl
    s = torch.from_numpy(np.ascontiguousarray(scores, np.float32)).cuda()
    n = scores.size
    if running is None:
        io_s = torch.full((k,), np.nan, dtype=torch.float32, device="cuda")
        io_i = torch.full((k,), -1, dtype=torch.int64, device="cuda")
        flags = 0
    else:
        io_s = torch.from_numpy(np.array(running[0], np.float32)).cuda()
        io_i = torch.from_numpy(np.array(running[1], np.int64)).cuda()
        flags = harl.HARL_TOPK_MERGE
    wsb = harl.harl_topk_workspace_size(n, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    harl.harl_topk(s if n > 0 else None, n, k, index_base, io_s, io_i, flags, ws, wsb)
    torch.cuda.synchronize()
    return io_s.cpu().numpy(), io_i.cpu().numpy()


def near_tie_ok(idx_got, idx_want, val, tol):
    """Ranked index lists may differ only at positions where the two candidates' oracle values
    lie within their combined tolerance.  Returns the number of such near-tie swaps."""
    swaps = 0
    for a, b in zip(idx_got, idx_want):
        if a != b:
            assert abs(val[a] - val[b]) <= tol[a] + tol[b], "rank differs beyond the near-tie band: %d vs %d" % (a, b)
            swaps += 1
    return swaps
