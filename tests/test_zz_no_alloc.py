"""harl_topk_static (the top-K entry point that allocates nothing, for callers that cannot: its
candidate buffers are a library-owned device array) against harl_topk with a workspace: identical
results on two calls in a row, the second with a smaller input, with and without the running-merge
flag, through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2211_11172_amd import harl
from tests.gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu


def _pair(score, n, k, base, merge, seed_run=None):
    import torch
    d = torch.from_numpy(np.ascontiguousarray(score[:n], np.float32)).cuda()
    outs = []
    for static in (False, True):
        s = torch.empty(k, dtype=torch.float32, device="cuda")
        i = torch.empty(k, dtype=torch.int64, device="cuda")
        if seed_run is not None:
            s.copy_(torch.from_numpy(seed_run[0]))
            i.copy_(torch.from_numpy(seed_run[1]))
        flags = harl.HARL_TOPK_MERGE if merge else 0
        if static:
            harl.harl_topk_static(d, n, k, base, s, i, flags)
        else:
            wsb = harl.harl_topk_workspace_size(n, k)
            ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
            harl.harl_topk(d, n, k, base, s, i, flags, ws, wsb)
        torch.cuda.synchronize()
        outs.append((s.cpu().numpy(), i.cpu().numpy()))
    return outs


@pytest.mark.parametrize("k", [1, 64, 1024, 2048])
def test_static_topk_equals_workspace_topk_twice(k):
    require_gpu()
    rng = np.random.default_rng(k)
    big, small = 1_048_576, 70_001
    score = rng.standard_normal(big).astype(np.float32)
    score[::97] = np.round(score[::97] * 4) / 4        # ties
    score[5::1013] = -0.0
    for n in (big, small):                               # two calls, the second smaller
        log("top-k static vs workspace: n=%d k=%d" % (n, k))
        (ws_s, ws_i), (st_s, st_i) = _pair(score, n, k, 12345, merge=False)
        np.testing.assert_array_equal(st_i, ws_i)
        assert st_s.tobytes() == ws_s.tobytes()


def test_static_topk_merge_twice():
    require_gpu()
    rng = np.random.default_rng(3)
    k = 1024
    run = (np.full(k, -np.inf, np.float32), np.full(k, np.iinfo(np.int64).max, np.int64))
    for b, n in enumerate((65_536, 9_999)):
        score = rng.standard_normal(n).astype(np.float32)
        log("top-k static vs workspace (merge): batch %d n=%d" % (b, n))
        (ws_s, ws_i), (st_s, st_i) = _pair(score, n, k, b * 65_536, merge=True, seed_run=run)
        np.testing.assert_array_equal(st_i, ws_i)
        assert st_s.tobytes() == ws_s.tobytes()
        run = (ws_s, ws_i)


def test_static_topk_rejects_oversized_requests():
    require_gpu()
    import torch
    s = torch.empty(2048, dtype=torch.float32, device="cuda")
    i = torch.empty(2048, dtype=torch.int64, device="cuda")
    d = torch.zeros(2_088_961, dtype=torch.float32, device="cuda")
    assert harl.harl_topk_workspace_size(2_088_961, 2048) > harl.HARL_TOPK_STATIC_SCRATCH_BYTES
    rc = harl.load().harl_topk_static(d.data_ptr(), 2_088_961, 2048, 0, s.data_ptr(), i.data_ptr(), 0, None)
    assert rc == harl.HARL_E_UNSUPPORTED
    assert "HARL_TOPK_STATIC_SCRATCH_BYTES" in harl.harl_last_error()
    # the largest request that fits runs
    harl.harl_topk_static(d, 2_088_960, 2048, 0, s, i, 0)
    torch.cuda.synchronize()
