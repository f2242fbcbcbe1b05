"""GPU parity of harl_topk: top-K of the heap H (Algorithm 1, top-K phase) and the running merge.
Selection is an integer result: bit-exact against the oracle on the same score array."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from tests.gpu_util import gpu_topk, log, require_gpu

pytestmark = pytest.mark.gpu


def _scores(n, rng, ties=True):
    s = rng.standard_normal(n).astype(np.float32)
    if ties and n > 10:
        s[rng.integers(0, n, n // 5)] = np.float32(0.75)
        s[rng.integers(0, n, n // 50)] = -0.0
        s[rng.integers(0, n, n // 50)] = 0.0
    return s


@pytest.mark.parametrize("n,k", [(1, 1), (7, 7), (100, 1), (4096, 128), (4097, 128), (3000, 129), (20000, 300),
                                 (8193, 1000), (65536, 512), (65536, 2048), (70001, 1024), (300000, 64),
                                 (9000, 2048)])
def test_topk_matches_oracle(n, k):
    require_gpu()
    rng = np.random.default_rng(n + k)
    s = _scores(n, rng)
    log("topk n=%d k=%d" % (n, k))
    gs, gi = gpu_topk(s, k, index_base=12345)
    ws, wi = oracle.topk(s, k, index_base=12345)
    np.testing.assert_array_equal(gi, wi)
    np.testing.assert_array_equal(gs.view(np.uint32), ws.view(np.uint32))   # bit copies of the inputs


def test_topk_specials():
    require_gpu()
    s = np.array([1.0, np.nan, 3.0, -np.inf, 3.0, -0.0, 0.0, np.inf, np.nan], np.float32)
    gs, gi = gpu_topk(s, 9)
    ws, wi = oracle.topk(s, 9)
    np.testing.assert_array_equal(gi, wi)
    gs, gi = gpu_topk(np.zeros(5000, np.float32), 64)
    assert gi.tolist() == list(range(64))


@pytest.mark.parametrize("k,n,nb", [(64, 1000, 5), (1024, 65536, 3), (2048, 3000, 4), (16, 5, 4)])
def test_running_merge_matches_oracle(k, n, nb):
    require_gpu()
    rng = np.random.default_rng(k * 7 + n)
    run_g = oracle.reset(k)
    run_o = oracle.reset(k)
    log("merge k=%d n=%d batches=%d" % (k, n, nb))
    for b in range(nb):
        s = (rng.integers(-50, 50, n) / 8).astype(np.float32)    # heavy ties across batches
        run_g = gpu_topk(s, k, index_base=b * n, running=run_g)
        run_o = oracle.merge(run_o[0], run_o[1], s, b * n)
        np.testing.assert_array_equal(run_g[1], run_o[1])
        np.testing.assert_array_equal(run_g[0], run_o[0])


def test_merge_batch_order_invariance_and_resume():
    require_gpu()
    rng = np.random.default_rng(3)
    k, n, nb = 256, 5000, 5
    batches = [(rng.integers(-30, 30, n) / 4).astype(np.float32) for _ in range(nb)]
    results = []
    for order in ([0, 1, 2, 3, 4], [4, 2, 0, 3, 1]):
        run = oracle.reset(k)
        for b in order:
            run = gpu_topk(batches[b], k, index_base=b * n, running=run)
        results.append(run)
    np.testing.assert_array_equal(results[0][1], results[1][1])
    want = oracle.topk(np.concatenate(batches), k)
    np.testing.assert_array_equal(results[0][1], want[1])


def test_merge_empty_batch_is_noop():
    require_gpu()
    run = oracle.merge(*oracle.reset(8), np.array([2.0, 1.0], np.float32), 0)
    got = gpu_topk(np.zeros(0, np.float32), 8, index_base=10, running=run)
    np.testing.assert_array_equal(got[1], run[1])
