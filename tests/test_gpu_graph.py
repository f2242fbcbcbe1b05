"""A round captured as a HIP graph replays to the same results as the eager calls, replay after
replay, with unrelated eager GPU work and synchronisations in between."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_batch, gen_ensemble, gen_policy, get_config
from tests.gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "standard"])
def test_graph_replay_matches_eager(name):
    require_gpu()
    import torch
    from paper_2211_11172_amd.round import Round, upload_batch
    cfg = get_config(name)
    ens, pol, b = gen_ensemble(cfg), gen_policy(cfg), gen_batch(cfg)
    log("graph replay: %s" % name)
    rnd = Round(ens, pol, b["n_rows"], cfg.n_prog, cfg.top_k, want_logits=True, want_stmt=True)
    batch = upload_batch(b["features"], b["prog_ptr"], b["states"])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        rnd.step(batch)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    want = {k: getattr(rnd, k).clone() for k in ("prog_score", "stmt_score", "action", "value", "logits", "top_index",
                                                 "top_score")}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rnd.step(batch)
    for rep in range(4):
        for k in want:                       # scribble over the outputs between replays
            getattr(rnd, k).fill_(-3)
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in want.items():
            assert torch.equal(getattr(rnd, k), v), "replay %d differs in %s" % (rep, k)
        del junk
    # and the eager round agrees with the oracle's top-K on its own scores
    ts, ti = oracle.topk(want["prog_score"].cpu().numpy(), cfg.top_k)
    np.testing.assert_array_equal(want["top_index"].cpu().numpy(), ti)
    rnd.close()
