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


def _replays_match(run, outputs, reset, reps=4):
    """Capture run() as a graph after one eager call; every replay (outputs scribbled over and in/out
    buffers reset to their inputs first, unrelated eager work in between) must equal the eager
    results bitwise."""
    import torch
    reset()
    run()
    torch.cuda.synchronize()
    want = [o.clone() for o in outputs]
    reset()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(reps):
        for o in outputs:  # scribble over every output, then restore the in/out buffers' inputs
            o.view(torch.uint8).fill_(0xA5)
        reset()
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (o, w) in enumerate(zip(outputs, want)):
            assert torch.equal(o.view(torch.uint8), w.view(torch.uint8)), "replay %d differs in output %d" % (rep, i)
        del junk


def test_graph_replay_refit():
    require_gpu()
    import torch
    from paper_2211_11172_amd import harl
    from synth import gen_measured
    m = gen_measured(get_config("standard"), n_cuts=254)
    N, P, F = m["n_rows"], get_config("standard").n_prog, 164
    log("graph replay: refit, %d rows" % N)
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    X, cuts, nc, ptr, lab, wt = (d(m["features"]), d(m["cuts"]), d(m["n_cuts"]), d(m["prog_ptr"]), d(m["label"]),
                                 d(m["weight"]))
    bins = torch.zeros((21, N, 8), dtype=torch.uint8, device="cuda")
    m0 = d(np.linspace(-0.1, 0.1, N).astype(np.float32))
    margin = m0.clone()
    prm = harl.gbdt_params()
    n_nodes = (1 << 11) - 1
    tree = [torch.zeros(n_nodes, dtype=t, device="cuda") for t in
            (torch.int32, torch.float32, torch.int32, torch.int32, torch.uint8, torch.float32)]
    wsb = harl.harl_gbdt_round_workspace_size(prm, F, N, P)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")

    def run():
        harl.harl_gbdt_bin(X, N, F, N, cuts, cuts.shape[1], nc, bins, N)
        harl.harl_gbdt_round(prm, bins, N, F, N, cuts, cuts.shape[1], nc, ptr, P, lab, wt, margin, *tree, ws, wsb)

    _replays_match(run, [bins, margin] + tree, lambda: margin.copy_(m0))


def test_graph_replay_ppo_update():
    require_gpu()
    import torch
    from oracle import ppo as oppo
    from paper_2211_11172_amd import harl
    from synth import gen_policy, gen_states
    segs = [0, 17, 20, 23, 26]
    M = 4096
    cfg = get_config("standard").with_(pol_a=26, n_prog=M)
    pol = gen_policy(cfg)
    flat = oppo.pack(dict(w1=pol["w1"], b1=pol["b1"], w2=pol["w2"], b2=pol["b2"], wa=pol["wa"], ba=pol["ba"],
                          wv=np.asarray(pol["wv"]).reshape(1, 256), bv=np.asarray(pol["bv"]).reshape(1)))
    rng = np.random.default_rng(3)
    acts = np.stack([rng.integers(segs[i], segs[i + 1], M) for i in range(4)], axis=1).astype(np.int32)
    c = harl.ppo_config(64, 256, 256, 26, segs)
    n = harl.harl_ppo_param_count(c)
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    p0 = d(flat.astype(np.float32))
    P, Mm, Vv = p0.clone(), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    st, ac = d(gen_states(cfg)), d(acts)
    lpo = d((rng.standard_normal(M) * 0.1 - 7.0).astype(np.float32))
    adv, ret = d(rng.standard_normal(M).astype(np.float32)), d(rng.standard_normal(M).astype(np.float32))
    wsb = harl.harl_ppo_workspace_size(c, M)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    grad, loss = torch.empty(n, device="cuda"), torch.empty(4, device="cuda")
    log("graph replay: PPO update, %d transitions" % M)

    def reset():
        P.copy_(p0)
        Mm.zero_()
        Vv.zero_()

    _replays_match(lambda: harl.harl_ppo_update(c, P, Mm, Vv, 1, st, ac, lpo, adv, ret, M, grad, loss, ws, wsb),
                   [P, Mm, Vv, grad, loss], reset)


def test_graph_replay_select_and_tracks():
    require_gpu()
    import torch
    from paper_2211_11172_amd import harl
    from synth import gen_track_step
    rng = np.random.default_rng(4)
    B, a, segs = 20000, 26, [0, 17, 20, 23, 26]
    z = torch.from_numpy(rng.standard_normal((B, a)).astype(np.float32)).cuda()
    seg = np.array(segs, np.int32)
    act = torch.zeros((B, 4), dtype=torch.int32, device="cuda")
    logp = torch.zeros((B, 4), device="cuda")
    probs = torch.zeros((B, a), device="cuda")
    n = 40000  # above the one-workgroup elimination path
    step = gen_track_step(get_config("throughput"), n=n)
    dv = {k: torch.from_numpy(v).cuda() for k, v in step.items()}
    rew, adv = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    keep = torch.zeros(n // 2, dtype=torch.int32, device="cuda")
    rows = torch.from_numpy(rng.standard_normal((n, 64)).astype(np.float32)).cuda()
    rows_out = torch.zeros((n // 2, 64), device="cuda")
    wsb = harl.harl_track_eliminate_workspace_size(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    log("graph replay: per-type selection (%d states) and tracks (%d)" % (B, n))

    def run():
        harl.harl_policy_select(z, B, a, seg, harl.HARL_SELECT_SAMPLE, 1234, 99, act, logp, probs)
        harl.harl_track_advantage(dv["c_prev"], dv["c_next"], dv["v_prev"], dv["v_next"], n, 0.9, 1e-6, rew, adv)
        harl.harl_track_eliminate(adv, n, n // 2, keep, rows, 256, rows_out, ws, wsb)

    _replays_match(run, [act, logp, probs, rew, adv, keep, rows_out], lambda: None)
