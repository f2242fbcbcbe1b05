"""Parity at the full workload sizes, in the launch configuration the benchmark uses.

standard round (4,096 programs, 300 trees of depth 8, fp32 MLP): every program score, logit,
value and action against the oracle; top-128 exact on the GPU's own scores and, end to end, equal to
the oracle's up to near-ties.  throughput round (65,536 programs, ~2.1M statement rows, 500 trees of
depth 8): every program score against the full oracle, top-512 as above, 512 sampled states'
logits, values and actions.  policy_heavy (65,536 bf16 states, 128-1024-1024 -> 64 + 1): the whole
batch on the GPU, 768 sampled states against the oracle.  streamed search (16 batches of 65,536
candidates, 10% missing features, 1000 trees of depth 10, bf16 MLP, running top-1024): every
batch, 1,024 sampled programs and 128 sampled states against the oracle, the running top-1024 equal
to the oracle's merge of the GPU's batch scores after every batch, and the final 1,024 winners'
programs scored by the oracle within tolerance of the running top-1024's scores.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from synth import gen_batch, gen_ensemble, gen_policy, gen_states, get_config
from tests.gpu_util import assert_close_scaled, gpu_policy, gpu_topk, log, near_tie_ok, require_gpu

pytestmark = pytest.mark.gpu


def _sample_programs(ptr, idx):
    """Feature columns and CSR pointer of a subset of programs (kept in order)."""
    rows = np.concatenate([np.arange(ptr[p], ptr[p + 1]) for p in idx])
    counts = np.array([ptr[p + 1] - ptr[p] for p in idx])
    sp = np.zeros(len(idx) + 1, np.int32)
    np.cumsum(counts, out=sp[1:])
    return rows, sp


def _policy_parity(rnd, pol, states, idx, rtol, what):
    """The round's logits, values and actions at states idx against the oracle (a position may
    differ only between near-tied logits)."""
    logits = rnd.logits.cpu().numpy()[idx]
    val = rnd.value.cpu().numpy()[idx]
    act = rnd.action.cpu().numpy()[idx]
    np.testing.assert_array_equal(act, np.argmax(logits, axis=1))
    wp = oracle.policy_step(pol, states[idx], want_probs=False)
    assert_close_scaled(logits, wp["logits"], wp["logit_scale"], rtol, what + " logits")
    assert_close_scaled(val, wp["value"], wp["value_scale"], rtol, what + " value")
    flips = np.nonzero(act != wp["action"])[0]
    for i in flips:
        a, c = act[i], wp["action"][i]
        assert wp["logits"][i, c] - wp["logits"][i, a] <= rtol * (wp["logit_scale"][i, a] + wp["logit_scale"][i, c])
    return flips.size


def test_standard_round_full():
    """The benchmarked standard round, standard (non-exact) variant, end to end."""
    require_gpu()
    import torch
    from paper_2211_11172_amd.round import Round, upload_batch
    cfg = get_config("standard")
    ens, pol, b = gen_ensemble(cfg), gen_policy(cfg), gen_batch(cfg)
    log("standard round: %d programs, %d rows" % (cfg.n_prog, b["n_rows"]))
    rnd = Round(ens, pol, b["n_rows"], cfg.n_prog, cfg.top_k, want_logits=True)
    batch = upload_batch(b["features"], b["prog_ptr"], b["states"])
    rnd.step(batch)
    torch.cuda.synchronize()
    got = rnd.prog_score.cpu().numpy()
    top_i = rnd.top_index.cpu().numpy()
    want = oracle.score_round(ens, b["features"], b["prog_ptr"])
    assert_close_scaled(got, want["prog"], want["scale"], 1e-5, "program scores")
    np.testing.assert_array_equal(top_i, oracle.topk(got, cfg.top_k)[1])
    _, oi = oracle.topk(want["prog32"], cfg.top_k)
    swaps = near_tie_ok(top_i, oi, want["prog"], 1e-5 * want["scale"])
    flips = _policy_parity(rnd, pol, b["states"], np.arange(cfg.n_prog), 1e-5, "policy")
    log("  top-%d near-tie swaps: %d, argmax near-tie flips: %d" % (cfg.top_k, swaps, flips))
    rnd.close()


def test_throughput_round_full():
    require_gpu()
    import torch
    from paper_2211_11172_amd.round import Round, upload_batch
    cfg = get_config("throughput")
    ens, pol, b = gen_ensemble(cfg), gen_policy(cfg), gen_batch(cfg)
    log("throughput round: %d programs, %d rows" % (cfg.n_prog, b["n_rows"]))
    rnd = Round(ens, pol, b["n_rows"], cfg.n_prog, cfg.top_k, want_logits=True)
    batch = upload_batch(b["features"], b["prog_ptr"], b["states"])
    rnd.step(batch)
    torch.cuda.synchronize()
    got = rnd.prog_score.cpu().numpy()
    top_i = rnd.top_index.cpu().numpy()
    log("  oracle on all programs")
    want = oracle.score_round(ens, b["features"], b["prog_ptr"])
    assert_close_scaled(got, want["prog"], want["scale"], 1e-5, "program scores")
    # top-K is exact on the GPU's own scores ...
    np.testing.assert_array_equal(top_i, oracle.topk(got, cfg.top_k)[1])
    # ... and equal to the oracle's top-K up to near-ties
    _, oi = oracle.topk(want["prog32"], cfg.top_k)
    swaps = near_tie_ok(top_i, oi, want["prog"], 1e-5 * want["scale"])
    log("  top-%d near-tie swaps: %d" % (cfg.top_k, swaps))
    # the fp32 policy on the same round, sampled states: logits, values and actions
    idx = np.random.default_rng(0).choice(cfg.n_prog, 512, replace=False)
    _policy_parity(rnd, pol, b["states"], idx, 1e-5, "policy")
    rnd.close()


def test_policy_heavy_full_batch_sampled():
    require_gpu()
    cfg = get_config("policy_heavy")
    pol = gen_policy(cfg)
    st = gen_states(cfg)
    log("policy_heavy: %d bf16 states" % st.shape[0])
    got = gpu_policy(pol, st)
    np.testing.assert_array_equal(got["action"], np.argmax(got["logits"], axis=1))
    idx = np.random.default_rng(1).choice(st.shape[0], 768, replace=False)
    want = oracle.policy_step(pol, st[idx])
    assert_close_scaled(got["logits"][idx], want["logits"], want["logit_scale"], 2e-2, "logits")
    assert_close_scaled(got["value"][idx], want["value"], want["value_scale"], 2e-2, "value")
    assert np.abs(got["probs"][idx] - want["probs"]).max() <= 2e-2
    ga = got["action"][idx]
    for i in np.nonzero(ga != want["action"])[0]:
        a, c = ga[i], want["action"][i]
        assert want["logits"][i, c] - want["logits"][i, a] <= 2e-2 * (want["logit_scale"][i, a] + want["logit_scale"][i, c])


def test_streamed_search_all_batches():
    require_gpu()
    import torch
    from concurrent.futures import ThreadPoolExecutor
    from paper_2211_11172_amd.round import Round, upload_batch
    cfg = get_config("streamed")
    ens, pol = gen_ensemble(cfg), gen_policy(cfg)
    rnd = None
    run_o = oracle.reset(cfg.top_k)
    rng = np.random.default_rng(2)
    feats, ptrs = {}, {}
    with ThreadPoolExecutor(max_workers=6) as ex:
        futs = [ex.submit(gen_batch, cfg, bi) for bi in range(cfg.n_batches)]
        for bi, fut in enumerate(futs):
            b = fut.result()
            futs[bi] = None
            log("streamed batch %d: %d rows" % (bi, b["n_rows"]))
            if rnd is None:
                rnd = Round(ens, pol, int(b["n_rows"] * 1.2), cfg.n_prog, cfg.top_k, want_logits=True,
                            want_probs=True)
                rnd.reset_running()
            batch = upload_batch(b["features"], b["prog_ptr"], b["states"])
            rnd.step(batch, merge=True, index_base=bi * cfg.n_prog)
            torch.cuda.synchronize()
            got = rnd.prog_score.cpu().numpy()
            idx = np.sort(rng.choice(cfg.n_prog, 1024, replace=False))
            rows, sp = _sample_programs(b["prog_ptr"], idx)
            want = oracle.score_round(ens, np.ascontiguousarray(b["features"][:, rows]), sp)
            assert_close_scaled(got[idx], want["prog"], want["scale"], 1e-5, "batch %d scores" % bi)
            run_o = oracle.merge(run_o[0], run_o[1], got, bi * cfg.n_prog)
            np.testing.assert_array_equal(rnd.top_index.cpu().numpy(), run_o[1])
            np.testing.assert_array_equal(rnd.top_score.cpu().numpy(), run_o[0])
            sidx = np.sort(rng.choice(cfg.n_prog, 128, replace=False))
            _policy_parity(rnd, pol, b["states"], sidx, 2e-2, "batch %d policy" % bi)
            # keep what the winners' re-scoring needs: the batch's candidates still in the running top-K
            keep = [int(g - bi * cfg.n_prog) for g in run_o[1] if bi * cfg.n_prog <= g < (bi + 1) * cfg.n_prog]
            if keep:
                kr, ksp = _sample_programs(b["prog_ptr"], np.array(sorted(keep)))
                feats[bi] = (np.array(sorted(keep)), np.ascontiguousarray(b["features"][:, kr]), ksp)
            for old_bi in [k for k in feats if k != bi]:
                gl = set(int(g) for g in run_o[1])
                idx_old = feats[old_bi][0]
                if not any(old_bi * cfg.n_prog + int(i) in gl for i in idx_old):
                    del feats[old_bi]
            del b, batch
    # the final winners, re-scored by the oracle from their own statements
    top_s, top_i = rnd.top_score.cpu().numpy(), rnd.top_index.cpu().numpy()
    checked = 0
    for bi, (idx_b, X_b, sp_b) in feats.items():
        want = oracle.score_round(ens, X_b, sp_b)
        for j, local in enumerate(idx_b):
            pos = np.nonzero(top_i == bi * cfg.n_prog + int(local))[0]
            if pos.size:
                err = abs(float(top_s[pos[0]]) - want["prog"][j])
                assert err <= 1e-5 * want["scale"][j], "winner %d off by %g" % (int(top_i[pos[0]]), err)
                checked += 1
    assert checked == cfg.top_k
    log("  %d winners re-scored by the oracle" % checked)
    rnd.close()
