"""Device buffers and launch sequence of one search round, over the libharl C ABI.

``Round`` owns the model handles and every per-round device buffer (allocated once, with torch, at
construction); ``Round.step`` enqueues the three hot-path calls of a round: the actor/critic
forward, cost-model scoring and top-K (optionally merged into the running top-K).  The policy and
scoring read disjoint inputs (the states and the candidates' statement features) and only top-K
depends on scoring.  With `two_streams` the policy runs on a second stream after scoring, beside
top-K; otherwise the three calls run in turn on one stream.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import harl


@dataclass
class Batch:
    feat: torch.Tensor          # [n_features, ld] fp32
    ld: int
    n_rows: int
    prog_ptr: torch.Tensor      # [n_prog + 1] int32
    n_prog: int
    states: torch.Tensor        # [n_prog, s] fp32 or int16 (bf16 bits)


def upload_batch(features: np.ndarray, prog_ptr: np.ndarray, states: np.ndarray, device="cuda") -> Batch:
    ld = features.shape[1]
    if ld % 4:
        pad = np.zeros((features.shape[0], 4 - ld % 4), np.float32)
        features = np.concatenate([features, pad], axis=1)
    st = torch.from_numpy(np.ascontiguousarray(states).view(np.int16) if states.dtype == np.uint16 else
                          np.ascontiguousarray(states, np.float32))
    return Batch(feat=torch.from_numpy(np.ascontiguousarray(features, np.float32)).to(device),
                 ld=features.shape[1], n_rows=int(prog_ptr[-1]),
                 prog_ptr=torch.from_numpy(np.ascontiguousarray(prog_ptr, np.int32)).to(device),
                 n_prog=len(prog_ptr) - 1, states=st.to(device))


class Round:
    def __init__(self, ens: dict, pol: dict, max_rows: int, max_prog: int, k: int, device="cuda",
                 want_stmt=False, want_logits=False, want_probs=False, two_streams=False):
        self.device = torch.device(device)
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        torch.cuda.set_device(self.device)
        self.ens = harl.harl_ensemble_create(ens, stream=0)
        self.pol = harl.harl_policy_create(pol, stream=0)
        self.k, self.max_rows, self.max_prog = k, max_rows, max_prog
        f32 = dict(dtype=torch.float32, device=self.device)
        self.prog_score = torch.empty(max_prog, **f32)
        self.stmt_score = torch.empty(max_rows, **f32) if want_stmt else None
        self.ws_score_bytes = harl.harl_score_round_workspace_size(self.ens, max_rows, max_prog)
        self.ws_score = torch.empty(self.ws_score_bytes, dtype=torch.uint8, device=self.device)
        self.ws_topk_bytes = harl.harl_topk_workspace_size(max_prog, k)
        self.ws_topk = torch.empty(self.ws_topk_bytes, dtype=torch.uint8, device=self.device)
        self.action = torch.empty(max_prog, dtype=torch.int32, device=self.device)
        self.value = torch.empty(max_prog, **f32)
        a = int(pol["a"])
        self.logits = torch.empty(max_prog, a, **f32) if want_logits else None
        self.probs = torch.empty(max_prog, a, **f32) if want_probs else None
        self.top_score = torch.empty(k, **f32)
        self.top_index = torch.empty(k, dtype=torch.int64, device=self.device)
        self.side = torch.cuda.Stream(device=self.device) if two_streams else None

    def reset_running(self, stream=None):
        harl.harl_topk_reset(self.top_score, self.top_index, self.k, stream=stream)

    def score(self, b: Batch, stream=None):
        harl.harl_score_round(self.ens, b.feat, b.ld, b.n_rows, b.prog_ptr, b.n_prog, self.prog_score,
                              self.stmt_score, self.ws_score, self.ws_score_bytes, stream=stream)

    def policy(self, b: Batch, stream=None):
        harl.harl_policy_step(self.pol, b.states, b.n_prog, self.action, self.value, self.probs, self.logits,
                              stream=stream)

    def topk(self, b: Batch, merge=False, index_base=0, stream=None):
        harl.harl_topk(self.prog_score, b.n_prog, self.k, index_base, self.top_score, self.top_index,
                       harl.HARL_TOPK_MERGE if merge else 0, self.ws_topk, self.ws_topk_bytes, stream=stream)

    def step(self, b: Batch, merge=False, index_base=0):
        """Enqueue one round on the current stream.

        With the side stream, scoring runs first on all CUs; the policy is then issued on the side
        stream, where it runs beside top-K (a one-workgroup kernel on the main stream, which needs
        the scores), and the main stream waits for both.  Without it, the three calls run in turn.
        """
        main = torch.cuda.current_stream(self.device)
        if self.side is not None:
            self.score(b, stream=main)
            self.side.wait_stream(main)
            self.policy(b, stream=self.side)
            self.topk(b, merge=merge, index_base=index_base, stream=main)
            main.wait_stream(self.side)
        else:
            self.policy(b, stream=main)
            self.score(b, stream=main)
            self.topk(b, merge=merge, index_base=index_base, stream=main)

    def close(self):
        self.ens.close()
        self.pol.close()
