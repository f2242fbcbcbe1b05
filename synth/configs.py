"""The five synthetic search-round workloads and small variants of them.

A *round* is one batched evaluation of all live candidates (one step of the parameter-search loop
of the paper's Algorithm 1).  A candidate is one tensor program with 1..s_max statements; each
statement is one row of ``n_features`` fp32 features.  The cost model is a complete-tree GBDT of
``n_trees`` trees of ``depth`` split levels; the actor/critic is a shared two-layer ReLU trunk with
an actor head of ``pol_a`` logits and a one-unit value head.

The paper prints none of these sizes (its cost model follows Ansor's XGBoost setup, Section 6.1 and
Appendix A.1; its actor/critic follows an external PPO code base).  The sizes below are the
workloads this implementation is measured on, each with its generation recipe in `synth.gen`.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class RoundConfig:
    name: str
    cfg_id: int                 # seeds: every stream is keyed by (cfg_id, variant, stream[, batch])
    n_prog: int                 # candidates per batch
    n_batches: int              # >1 only for the streamed search
    s_max: int                  # statements per program ~ U{1..s_max}
    n_trees: int
    depth: int                  # split levels of every (complete) tree
    top_k: int
    n_features: int = 164
    p_nan: float = 0.0          # per-element probability of a missing (NaN) feature
    p_zero: float = 0.4         # per-element probability of an exact 0.0
    lu_lo_exp: float = -3.0     # non-zero, non-missing values are 10**U[lo, hi)
    lu_hi_exp: float = 3.0
    n_calib: int = 4096         # calibration rows per feature for threshold quantiles
    leaf_sigma: float = 0.1
    pol_dtype: str = "f32"      # "f32" or "bf16"
    pol_s: int = 64
    pol_h1: int = 256
    pol_h2: int = 256
    pol_a: int = 24
    softmax: bool = False
    exact: bool = False         # dyadic leaves and integer MLP: every sum is exact in fp32
    seed: int = 0

    @property
    def variant(self) -> int:
        return 1 if self.exact else 0

    @property
    def n_candidates(self) -> int:
        return self.n_prog * self.n_batches

    def with_(self, **kw) -> "RoundConfig":
        return dataclasses.replace(self, **kw)


_STD_MLP = dict(pol_dtype="f32", pol_s=64, pol_h1=256, pol_h2=256, pol_a=24, softmax=False)
_BIG_MLP = dict(pol_dtype="bf16", pol_s=128, pol_h1=1024, pol_h2=1024, pol_a=64, softmax=True)

CONFIGS = {
    # 512 programs, U{1..8} statements, 64 trees of depth 6, fp32 MLP 64-256-256 -> 24 (+1), top-64
    "tiny": RoundConfig("tiny", 1, n_prog=512, n_batches=1, s_max=8, n_trees=64, depth=6,
                        top_k=64, **_STD_MLP),
    # 4,096 programs, U{1..32} statements, 300 trees of depth 8, same MLP, top-128
    "standard": RoundConfig("standard", 2, n_prog=4096, n_batches=1, s_max=32, n_trees=300,
                            depth=8, top_k=128, **_STD_MLP),
    # 65,536 programs, U{1..64} statements, 500 trees of depth 8, same MLP, top-512
    "throughput": RoundConfig("throughput", 3, n_prog=65536, n_batches=1, s_max=64, n_trees=500,
                              depth=8, top_k=512, **_STD_MLP),
    # scoring as "throughput"; bf16 MLP 128-1024-1024 -> 64 (+1) with softmax
    "policy_heavy": RoundConfig("policy_heavy", 4, n_prog=65536, n_batches=1, s_max=64,
                                n_trees=500, depth=8, top_k=512, **_BIG_MLP),
    # 1,048,576 candidates in 16 batches of 65,536; 10% NaN; 1000 trees of depth 10;
    # running global top-1024 across batches; bf16 MLP as "policy_heavy"
    "streamed": RoundConfig("streamed", 5, n_prog=65536, n_batches=16, s_max=64, n_trees=1000,
                            depth=10, top_k=1024, p_nan=0.1, **_BIG_MLP),
}

CONFIG_ORDER = ["tiny", "standard", "throughput", "policy_heavy", "streamed"]


def get_config(name: str, exact: bool = False) -> RoundConfig:
    """Return a named workload; ``name`` may carry an ``-exact`` suffix."""
    if name.endswith("-exact"):
        name, exact = name[: -len("-exact")], True
    cfg = CONFIGS[name]
    return cfg.with_(exact=True) if exact else cfg


def mini_config(**kw) -> RoundConfig:
    """A small workload for brute-force checks and quick parity cases (seeded like the others)."""
    base = RoundConfig("mini", 99, n_prog=48, n_batches=1, s_max=5, n_trees=4, depth=3,
                       top_k=8, n_features=8, pol_s=8, pol_h1=32, pol_h2=32, pol_a=6)
    return base.with_(**kw)
