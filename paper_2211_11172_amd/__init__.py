"""HARL search-round candidate evaluation on MI355X (gfx950).

The product is ``libharl.so`` (HIP kernels behind the C ABI of ``include/harl.h``); ``harl`` is
its ctypes binding and ``round`` a small helper that owns the device buffers of one round.
"""
from . import harl  # noqa: F401
from .harl import (  # noqa: F401
    HarlError, harl_ensemble_create, harl_policy_create, harl_policy_step, harl_score_round,
    harl_score_round_workspace_size, harl_topk, harl_topk_reset, harl_topk_workspace_size,
    harl_last_error, harl_version, HARL_TOPK_MERGE,
)
