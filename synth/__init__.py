"""Seeded synthetic inputs for one HARL search round (candidate features, GBDT cost model,
actor/critic weights and states).

This module holds no part of the method's arithmetic: it only draws inputs. Both the CPU oracle
(``oracle/``) and the HIP path consume exactly these arrays, which is the only thing the two share.
"""
from .configs import RoundConfig, CONFIGS, get_config, mini_config  # noqa: F401
from .gen import (  # noqa: F401
    gen_ensemble,
    gen_batch,
    gen_policy,
    gen_states,
    gen_track_step,
    gen_measured,
    gen_features,
    gen_prog_ptr,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
)
