"""Seeded synthetic inputs for the fused sampler.

This package only draws random numbers and lays them out; it holds none of the
sampling arithmetic.  Both the CPU oracle (``oracle/``) and the HIP path are fed
from here, so the two see identical inputs.
"""
from .workloads import (  # noqa: F401
    MODE_GRAMMAR, MODE_REP, MODE_FREQ, MODE_PRES, MODE_BIAS, MODE_TEMP,
    MODE_GREEDY, MODE_TOPK, MODE_TOPP, MODE_MINP, MODE_LOGPROBS,
    F32, BF16,
    bf16_bits_from_f32, f32_from_bf16_bits,
    config0, config1, config2, config3, config4, config4_sparse, sparse_drafts, gumbel_noise, tree_from_path,
    make_config,
    CONFIG_NAMES,
    custom_rows, empty_params,
)
