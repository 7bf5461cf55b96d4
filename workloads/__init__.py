"""Seeded synthetic VLM-shaped workloads for the TGV-KV eviction path.

This package draws the inputs that both the fp64 oracle and the GPU library
consume: text queries, keys, values and decode-step tokens, laid out as the
library expects and rounded once to bf16.  It holds none of the method's
arithmetic (no attention, scores, budgets or selection), only the random
recipes and the shapes.
"""

from .configs import WorkloadConfig, CONFIGS, DEPTH_PROFILE_TV_GAP, get_config, custom_config, depth_profile  # noqa: F401
from .gen import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    gen_decode_slice,
    gen_k_slice,
    gen_qtext_slice,
    gen_v_slice,
    make_decode_tensors,
    make_prefill_tensors,
    total_budget,
)
