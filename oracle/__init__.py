"""fp64 CPU oracle for TGV-KV (test infrastructure only; see tgvkv_oracle)."""

from .tgvkv_oracle import (  # noqa: F401
    compact_slice,
    decode_attention,
    decode_reference,
    default_scale,
    evict_sequence,
    flat_offsets,
    forced_positions,
    forced_vision_count,
    head_average,
    layer_budgets,
    score_slice,
    text_positions,
    text_row_softmax,
    text_scores,
    text_weights,
    tpr_select,
    tv_mass,
    vision_positions,
    vision_only_budgets,
    vision_scores,
)
