"""MI355X-native selective-computation gated FFN (SelectInfer's hot path).

The C ABI (include/selectinfer.h) is implemented in HIP for gfx950 in ``csrc/`` and built into
``libselectinfer.so``; this package is its thin Python binding.
"""
from .api import (  # noqa: F401
    BF16,
    F16,
    F32,
    FLAG_CHECK,
    FLAG_EXACT_H,
    FLAG_FAST_H,
    FLAG_PER_TOKEN,
    FLAG_SORTED,
    FLAG_UNION,
    TOPK_ABS,
    TOPK_RAW,
    CompactLayer,
    SelectInferError,
    build_loaded_set,
    ceiling_gather,
    ceiling_stream,
    compact_ffn,
    load_selected,
    dynamic_set,
    merge_scores,
    profile_scores,
    rank_neurons,
    remap_ids,
    residual_rmsnorm,
    select_topk,
    selective_ffn,
    selective_ffn_noalloc,
    selective_ffn_resnorm,
    selective_ffn_workspace,
    selective_layers,
    set_timing_events,
    version,
)
