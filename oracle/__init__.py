"""Oracle for the selective-computation gated FFN — TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 NumPy definitions of what the GPU path computes. Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import this package. It shares no code
with the GPU library or its Python binding, and imports neither.
"""
from .ffn import (  # noqa: F401
    DuplicateError,
    NotLoadedError,
    OracleError,
    RangeError,
    compact,
    compacted_bytes,
    decode,
    dense_swiglu,
    memory_saving,
    remap,
    residual_rmsnorm_bf16,
    round_to_bf16_bits,
    select_topk,
    selective_ffn,
    sigmoid,
    silu,
    stack_step,
)
from .selection import (  # noqa: F401
    activations,
    build_loaded_set,
    dynamic_set,
    merge_scores,
    profile_scores,
    rank_neurons,
    select_dynamic,
    selective_layers,
)
