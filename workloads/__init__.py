"""Seeded synthetic inputs for the selective-FFN workloads (shared by tests and the benchmark)."""
from .synth import (  # noqa: F401
    CONFIGS,
    FFNConfig,
    active_sets,
    csr_from_sets,
    es_keys,
    layer_weights,
    loaded_ids,
    popularity,
    storage_from_f32,
    tokens_x,
)
