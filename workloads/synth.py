"""Seeded synthetic inputs for the selective-computation gated FFN.

The paper evaluates on Llama3.2 / Qwen2.5 checkpoints and on QA, translation and summarisation
datasets (Evaluation, "Datasets and Neuron-Files Selection"). None of those is used here: every
input below is drawn from a seed, with the shapes and value distributions of the workloads the
benchmark names (7B-, 8B- and 13B-shape FFN layers and a tiny fp32 layer).

This module only draws random numbers and lays them out in storage form. It holds none of the
method's arithmetic: no dot products, no activation, no compaction, no ordering rule of the
top-k selection, no normalisation. Both the oracle and the GPU path receive exactly the arrays
produced here.

Recipe (all seeds are ``SeedSequence([cfg_id, layer, purpose, ...])``):

* purpose 0: popularity permutation pi of the N neurons; rank r (1-based) belongs to neuron
  pi[r-1] and carries Zipf weight r**-1.1.
* purpose 1/2/3: W_gate [N][d], W_up [N][d], W_down [d][N] (row-major, the storage order of
  a PyTorch ``nn.Linear``), iid N(0, 0.02), drawn in float32 row blocks of 512 rows (block b
  seeded with ``[..., purpose, b]``), then rounded once to bf16 (round-to-nearest-even) or kept
  as float32.
* purpose 4: token activations x ~ N(0, 1), one seed per token ``[..., 4, t]``.
* purpose 5: per-token sampling keys, one seed per token ``[..., 5, t]``.
* loaded set: the L most popular neurons (pi[:L]), listed in popularity order, i.e. the
  ranked "neuron file" the profiler would emit.
* active set of a token: weighted sampling without replacement from the loaded set with the
  popularity weights, done with Efraimidis-Spirakis keys log(u)/w (the k largest keys win).
  With a hot core (7B batch-16 workload), the ``hot`` most popular neurons get key +inf so
  they are in every token's set, and the remaining k - hot members are sampled from the rest.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

P_PERM, P_GATE, P_UP, P_DOWN, P_X, P_KEYS = 0, 1, 2, 3, 4, 5
ZIPF_S = 1.1
W_STD = 0.02
ROW_BLOCK = 512


@dataclass(frozen=True)
class FFNConfig:
    name: str
    cfg_id: int
    d: int          # model (hidden) width
    N: int          # FFN neurons (intermediate width)
    L: int          # loaded neurons
    k: int          # active neurons per token
    B: int          # tokens per step
    steps: int      # steps in the workload (tokens for B == 1)
    layers: int     # FFN layers (stack workload)
    wdtype: str     # 'f32' or 'bf16' (weights and x)
    hot: int = 0    # size of the shared hot core forced into every token's set
    # layers whose FFN stays whole: every neuron loaded (L = N) and active in every token's
    # set (k = N); the others load L and compute k neurons
    dense_layers: tuple = ()

    def with_(self, **kw) -> "FFNConfig":
        return replace(self, **kw)

    def L_of(self, layer: int) -> int:
        return self.N if layer in self.dense_layers else self.L

    def k_of(self, layer: int) -> int:
        return self.N if layer in self.dense_layers else self.k


def _r(frac: float, n: int) -> int:
    # counts stated as fractions of N are rounded half-to-even; no exact .5 occurs here
    return int(round(frac * n))


CONFIGS = {
    "tiny_f32": FFNConfig("tiny_f32", 0, d=256, N=1024, L=512, k=128, B=1, steps=64,
                          layers=1, wdtype="f32"),
    "llama2_7b_decode": FFNConfig("llama2_7b_decode", 1, d=4096, N=11008, L=_r(0.7, 11008),
                                  k=_r(0.2, 11008), B=1, steps=1024, layers=1, wdtype="bf16"),
    "llama2_7b_b16": FFNConfig("llama2_7b_b16", 2, d=4096, N=11008, L=_r(0.7, 11008),
                               k=_r(0.2, 11008), B=16, steps=256, layers=1, wdtype="bf16",
                               hot=_r(0.1, 11008)),
    "llama3_8b_stack": FFNConfig("llama3_8b_stack", 3, d=4096, N=14336, L=_r(0.6, 14336),
                                 k=_r(0.15, 14336), B=1, steps=512, layers=32, wdtype="bf16"),
    # the 8B-shape stack with the layer range of the paper's Table 1: selective from layer 5 to
    # the second-last (exclusive); the first five and the last two layers keep the whole FFN.
    # Same seeds as llama3_8b_stack, so its selective layers are that workload's layers.
    "llama3_8b_stack_table1": FFNConfig("llama3_8b_stack_table1", 3, d=4096, N=14336,
                                        L=_r(0.6, 14336), k=_r(0.15, 14336), B=1, steps=512,
                                        layers=32, wdtype="bf16",
                                        dense_layers=(0, 1, 2, 3, 4, 30, 31)),
    "llama2_13b_prefill": FFNConfig("llama2_13b_prefill", 4, d=5120, N=13824,
                                    L=_r(0.7, 13824), k=_r(0.25, 13824), B=512, steps=1,
                                    layers=1, wdtype="bf16"),
}


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _threads() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def storage_from_f32(a: np.ndarray, wdtype: str) -> np.ndarray:
    """float32 values -> storage array: float32 itself, or bf16 bit patterns (uint16, RNE).

    No NaN or infinity is ever drawn, so the plain round-half-to-even bit trick is exact.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    if wdtype == "f32":
        return a
    if wdtype != "bf16":
        raise ValueError(wdtype)
    u = a.view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def _normal_matrix(rows: int, cols: int, std: float, wdtype: str, key: tuple) -> np.ndarray:
    out = np.empty((rows, cols), dtype=np.float32 if wdtype == "f32" else np.uint16)
    nblk = (rows + ROW_BLOCK - 1) // ROW_BLOCK

    def fill(b: int) -> None:
        r0, r1 = b * ROW_BLOCK, min(rows, (b + 1) * ROW_BLOCK)
        a = _rng(*key, b).standard_normal((r1 - r0, cols), dtype=np.float32)
        a *= np.float32(std)
        out[r0:r1] = storage_from_f32(a, wdtype)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def popularity(cfg: FFNConfig, layer: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """(pi, weight): pi[r] is the neuron of popularity rank r+1; weight[n] = rank(n)**-1.1."""
    pi = _rng(cfg.cfg_id, layer, P_PERM).permutation(cfg.N).astype(np.int64)
    w = np.empty(cfg.N, dtype=np.float64)
    w[pi] = np.arange(1, cfg.N + 1, dtype=np.float64) ** (-ZIPF_S)
    return pi, w


def loaded_ids(cfg: FFNConfig, layer: int = 0) -> np.ndarray:
    """The L most popular neurons, in popularity order (int32, not sorted by id); every neuron
    for a dense layer."""
    pi, _ = popularity(cfg, layer)
    return pi[: cfg.L_of(layer)].astype(np.int32)


def layer_weights(cfg: FFNConfig, layer: int = 0):
    """(W_gate [N][d], W_up [N][d], W_down [d][N]) in storage form (uint16 bf16 bits or f32)."""
    d, N = cfg.d, cfg.N
    wg = _normal_matrix(N, d, W_STD, cfg.wdtype, (cfg.cfg_id, layer, P_GATE))
    wu = _normal_matrix(N, d, W_STD, cfg.wdtype, (cfg.cfg_id, layer, P_UP))
    wd = _normal_matrix(d, N, W_STD, cfg.wdtype, (cfg.cfg_id, layer, P_DOWN))
    return wg, wu, wd


def tokens_x(cfg: FFNConfig, tokens, layer: int = 0) -> np.ndarray:
    """x rows for the given token numbers, N(0, 1), storage form, shape [len(tokens)][d]."""
    tokens = list(tokens)
    out = np.empty((len(tokens), cfg.d), dtype=np.float32 if cfg.wdtype == "f32" else np.uint16)
    for i, t in enumerate(tokens):
        a = _rng(cfg.cfg_id, layer, P_X, t).standard_normal(cfg.d, dtype=np.float32)
        out[i] = storage_from_f32(a, cfg.wdtype)
    return out


def _loaded_sorted(cfg: FFNConfig, layer: int) -> np.ndarray:
    return np.sort(loaded_ids(cfg, layer)).astype(np.int64)


def es_keys(cfg: FFNConfig, tokens, layer: int = 0) -> np.ndarray:
    """Efraimidis-Spirakis sampling keys log(u)/w over the loaded neurons.

    Shape [len(tokens)][L], float32; column s belongs to the loaded neuron with the s-th
    smallest original id. Hot-core neurons (if any) get +inf.
    """
    tokens = list(tokens)
    ids = _loaded_sorted(cfg, layer)
    L = len(ids)
    pi, w = popularity(cfg, layer)
    wl = w[ids]
    hot = np.zeros(cfg.N, dtype=bool)
    if cfg.hot:
        hot[pi[: cfg.hot]] = True
    hot_l = hot[ids]
    out = np.empty((len(tokens), L), dtype=np.float32)
    for i, t in enumerate(tokens):
        u = _rng(cfg.cfg_id, layer, P_KEYS, t).random(L)
        u = np.maximum(u, np.finfo(np.float64).tiny)
        key = np.log(u) / wl
        key[hot_l] = np.inf
        out[i] = key.astype(np.float32)
    return out


def active_sets(cfg: FFNConfig, tokens, layer: int = 0) -> list[np.ndarray]:
    """Per-token active sets as original neuron ids (int32, ascending).

    The k members with the largest sampling keys; keys are continuous, so ties do not occur.
    A dense layer's set is every neuron.
    """
    ids = _loaded_sorted(cfg, layer)
    if layer in cfg.dense_layers:
        return [ids.astype(np.int32) for _ in tokens]
    keys = es_keys(cfg, tokens, layer)
    out = []
    for row in keys:
        pick = np.argpartition(-row.astype(np.float64), cfg.k - 1)[: cfg.k] if cfg.k else []
        out.append(np.sort(ids[np.asarray(pick, dtype=np.int64)]).astype(np.int32))
    return out


def csr_from_sets(sets) -> tuple[np.ndarray, np.ndarray]:
    """Concatenate per-token id lists into (offsets [T+1] int32, ids [nnz] int32)."""
    offsets = np.zeros(len(sets) + 1, dtype=np.int64)
    for i, s in enumerate(sets):
        offsets[i + 1] = offsets[i] + len(s)
    ids = np.concatenate([np.asarray(s, dtype=np.int32) for s in sets]) if sets else \
        np.zeros(0, dtype=np.int32)
    return offsets.astype(np.int32), ids.astype(np.int32)
