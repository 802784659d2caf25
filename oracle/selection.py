"""Oracle for the neuron-selection steps around the hot path — TEST INFRASTRUCTURE ONLY.

Imported by the tests, the smoke check and the benchmark's CPU baseline, never by the product
path; it shares no code with the GPU library or its binding.

* ``activations`` (LLM Profiler section): the activation of neuron n on token t is the value at
  the down_proj input, a_n(t) = SiLU(gate_n . x_t) * (up_n . x_t) for a SwiGLU FFN. Computed in
  float64 with library matrix products for the two projections.
* ``select_dynamic`` / ``dynamic_set`` (Selective Computation section): for each prompt token,
  the loaded neurons are ranked by activation, descending, and the top alpha kept; the
  frequency of every neuron over these per-token lists is counted; the most frequent neurons
  form the dynamic set, which is combined with the static neurons until the computed total is
  reached.
* ``profile_scores`` (LLM Profiler section, Eq. 1): s_n = sum over the scored tokens of
  |a_n(t)|, stored with the number of tokens.
* ``merge_scores`` (LLM Profiler section): score files are merged by dividing each by its token
  count and summing.
* ``rank_neurons`` (LLM Profiler section): neuron indices in decreasing order of importance.
* ``build_loaded_set`` (Selective Loading section): the base neurons are the top delta of the
  task-specific ranking; secondary neurons are added from the model-level ranking, most
  relevant first, until the loading threshold gamma is reached.
* ``selective_layers`` (Table 1): selective loading applies to the FFN layers from the fifth
  to the second-to-last, 0-based [5, n - 2).

Readings taken where the paper is silent:

* ranking key of the per-token selection: |a| (the profiler scores absolute activations),
  or a itself (``mode="raw"``, the section's literal "descending order"); ties go to the lower
  index, -0 equals +0, NaN ranks below every number (as ``select_topk``); the activations are
  the exact float64 values of the definition (the paper fixes no precision for them);
* ties in frequency go to the lower slot;
* "combine until phi is reached": the result holds every static slot plus the
  n_total - n_static most frequent non-static slots, so its size is exactly n_total; a slot
  that no token selected can fill the remainder (count 0, lower slots first);
* ties in the importance ranking go to the lower neuron index;
* the loaded set is returned in the order it is filled (base, then secondary); a secondary
  neuron already in the base set is skipped, not counted.
"""
from __future__ import annotations

import math

import numpy as np

from .ffn import OracleError, DuplicateError, RangeError, decode, select_topk, silu


def activations(X: np.ndarray, gate_up_c: np.ndarray) -> np.ndarray:
    """a[t][j] = SiLU(gate_j . x_t) * (up_j . x_t) for every token t and slot j (float64)."""
    Xf = decode(X).reshape(-1, gate_up_c.shape[-1])
    G = Xf @ decode(gate_up_c[:, 0]).T
    U = Xf @ decode(gate_up_c[:, 1]).T
    A = np.empty_like(G)
    for t in range(G.shape[0]):
        for j in range(G.shape[1]):
            A[t, j] = silu(float(G[t, j])) * float(U[t, j])
    return A


def select_dynamic(A: np.ndarray, static_slots, alpha: int, n_total: int, mode: str = "abs"):
    """The Selective Computation steps on a given activation matrix A[T][L].

    Returns (slots ascending, counts[L]).
    """
    A = np.asarray(A, dtype=np.float64)
    T, L = A.shape
    static = [int(v) for v in np.asarray(static_slots).reshape(-1).tolist()]
    if len(set(static)) != len(static):
        raise DuplicateError("static slots repeat")
    for v in static:
        if v < 0 or v >= L:
            raise RangeError(f"static slot {v} outside [0, {L})")
    if alpha < 0 or alpha > L or n_total < len(static) or n_total > L:
        raise OracleError(f"alpha={alpha}, n_total={n_total}, {len(static)} static, L={L}")
    # 1. per token: the top alpha loaded neurons by activation
    counts = np.zeros(L, dtype=np.int64)
    for t in range(T):
        for j in select_topk(A[t], alpha, mode).tolist():
            counts[j] += 1
    # 2. the most frequent neurons that are not static, until n_total slots in all
    keys = counts.astype(np.float64)
    for v in static:
        keys[v] = -1.0
    dyn = select_topk(keys, n_total - len(static), "raw").tolist()
    return np.array(sorted(set(static) | set(dyn)), dtype=np.int32), counts


def dynamic_set(X: np.ndarray, gate_up_c: np.ndarray, static_slots, alpha: int, n_total: int,
                mode: str = "abs"):
    """Dynamic-set construction for a prompt X[T][d] over a compacted layer, on the float64
    activations of every loaded slot."""
    return select_dynamic(activations(X, gate_up_c), static_slots, alpha, n_total, mode)


def profile_scores(X: np.ndarray, gate_up: np.ndarray):
    """Eq. 1 over the tokens X[T][d]: (s[n] = sum_t |a_n(t)|, T)."""
    A = activations(X, gate_up)
    s = np.zeros(A.shape[1], dtype=np.float64)
    for t in range(A.shape[0]):
        for n in range(A.shape[1]):
            s[n] += abs(A[t, n])
    return s, A.shape[0]


def merge_scores(files) -> np.ndarray:
    """Sum of the score files' scores, each divided by its token count."""
    out = None
    for s, T in files:
        if T <= 0:
            raise OracleError("a score file needs at least one token")
        v = np.asarray(s, dtype=np.float64) / float(T)
        out = v if out is None else out + v
    if out is None:
        raise OracleError("no score files")
    return out


def rank_neurons(scores) -> np.ndarray:
    """Neuron indices by decreasing score; equal scores keep the lower index first."""
    v = np.asarray(scores, dtype=np.float64).reshape(-1)
    keys = [((1, 0.0) if math.isnan(v[n]) else (0, -float(v[n])), n) for n in range(v.shape[0])]
    return np.array([n for _, n in sorted(keys)], dtype=np.int32)


def build_loaded_set(task_rank, model_rank, n_base: int, n_loaded: int) -> np.ndarray:
    """Base = task_rank[:n_base]; then model_rank in order, skipping chosen neurons, until
    n_loaded neurons in all. Both rankings list every neuron once."""
    task = [int(v) for v in np.asarray(task_rank).reshape(-1).tolist()]
    model = [int(v) for v in np.asarray(model_rank).reshape(-1).tolist()]
    N = len(task)
    if len(model) != N:
        raise OracleError("rankings of different lengths")
    for r in (task, model):
        if sorted(r) != list(range(N)):
            raise OracleError("a ranking must list every neuron exactly once")
    if n_base < 0 or n_loaded < n_base or n_loaded > N:
        raise OracleError(f"n_base={n_base}, n_loaded={n_loaded}, N={N}")
    chosen = task[:n_base]
    seen = set(chosen)
    for n in model:
        if len(chosen) == n_loaded:
            break
        if n not in seen:
            chosen.append(n)
            seen.add(n)
    return np.array(chosen, dtype=np.int32)


def selective_layers(n_layers: int, first: int = 5, last: int = -2) -> list:
    """0-based indices of the layers whose FFN is loaded selectively: [first, n + last)."""
    return [i for i in range(n_layers) if first <= i < n_layers + last]
