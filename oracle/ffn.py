"""Oracle: fp64 CPU definition of selective loading and selective computation.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the benchmark's CPU
baseline, never by the product path.

What the paper fixes, and what each function follows:

* Neurons (LLM Profiler section): in a Llama/Qwen FFN, neuron n is row n of gate_proj and of
  up_proj in PyTorch [out, in] storage (a "column" in the paper's x·W convention) and column n
  of down_proj. The activation at the down_proj input is a_n = SiLU(gate_n · x) · (up_n · x)
  (SwiGLU).
* Selective loading (Selective Loading section): only the slices of the selected neurons are
  kept; the rest of the FFN is discarded.  -> ``compact``
* Selective computation (Selective Computation section): only active neurons, all of them
  loaded, are computed; inactive ones contribute nothing.  -> ``remap``, ``selective_ffn``
* Dynamic-neuron selection (Selective Computation section): per token, the loaded neurons are
  ranked by activation, descending, and the top alpha kept.  -> ``select_topk``
* Eq. 2 (Memory Footprint section): saving = N_ffn (1 - r_load) r_layer s.  -> ``memory_saving``

Readings taken where the paper is silent:

* ranking key: |value| by default (the profiler scores absolute activations, Eq. 1); raw value
  on request. Ties go to the lower index, -0 equals +0, NaN ranks below every number.
  Returned indices are ascending.
* compacted slots are assigned in ascending original id; duplicates or out-of-range ids are
  errors; an active id that is not loaded is an error.
* the SwiGLU form is SiLU on the gate projection times the up projection.
* the stack workload's layer step is x' = bf16_RNE(r / sqrt(mean(r^2) + 1e-5)) with
  r = x + y and unit gain.

Inputs are the exact storage arrays the GPU receives: float32, IEEE half (float16), or bf16
bit patterns held in uint16. ``decode`` widens them to float64 exactly, so there is no input-rounding ambiguity.
All arithmetic is float64.
"""
from __future__ import annotations

import math

import numpy as np


class OracleError(ValueError):
    pass


class RangeError(OracleError):
    pass


class DuplicateError(OracleError):
    pass


class NotLoadedError(OracleError):
    pass


# --------------------------------------------------------------------------------------------
# storage <-> float64
# --------------------------------------------------------------------------------------------
def decode(a: np.ndarray) -> np.ndarray:
    """Storage array -> float64. uint16 is read as bf16 bits (the upper half of a float32);
    float16 (the paper's weight storage, 2 bytes per parameter in the Memory Footprint section)
    and float32 widen exactly."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if a.dtype == np.float32 or a.dtype == np.float16:
        return a.astype(np.float64)
    raise TypeError(f"unsupported storage dtype {a.dtype}")


def round_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """float64 -> nearest bf16 (ties to even), returned as uint16 bits.

    bf16 keeps 8 significant bits. With v = m * 2**e and 0.5 <= |m| < 1, the rounded value is
    rint(m * 2**8) * 2**(e - 8), where rint rounds half to even. Values here are O(1), far from
    the bf16 subnormal and overflow ranges.
    """
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)
    r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)
    return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# --------------------------------------------------------------------------------------------
# O1 selective loading: compaction (Selective Loading section; Eq. 2 for the sizes)
# --------------------------------------------------------------------------------------------
def compact(w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray, loaded) -> dict:
    """Keep only the loaded neurons' slices.

    w_gate, w_up: [N][d]; w_down: [d][N] (PyTorch [out, in] storage). ``loaded``: ids in any
    order. Slot s holds the loaded neuron with the s-th smallest id. Returns storage-dtype
    copies (bit-exact): gate_up_c [L][2][d] (gate row, then up row), down_c [L][d] (the
    neuron's down_proj column laid out contiguously), slot_to_orig [L], orig_to_slot [N]
    (-1 where not loaded).
    """
    N, d = w_gate.shape
    if w_up.shape != (N, d) or w_down.shape != (d, N):
        raise OracleError("shape mismatch")
    ids = [int(v) for v in np.asarray(loaded).reshape(-1)]
    for v in ids:
        if v < 0 or v >= N:
            raise RangeError(f"loaded id {v} outside [0, {N})")
    if len(set(ids)) != len(ids):
        raise DuplicateError("loaded list has a duplicate id")
    S = sorted(ids)
    L = len(S)
    gate_up_c = np.empty((L, 2, d), dtype=w_gate.dtype)
    down_c = np.empty((L, d), dtype=w_down.dtype)
    orig_to_slot = np.full(N, -1, dtype=np.int32)
    for s, n in enumerate(S):
        gate_up_c[s, 0, :] = w_gate[n, :]
        gate_up_c[s, 1, :] = w_up[n, :]
        down_c[s, :] = w_down[:, n]
        orig_to_slot[n] = s
    return {
        "gate_up_c": gate_up_c,
        "down_c": down_c,
        "slot_to_orig": np.array(S, dtype=np.int32),
        "orig_to_slot": orig_to_slot,
    }


def compacted_bytes(d: int, L: int, s: int) -> int:
    """Bytes of one compacted FFN layer: three matrices of L neurons x d values x s bytes."""
    return 3 * d * L * s


def memory_saving(n_ffn: float, r_load: float, r_layer: float, s: float) -> float:
    """Eq. 2: bytes saved = N_ffn * (1 - r_load) * r_layer * s."""
    return n_ffn * (1.0 - r_load) * r_layer * s


# --------------------------------------------------------------------------------------------
# O2 original id -> slot (Selective Computation: only loaded neurons are computed)
# --------------------------------------------------------------------------------------------
def remap(orig_to_slot: np.ndarray, ids) -> np.ndarray:
    N = len(orig_to_slot)
    out = []
    for v in np.asarray(ids).reshape(-1).tolist():
        if v < 0 or v >= N:
            raise RangeError(f"id {v} outside [0, {N})")
        s = int(orig_to_slot[v])
        if s < 0:
            raise NotLoadedError(f"neuron {v} is not loaded")
        out.append(s)
    return np.array(out, dtype=np.int32)


# --------------------------------------------------------------------------------------------
# O3 per-token top-k over loaded neurons (dynamic-neuron selection)
# --------------------------------------------------------------------------------------------
def select_topk(scores, k: int, mode: str = "abs") -> np.ndarray:
    """Indices of the k best entries of one score row, returned ascending.

    Key: |score| ("abs") or score ("raw"). j precedes i when key_j > key_i, or when they are
    equal and j < i. -0 and +0 are equal keys; NaN ranks after every number.
    """
    v = np.asarray(scores, dtype=np.float64).reshape(-1)
    L = v.shape[0]
    if k < 0 or k > L:
        raise OracleError(f"k={k} outside [0, {L}]")
    if mode == "abs":
        v = np.abs(v)
    elif mode != "raw":
        raise OracleError(mode)
    keys = []
    for j in range(L):
        if math.isnan(v[j]):
            keys.append((1, 0.0, j))
        else:
            keys.append((0, -float(v[j]), j))
    order = sorted(range(L), key=lambda j: keys[j])
    return np.array(sorted(order[:k]), dtype=np.int32)


# --------------------------------------------------------------------------------------------
# O4/O5 selective computation of the SwiGLU FFN
# --------------------------------------------------------------------------------------------
def sigmoid(g: float) -> float:
    """Logistic function, evaluated without overflow on either side."""
    if g >= 0.0:
        return 1.0 / (1.0 + math.exp(-g))
    e = math.exp(g)
    return e / (1.0 + e)


def silu(g: float) -> float:
    return g * sigmoid(g)


def selective_ffn(x: np.ndarray, slots, gate_up_c: np.ndarray, down_c: np.ndarray) -> np.ndarray:
    """y = sum over active slots j of SiLU(gate_j . x) * (up_j . x) * down_j, in float64.

    ``slots`` are compacted slot ids, visited in the order given. An empty set gives y = 0.
    """
    xf = decode(x).reshape(-1)
    d = xf.shape[0]
    L = gate_up_c.shape[0]
    y = np.zeros(d, dtype=np.float64)
    for j in np.asarray(slots).reshape(-1).tolist():
        if j < 0 or j >= L:
            raise RangeError(f"slot {j} outside [0, {L})")
        g = float(np.dot(decode(gate_up_c[j, 0]), xf))
        u = float(np.dot(decode(gate_up_c[j, 1]), xf))
        h = silu(g) * u
        y += h * decode(down_c[j])
    return y


def dense_swiglu(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
                 neuron_mask=None) -> np.ndarray:
    """Dense FFN with library matmuls and SciPy's logistic; optional 0/1 mask over neurons.

    Used only to pin ``selective_ffn`` by invariants; it shares none of its loop.
    """
    from scipy.special import expit

    xf = decode(x).reshape(-1)
    G = decode(w_gate) @ xf
    U = decode(w_up) @ xf
    H = G * expit(G) * U
    if neuron_mask is not None:
        H = H * np.asarray(neuron_mask, dtype=np.float64)
    return decode(w_down) @ H


# --------------------------------------------------------------------------------------------
# O6 layer step of the FFN stack workload
# --------------------------------------------------------------------------------------------
def residual_rmsnorm_bf16(x: np.ndarray, y: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """x' = bf16_RNE(r / sqrt(mean(r^2) + eps)), r = x + y, unit gain; returns uint16 bits."""
    r = decode(x).reshape(-1) + np.asarray(y, dtype=np.float64).reshape(-1)
    ms = float(np.mean(r * r))
    return round_to_bf16_bits(r / math.sqrt(ms + eps))


def stack_step(x: np.ndarray, slots, gate_up_c, down_c, eps: float = 1e-5):
    """One layer of the stack: (y, x_next) with y the selective FFN output."""
    y = selective_ffn(x, slots, gate_up_c, down_c)
    return y, residual_rmsnorm_bf16(x, y, eps)
