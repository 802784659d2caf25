"""Plant plausible mistakes in copies of the oracle and check that the pins catch each one.

This shows the pins constrain every part of the oracle: a dropped term, a wrong sign, a
transposed operand, an off-by-one index or a wrong tie rule must make at least one pin fail.
"""
import math
import types

import numpy as np
import pytest

import oracle
from oracle import ffn as O
from tests import pins


def _impl(**over):
    ns = types.SimpleNamespace(**{k: getattr(oracle, k) for k in oracle.__all__}) \
        if hasattr(oracle, "__all__") else types.SimpleNamespace(**vars(oracle))
    for k, v in over.items():
        setattr(ns, k, v)
    return ns


def _ffn_with(hfun, rowsel=None):
    """selective_ffn with a replaced activation h(g, u) or a replaced down-row selection."""
    def f(x, slots, gate_up_c, down_c):
        xf = O.decode(x).reshape(-1)
        y = np.zeros(xf.shape[0])
        for j in np.asarray(slots).reshape(-1).tolist():
            g = float(np.dot(O.decode(gate_up_c[j, 0]), xf))
            u = float(np.dot(O.decode(gate_up_c[j, 1]), xf))
            row = O.decode(down_c[j]) if rowsel is None else rowsel(gate_up_c, down_c, j)
            y += hfun(g, u) * row
        return y
    return f


def _silu_wrong_sign(g):
    return g * O.sigmoid(-g)


def _topk_high_index_ties(scores, k, mode="abs"):
    v = np.abs(np.asarray(scores, float)) if mode == "abs" else np.asarray(scores, float)
    order = sorted(range(len(v)), key=lambda j: (math.isnan(v[j]), -v[j] if not math.isnan(v[j]) else 0, -j))
    if k > len(v):
        raise ValueError
    return np.array(sorted(order[:k]), dtype=np.int32)


def _topk_no_abs(scores, k, mode="abs"):
    return O.select_topk(scores, k, "raw")


def _topk_nan_high(scores, k, mode="abs"):
    v = np.abs(np.asarray(scores, float)) if mode == "abs" else np.asarray(scores, float)
    if k > len(v):
        raise ValueError
    order = sorted(range(len(v)), key=lambda j: (0, j) if math.isnan(v[j]) else (1, -v[j], j))
    return np.array(sorted(order[:k]), dtype=np.int32)


def _compact_transposed_down(wg, wu, wd, loaded):
    c = O.compact(wg, wu, wd, loaded)
    S = c["slot_to_orig"]
    d = wg.shape[1]
    # mistake: reads row n of W_down (wrapping) instead of column n
    c["down_c"] = np.stack([wd[int(n) % wd.shape[0], :d] if wd.shape[1] >= d else
                            np.resize(wd[int(n) % wd.shape[0]], d) for n in S]).astype(wd.dtype)
    return c


def _compact_unsorted(wg, wu, wd, loaded):
    # mistake: slots in list order instead of ascending id
    ids = [int(v) for v in loaded]
    c = O.compact(wg, wu, wd, loaded)
    N = wg.shape[0]
    o2s = np.full(N, -1, np.int32)
    for s, n in enumerate(ids):
        o2s[n] = s
    c["slot_to_orig"] = np.array(ids, np.int32)
    c["orig_to_slot"] = o2s
    c["gate_up_c"] = np.stack([np.stack([wg[n], wu[n]]) for n in ids])
    c["down_c"] = np.stack([wd[:, n] for n in ids])
    return c


def _remap_off_by_one(o2s, ids):
    out = O.remap(o2s, ids)
    return np.minimum(out + 1, len(o2s) - 1).astype(np.int32)


def _ffn_drops_last(x, slots, gate_up_c, down_c):
    s = np.asarray(slots).reshape(-1)
    return O.selective_ffn(x, s[:-1] if len(s) > 1 else s, gate_up_c, down_c)


def _rms_no_sq(x, y, eps=1e-5):
    r = O.decode(x) + np.asarray(y, float)
    return O.round_to_bf16_bits(r / math.sqrt(abs(float(np.mean(r))) + eps))


def _rms_truncate(x, y, eps=1e-5):
    r = O.decode(x) + np.asarray(y, float)
    v = (r / math.sqrt(float(np.mean(r * r)) + eps)).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def _saving_wrong(n, rl, rlay, s):
    return n * rl * rlay * s


from oracle import selection as S


def _dyn_with(per_token_mode="abs", freq_high_ties=False, exclude_static=True, first_token_only=False):
    def f(A, static_slots, alpha, n_total, mode="abs"):
        A = np.asarray(A, float)
        T, L = A.shape
        static = [int(v) for v in np.asarray(static_slots).reshape(-1).tolist()]
        if len(set(static)) != len(static) or any(v < 0 or v >= L for v in static):
            raise ValueError
        if n_total < len(static) or n_total > L:
            raise ValueError
        counts = np.zeros(L, np.int64)
        for t in range(1 if first_token_only else T):
            for j in O.select_topk(A[t], alpha, per_token_mode).tolist():
                counts[j] += 1
        keys = counts.astype(float)
        if exclude_static:
            keys[static] = -1.0
        order = sorted(range(L), key=lambda j: (-keys[j], -j if freq_high_ties else j))
        dyn = order[:n_total - len(static)]
        return np.array(sorted(set(static) | set(dyn)), np.int32), counts
    return f


def _dyn_float32(X, gate_up_c, static_slots, alpha, n_total, mode="abs"):
    # mistake: the ranking decision taken on activations rounded to float32
    A = S.activations(X, gate_up_c).astype(np.float32).astype(np.float64)
    return S.select_dynamic(A, static_slots, alpha, n_total, mode)


def _dyn_mode_ignored(X, gate_up_c, static_slots, alpha, n_total, mode="abs"):
    return S.select_dynamic(S.activations(X, gate_up_c), static_slots, alpha, n_total)


def _act_swapped(X, gate_up_c):
    sw = gate_up_c[:, ::-1].copy()
    return S.activations(X, sw)


def _profile_signed(X, gate_up):
    A = S.activations(X, gate_up)
    return A.sum(axis=0), A.shape[0]


def _merge_no_norm(files):
    return sum(np.asarray(s, float) for s, _ in files)


def _rank_ascending(scores):
    return S.rank_neurons(scores)[::-1].copy()


def _loaded_counts_skips(task_rank, model_rank, n_base, n_loaded):
    task = [int(v) for v in task_rank]
    chosen = task[:n_base]
    for n in [int(v) for v in model_rank][:n_loaded - n_base]:   # mistake: skips use up slots
        if n not in chosen:
            chosen.append(n)
    return np.array(chosen, np.int32)


def _loaded_model_first(task_rank, model_rank, n_base, n_loaded):
    return S.build_loaded_set(model_rank, task_rank, n_base, n_loaded)


def _layers_inclusive(n_layers, first=5, last=-2):
    return [i for i in range(n_layers) if first <= i <= n_layers + last]


MUTANTS = {
    "loaded_skips_count": dict(build_loaded_set=_loaded_counts_skips),
    "loaded_model_first": dict(build_loaded_set=_loaded_model_first),
    "layers_inclusive": dict(selective_layers=_layers_inclusive),
    "dyn_raw_key": dict(select_dynamic=_dyn_with(per_token_mode="raw")),
    "dyn_freq_high_index_ties": dict(select_dynamic=_dyn_with(freq_high_ties=True)),
    "dyn_static_not_excluded": dict(select_dynamic=_dyn_with(exclude_static=False)),
    "dyn_first_token_only": dict(select_dynamic=_dyn_with(first_token_only=True)),
    "dyn_float32_activations": dict(dynamic_set=_dyn_float32),
    "dyn_mode_ignored": dict(dynamic_set=_dyn_mode_ignored),
    "activations_gate_up_swapped": dict(activations=_act_swapped),
    "profile_signed": dict(profile_scores=_profile_signed),
    "merge_not_normalised": dict(merge_scores=_merge_no_norm),
    "rank_ascending": dict(rank_neurons=_rank_ascending),
    "silu_sign": dict(silu=_silu_wrong_sign,
                      selective_ffn=_ffn_with(lambda g, u: _silu_wrong_sign(g) * u)),
    "drop_up": dict(selective_ffn=_ffn_with(lambda g, u: O.silu(g))),
    "drop_sigmoid": dict(selective_ffn=_ffn_with(lambda g, u: g * u)),
    "gate_up_swapped": dict(selective_ffn=_ffn_with(lambda g, u: O.silu(u) * g)),
    "down_from_gate": dict(selective_ffn=_ffn_with(lambda g, u: O.silu(g) * u,
                                                   rowsel=lambda gu, dn, j: O.decode(gu[j, 0]))),
    "drops_last_term": dict(selective_ffn=_ffn_drops_last),
    "topk_high_index_ties": dict(select_topk=_topk_high_index_ties),
    "topk_no_abs": dict(select_topk=_topk_no_abs),
    "topk_nan_high": dict(select_topk=_topk_nan_high),
    "compact_transposed_down": dict(compact=_compact_transposed_down),
    "compact_unsorted_slots": dict(compact=_compact_unsorted),
    "remap_off_by_one": dict(remap=_remap_off_by_one),
    "rmsnorm_mean_not_square": dict(residual_rmsnorm_bf16=_rms_no_sq),
    "rmsnorm_truncates": dict(residual_rmsnorm_bf16=_rms_truncate),
    "eq2_uses_r_load": dict(memory_saving=_saving_wrong),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    impl = _impl(**MUTANTS[name])
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, IndexError, TypeError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
