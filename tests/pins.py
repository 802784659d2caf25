"""Pins for the oracle: checks fixed by the paper and by mathematics, not by the oracle itself.

Every check takes an implementation namespace ``impl`` (the oracle module, or a copy of it
with a planted mistake) and raises AssertionError on failure. The references used here are
closed forms, brute force on tiny inputs, hand-typed expectations, printed values of the paper,
and library routines (NumPy matmul, SciPy's logistic, PyTorch's bf16 conversion) — never the
oracle's own code.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0.0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def _f64(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _masked_dense(x, wg, wu, wd, mask):
    """Library reference: W_down @ (mask * SiLU(W_gate x) * (W_up x)) with SciPy's logistic."""
    from scipy.special import expit

    xf = _f64(x)
    G = _f64(wg) @ xf
    U = _f64(wu) @ xf
    return _f64(wd) @ (np.asarray(mask, np.float64) * G * expit(G) * U)


def _problem(seed, N, d, wdtype="f32", scale=0.3):
    rng = np.random.default_rng(seed)
    def draw(*shape):
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
        if wdtype == "bf16":
            return (a.view(np.uint32) >> 16).astype(np.uint16)   # truncation is fine for inputs
        return a
    return draw(N, d), draw(N, d), draw(d, N), draw(d)


# ------------------------------------------------------------------------------------------
def pin_silu(impl):
    assert impl.silu(0.0) == 0.0
    assert impl.sigmoid(0.0) == 0.5
    assert abs(impl.sigmoid(math.log(3.0)) - 0.75) < 1e-15
    for g in [-30.0, -5.0, -1.5, -0.25, 0.3, 2.0, 7.0, 30.0]:
        # SiLU(-g) = -g * (1 - sigma(g)) = SiLU(g) - g
        assert abs(impl.silu(-g) - (impl.silu(g) - g)) <= 1e-12 * max(1.0, abs(g))
    assert abs(impl.silu(60.0) - 60.0) <= 1e-13
    assert abs(impl.silu(-60.0) - (-60.0 * math.exp(-60.0))) <= 1e-12 * 60.0 * math.exp(-60.0)
    from scipy.special import expit
    for g in np.linspace(-12, 12, 97):
        ref = g * expit(g)
        assert abs(impl.silu(float(g)) - ref) <= 1e-14 * max(1.0, abs(ref))


# ------------------------------------------------------------------------------------------
def _topk_bruteforce(s, k, mode):
    """O(L^2) definition: i is chosen iff fewer than k entries precede it."""
    v = np.abs(s) if mode == "abs" else np.array(s, dtype=np.float64)
    L = len(v)

    def precedes(j, i):  # does j come before i?
        nj, ni = math.isnan(v[j]), math.isnan(v[i])
        if nj and ni:
            return j < i
        if nj:
            return False
        if ni:
            return True
        if v[j] != v[i]:
            return v[j] > v[i]
        return j < i

    rank = [sum(1 for j in range(L) if j != i and precedes(j, i)) for i in range(L)]
    return [i for i in range(L) if rank[i] < k]


def pin_topk(impl):
    # hand cases
    assert list(impl.select_topk([5.0, 5.0, 5.0, 5.0], 2)) == [0, 1]
    assert list(impl.select_topk([-0.0, 0.0], 1, "raw")) == [0]
    assert list(impl.select_topk([0.0, -0.0], 1, "raw")) == [0]
    assert list(impl.select_topk([float("nan"), -math.inf], 1, "raw")) == [1]
    assert list(impl.select_topk([float("nan"), 0.0], 1, "abs")) == [1]
    assert list(impl.select_topk([-3.0, 2.0], 1, "abs")) == [0]
    assert list(impl.select_topk([-3.0, 2.0], 1, "raw")) == [1]
    assert list(impl.select_topk([1.0, 9.0, 3.0, 7.0], 2, "raw")) == [1, 3]
    assert list(impl.select_topk([1.0, 2.0, 3.0], 0)) == []
    assert list(impl.select_topk([1.0, 2.0, 3.0], 3)) == [0, 1, 2]
    try:
        impl.select_topk([1.0, 2.0], 3)
    except ValueError:
        pass
    else:
        raise AssertionError("k > L must be rejected")
    # brute force with ties, signed zeros, NaN and infinities
    rng = np.random.default_rng(7)
    pool = np.array([0.0, -0.0, 1.0, -1.0, 2.5, -2.5, math.inf, -math.inf, math.nan, 0.125])
    for trial in range(60):
        L = int(rng.integers(1, 23))
        s = pool[rng.integers(0, len(pool), L)] if trial % 2 else rng.standard_normal(L).round(1)
        for mode in ("abs", "raw"):
            for k in range(L + 1):
                got = list(impl.select_topk(s, k, mode))
                assert got == _topk_bruteforce(s, k, mode), (s, k, mode, got)


# ------------------------------------------------------------------------------------------
def pin_compact(impl):
    N, d = 5, 3
    wg = np.array([[100 * n + i for i in range(d)] for n in range(N)], dtype=np.float32)
    wu = np.array([[1000 + 100 * n + i for i in range(d)] for n in range(N)], dtype=np.float32)
    wd = np.array([[10 * i + n for n in range(N)] for i in range(d)], dtype=np.float32)
    c = impl.compact(wg, wu, wd, [4, 1, 3])
    assert list(c["slot_to_orig"]) == [1, 3, 4]
    assert list(c["orig_to_slot"]) == [-1, 0, -1, 1, 2]
    assert c["gate_up_c"].shape == (3, 2, 3) and c["down_c"].shape == (3, 3)
    assert c["gate_up_c"][0].tolist() == [[100, 101, 102], [1100, 1101, 1102]]
    assert c["gate_up_c"][1].tolist() == [[300, 301, 302], [1300, 1301, 1302]]
    assert c["gate_up_c"][2].tolist() == [[400, 401, 402], [1400, 1401, 1402]]
    # down_proj column n of W_down [d][N] = (n, 10+n, 20+n)
    assert c["down_c"].tolist() == [[1, 11, 21], [3, 13, 23], [4, 14, 24]]
    # order of the loaded list does not matter
    c2 = impl.compact(wg, wu, wd, [3, 4, 1])
    for key in c:
        assert np.array_equal(c[key], c2[key])
    # bf16 bit patterns are copied, not converted
    bits = (np.arange(N * d, dtype=np.uint16) * 257).reshape(N, d)
    dbits = (np.arange(d * N, dtype=np.uint16) * 131).reshape(d, N)
    cb = impl.compact(bits, bits ^ np.uint16(0x8000), dbits, [0, 2])
    assert cb["gate_up_c"].dtype == np.uint16
    assert np.array_equal(cb["gate_up_c"][1, 0], bits[2])
    assert np.array_equal(cb["gate_up_c"][1, 1], bits[2] ^ np.uint16(0x8000))
    assert np.array_equal(cb["down_c"][1], dbits[:, 2])
    # compacted size: three matrices of L neurons (Eq. 2's complement)
    L = 2
    nbytes = cb["gate_up_c"].nbytes + cb["down_c"].nbytes
    assert nbytes == 3 * d * L * 2 == impl.compacted_bytes(d, L, 2)
    for bad, exc in (([0, 0], "Duplicate"), ([5], "Range"), ([-1], "Range")):
        try:
            impl.compact(wg, wu, wd, bad)
        except ValueError as e:
            assert exc in type(e).__name__, (bad, type(e))
        else:
            raise AssertionError(f"compact({bad}) must fail")


def pin_remap(impl):
    o2s = np.array([-1, 0, -1, 1, 2], dtype=np.int32)
    assert list(impl.remap(o2s, [4, 1, 3])) == [2, 0, 1]
    assert list(impl.remap(o2s, [])) == []
    for bad, exc in (([2], "NotLoaded"), ([5], "Range"), ([-1], "Range")):
        try:
            impl.remap(o2s, bad)
        except ValueError as e:
            assert exc in type(e).__name__
        else:
            raise AssertionError(f"remap({bad}) must fail")


# ------------------------------------------------------------------------------------------
def pin_ffn_invariants(impl):
    for wdtype in ("f32", "bf16"):
        N, d = 40, 24
        wg, wu, wd, x = _problem(11, N, d, wdtype)
        # (1) every neuron loaded and active == dense SwiGLU
        full = impl.compact(wg, wu, wd, list(range(N)))
        y_all = impl.selective_ffn(x, list(range(N)), full["gate_up_c"], full["down_c"])
        assert _rel(y_all, _masked_dense(x, wg, wu, wd, np.ones(N))) <= 1e-12
        # (2) compaction + remap == full matrices restricted to the active set
        rng = np.random.default_rng(3)
        loaded = rng.permutation(N)[:30]
        c = impl.compact(wg, wu, wd, loaded)
        active = rng.permutation(loaded)[:13]
        slots = impl.remap(c["orig_to_slot"], active)
        mask = np.zeros(N)
        mask[active] = 1.0
        y = impl.selective_ffn(x, slots, c["gate_up_c"], c["down_c"])
        assert _rel(y, _masked_dense(x, wg, wu, wd, mask)) <= 1e-12
        # (3) empty set -> exact zeros
        y0 = impl.selective_ffn(x, [], c["gate_up_c"], c["down_c"])
        assert y0.shape == (d,) and not np.any(y0)
        # (4) order of the index list does not matter
        y_perm = impl.selective_ffn(x, slots[::-1].copy(), c["gate_up_c"], c["down_c"])
        assert _rel(y_perm, y) <= 1e-12
        # (5) additivity over disjoint sets
        a, b = slots[:6], slots[6:]
        ya = impl.selective_ffn(x, a, c["gate_up_c"], c["down_c"])
        yb = impl.selective_ffn(x, b, c["gate_up_c"], c["down_c"])
        assert _rel(ya + yb, y) <= 1e-12
        # (6) one neuron: its activation times its down_proj column
        n = int(active[0])
        m1 = np.zeros(N)
        m1[n] = 1.0
        y1 = impl.selective_ffn(x, [int(c["orig_to_slot"][n])], c["gate_up_c"], c["down_c"])
        assert _rel(y1, _masked_dense(x, wg, wu, wd, m1)) <= 1e-12
        # (7) x = 0 -> y = 0
        xz = np.zeros_like(x)
        assert not np.any(impl.selective_ffn(xz, slots, c["gate_up_c"], c["down_c"]))
    # (8) brute force over every subset of a 6-neuron FFN
    N, d = 6, 5
    wg, wu, wd, x = _problem(5, N, d)
    c = impl.compact(wg, wu, wd, list(range(N)))
    for r in range(N + 1):
        for sub in itertools.combinations(range(N), r):
            mask = np.zeros(N)
            mask[list(sub)] = 1.0
            y = impl.selective_ffn(x, list(sub), c["gate_up_c"], c["down_c"])
            ref = _masked_dense(x, wg, wu, wd, mask)
            if r == 0:
                assert not np.any(y)
            else:
                assert _rel(y, ref) <= 1e-12, sub


def pin_hand_integer(impl):
    """Integer weights and x: g and u are integers, y has a closed form in exp()."""
    x = np.array([2.0, -1.0], dtype=np.float32)
    wg = np.array([[1, 0], [0, 0], [1, 1]], dtype=np.float32)       # g = (2, 0, 1)
    wu = np.array([[1, -1], [2, 1], [0, 2]], dtype=np.float32)       # u = (3, 3, -2)
    wd = np.array([[1, 2, 3], [-1, 0, 4]], dtype=np.float32)         # [d=2][N=3]
    c = impl.compact(wg, wu, wd, [0, 1, 2])
    s2 = 1.0 / (1.0 + math.exp(-2.0))
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    h = [2.0 * s2 * 3.0, 0.0, 1.0 * s1 * (-2.0)]
    y = impl.selective_ffn(x, [0, 1, 2], c["gate_up_c"], c["down_c"])
    expect = [h[0] * 1 + h[1] * 2 + h[2] * 3, h[0] * (-1) + h[1] * 0 + h[2] * 4]
    assert np.allclose(y, expect, rtol=1e-15, atol=1e-15), (y, expect)
    y2 = impl.selective_ffn(x, [2], c["gate_up_c"], c["down_c"])
    assert np.allclose(y2, [3 * h[2], 4 * h[2]], rtol=1e-15, atol=0)


# ------------------------------------------------------------------------------------------
def pin_rmsnorm(impl):
    import torch

    def bits(vals):
        return (np.asarray(vals, np.float32).view(np.uint32) >> 16).astype(np.uint16)

    # exactly representable values are kept; halfway cases go to the even neighbour
    assert list(impl.round_to_bf16_bits(np.array([1.0, -2.5, 0.0]))) == list(bits([1.0, -2.5, 0.0]))
    assert impl.round_to_bf16_bits(np.array([1.0 + 2.0**-8]))[0] == bits([1.0])[0]
    assert impl.round_to_bf16_bits(np.array([1.0 + 3 * 2.0**-8]))[0] == bits([1.0 + 2.0**-6])[0]
    assert impl.round_to_bf16_bits(np.array([1.0 + 2.0**-8 + 2.0**-20]))[0] == bits([1.0 + 2.0**-7])[0]
    # agrees with PyTorch's bf16 conversion on float32-representable values
    v = np.random.default_rng(2).standard_normal(4096).astype(np.float32)
    tb = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(impl.round_to_bf16_bits(v.astype(np.float64)), tb)
    # r = x + y = (3, 4): mean square 12.5
    x = bits([1.0, 2.0])
    out = impl.residual_rmsnorm_bf16(x, np.array([2.0, 2.0]), eps=1e-5)
    want = torch.tensor([3.0 / math.sqrt(12.5 + 1e-5), 4.0 / math.sqrt(12.5 + 1e-5)],
                        dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(out, want), (out, want)
    # with eps = 0, scaling r by a power of two changes nothing
    xr = bits(np.random.default_rng(4).standard_normal(64))
    yr = np.random.default_rng(5).standard_normal(64)
    a = impl.residual_rmsnorm_bf16(xr, yr, eps=0.0)
    xs = bits(_f64(xr) * 8.0)
    b = impl.residual_rmsnorm_bf16(xs, yr * 8.0, eps=0.0)
    assert np.array_equal(a, b)
    # the normalised vector has unit mean square (before rounding)
    rv = _f64(a)
    assert abs(float(np.mean(rv * rv)) - 1.0) < 1e-2


def pin_memory(impl):
    with open(os.path.join(GOLDEN, "eq2_llama32_3b.json")) as f:
        g = json.load(f)
    dm = impl.memory_saving(g["n_ffn"], g["r_load"], g["r_layer"], g["s_bytes"])
    assert abs(dm / 1e9 - g["delta_m_gb"]) < 5e-4
    # per layer: compacted + saved == the whole FFN layer
    d, N, L = 4096, 11008, 7706
    assert impl.compacted_bytes(d, L, 2) + 3 * d * (N - L) * 2 == 3 * d * N * 2
    assert impl.compacted_bytes(d, L, 2) == 189_382_656


# --------------------------------------------------------------------------------------------
# Neuron selection (Selective Computation section) and the profiler score (Eq. 1)
# --------------------------------------------------------------------------------------------
def _lib_activations(X, wg, wu):
    """Library reference: SiLU(X W_gate^T) * (X W_up^T) with NumPy matmul and SciPy's logistic."""
    from scipy.special import expit

    Xf = _f64(X)
    G = Xf @ _f64(wg).T
    U = Xf @ _f64(wu).T
    return G * expit(G) * U


def _gu(wg, wu):
    return np.stack([np.stack([wg[n], wu[n]]) for n in range(wg.shape[0])])


def pin_activations(impl):
    for wdtype in ("f32", "bf16"):
        rng = np.random.default_rng(11)
        wg, wu, wd, _ = _problem(12, 23, 10, wdtype)
        X = (rng.standard_normal((5, 10)) * 0.7).astype(np.float32)
        A = impl.activations(X, _gu(wg, wu))
        assert A.shape == (5, 23)
        assert _rel(A, _lib_activations(X, wg, wu)) <= 1e-13


# hand example: per-token top-2 by |a| (ties to the lower index), frequency over the 3 tokens
_HAND_A = np.array([[0.1, -5.0, 3.0, 0.0, 2.0, -0.5],    # top-2 {1, 2}
                    [4.0, 1.0, -1.0, 6.0, 0.2, 0.3],     # top-2 {0, 3}
                    [-2.0, 2.0, 0.5, 0.0, 7.0, 1.0]])    # top-2 {0, 4}: |-2| = |2|, lower wins
_HAND_COUNTS = [2, 1, 1, 1, 1, 0]


def _dyn_properties(impl, A, static, alpha, n_total):
    """Checks of a dynamic-set result that do not restate the oracle's steps."""
    out, counts = impl.select_dynamic(A, static, alpha, n_total)
    out = [int(v) for v in out]
    T, L = A.shape
    ref = np.zeros(L, dtype=np.int64)
    for t in range(T):
        for j in _topk_bruteforce(A[t], alpha, "abs"):
            ref[j] += 1
    assert np.array_equal(np.asarray(counts), ref)
    assert out == sorted(set(out)) and len(out) == n_total
    assert set(static) <= set(out)
    dyn = [j for j in out if j not in static]
    rest = [j for j in range(L) if j not in out]
    for i in dyn:
        for j in rest:
            assert (ref[i], -i) > (ref[j], -j)


def pin_dynamic_set(impl):
    out, counts = impl.select_dynamic(_HAND_A, [5], 2, 3)
    assert [int(v) for v in out] == [0, 1, 5]
    assert [int(v) for v in counts] == _HAND_COUNTS
    out, _ = impl.select_dynamic(_HAND_A, [0], 2, 4)
    assert [int(v) for v in out] == [0, 1, 2, 3]
    out, _ = impl.select_dynamic(_HAND_A, [], 6, 6)          # alpha = L: every slot
    assert [int(v) for v in out] == list(range(6))
    rng = np.random.default_rng(5)
    for T, L, alpha, ns, n_total in [(7, 20, 5, 3, 9), (1, 12, 4, 2, 5), (9, 16, 1, 0, 4)]:
        A = rng.standard_normal((T, L))
        A[:, rng.integers(0, L, 3)] = 0.5                      # exact ties in |a|
        static = sorted(rng.permutation(L)[:ns].tolist())
        _dyn_properties(impl, A, static, alpha, n_total)
    # from a prompt: the activations are the library's, in float64
    wg, wu, _, _ = _problem(13, 18, 8, "bf16")
    X = (rng.standard_normal((6, 8))).astype(np.float32)
    for mode in ("abs", "raw"):
        got, _ = impl.dynamic_set(X, _gu(wg, wu), [2, 9], 4, 7, mode=mode)
        want, _ = impl.select_dynamic(_lib_activations(X, wg, wu), [2, 9], 4, 7, mode=mode)
        assert np.array_equal(got, want)
    # activations 2^-30 apart in relative terms: float64 tells them apart (the higher slot
    # wins), float32 would round both to one value and give the tie to the lower slot
    wg2 = np.array([[4.0, 0.0], [4.0, 0.0]], np.float32)
    wu2 = np.array([[1.0, 0.0], [1.0, 1.0]], np.float32)
    X2 = np.array([[1.0, 2.0 ** -30]], np.float32)
    got, counts = impl.dynamic_set(X2, _gu(wg2, wu2), [], 1, 1)
    assert [int(v) for v in got] == [1] and [int(v) for v in counts] == [0, 1]
    # the literal "descending order": a large negative activation is not taken in raw mode
    out, counts = impl.select_dynamic(_HAND_A, [], 2, 2, mode="raw")
    assert [int(v) for v in counts] == [1, 1, 1, 1, 2, 0]    # {2, 4}, {0, 3}, {1, 4}
    assert [int(v) for v in out] == [0, 4]
    for bad in (dict(static_slots=[1, 1], alpha=2, n_total=3),
                dict(static_slots=[0, 1, 2], alpha=2, n_total=2),
                dict(static_slots=[7], alpha=2, n_total=3)):
        try:
            impl.select_dynamic(_HAND_A, bad["static_slots"], bad["alpha"], bad["n_total"])
        except Exception:
            continue
        raise AssertionError(f"accepted {bad}")


def pin_profile_scores(impl):
    wg, wu, _, _ = _problem(14, 21, 12, "bf16")
    rng = np.random.default_rng(6)
    X = rng.standard_normal((9, 12)).astype(np.float32)
    s, T = impl.profile_scores(X, _gu(wg, wu))
    assert T == 9
    assert _rel(s, np.abs(_lib_activations(X, wg, wu)).sum(axis=0)) <= 1e-13
    s2, T2 = impl.profile_scores(np.concatenate([X, X]), _gu(wg, wu))
    assert T2 == 18 and _rel(s2, 2 * s) <= 1e-14
    # merging normalises each file by its token count
    m = impl.merge_scores([(np.array([2.0, 4.0]), 2), (np.array([3.0, 0.0]), 3)])
    assert np.allclose(m, [2.0, 2.0], rtol=0, atol=1e-15)
    assert _rel(impl.merge_scores([(s, T), (s2, T2)]), 2 * s / T) <= 1e-14
    # ranking: decreasing score, ties to the lower index, NaN last
    assert [int(v) for v in impl.rank_neurons([1.0, 3.0, 3.0, 0.5])] == [1, 2, 0, 3]
    assert [int(v) for v in impl.rank_neurons([float("nan"), 0.0, -1.0])] == [1, 2, 0]


def pin_loaded_set(impl):
    task = [4, 1, 7, 0, 2, 6, 5, 3]
    model = [1, 2, 4, 3, 0, 7, 6, 5]
    got = [int(v) for v in impl.build_loaded_set(task, model, 2, 5)]
    assert got == [4, 1, 2, 3, 0]          # 1 and 4 are already base: skipped, not counted
    assert [int(v) for v in impl.build_loaded_set(task, model, 3, 3)] == [4, 1, 7]
    assert [int(v) for v in impl.build_loaded_set(task, model, 0, 2)] == [1, 2]
    assert sorted(int(v) for v in impl.build_loaded_set(task, model, 3, 8)) == list(range(8))
    rng = np.random.default_rng(9)
    for _ in range(5):
        N = 50
        t, m = rng.permutation(N), rng.permutation(N)
        nb, nl = int(rng.integers(0, 20)), int(rng.integers(20, 40))
        got = [int(v) for v in impl.build_loaded_set(t, m, nb, nl)]
        assert len(got) == nl == len(set(got))
        assert got[:nb] == t[:nb].tolist()
        # the secondary neurons are the most relevant model-level ones outside the base
        rest = [int(v) for v in m if int(v) not in set(t[:nb].tolist())]
        assert got[nb:] == rest[:nl - nb]
    for bad in ((task, model, 3, 2), (task, model, 1, 9), ([0, 0, 1], [0, 1, 2], 1, 2)):
        try:
            impl.build_loaded_set(*bad)
        except Exception:
            continue
        raise AssertionError(f"accepted {bad}")
    # Table 1 layer range: 21 of 28 layers (r_layer = 0.75 in Eq. 2) and 9 of 16
    with open(os.path.join(GOLDEN, "table1_parameters.json")) as f:
        t1 = json.load(f)
    assert len(impl.selective_layers(t1["n_layers_llama32_3b"])) == 21
    assert len(impl.selective_layers(t1["n_layers_llama32_1b"])) == t1["selected_layers_llama32_1b"]
    assert impl.selective_layers(8) == [5]


def pin_decode(impl):
    # storage formats widen exactly: bf16 bits, IEEE half (closed-form values), float32
    # 0x7F7F: exponent 254 - 127, mantissa 1 + 127/128 -> 255 * 2^120
    assert impl.decode(np.array([0x3F80, 0xBF40, 0x7F7F], np.uint16)).tolist() == \
        [1.0, -0.75, 255.0 * 2.0 ** 120]
    h = impl.decode(np.array([1 / 3, 65504.0, 2.0 ** -24, -2.5], np.float16))
    assert h.tolist() == [0.333251953125, 65504.0, 5.960464477539063e-08, -2.5]
    assert impl.decode(np.array([0.1], np.float32)).tolist() == [float(np.float32(0.1))]
    # a half-precision layer computes like its float64 widening (compaction copies bits)
    wg, wu, wd, x = _problem(21, 9, 8, "f32")
    c16 = impl.compact(wg.astype(np.float16), wu.astype(np.float16), wd.astype(np.float16),
                       range(9))
    assert c16["gate_up_c"].dtype == np.float16
    y = impl.selective_ffn(x.astype(np.float16), [0, 3, 8], c16["gate_up_c"], c16["down_c"])
    mask = np.isin(np.arange(9), [0, 3, 8]).astype(float)
    ref = _masked_dense(x.astype(np.float16).astype(np.float32), wg.astype(np.float16).astype(
        np.float32), wu.astype(np.float16).astype(np.float32),
        wd.astype(np.float16).astype(np.float32), mask)
    assert _rel(y, ref) <= 1e-13


ALL_PINS = [pin_silu, pin_topk, pin_compact, pin_remap, pin_ffn_invariants, pin_hand_integer,
            pin_rmsnorm, pin_memory, pin_activations, pin_dynamic_set, pin_profile_scores,
            pin_loaded_set, pin_decode]
