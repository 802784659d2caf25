"""GPU parity of the neuron-selection entry points against the oracle.

- si_dynamic_set: with integer-valued weights and x every gate/up product is exact in float32,
  and both sides rank the activations rounded to float32 (the kernels' precision), so the
  result and the counts must agree exactly (ties included: equal inputs give bitwise equal
  activations on both sides). The data is checked to have no near-tie at a boundary. At a
  realistic shape the result is checked for validity against the GPU's own counts, and the
  counts against the oracle's up to ranking near-ties.
- si_profile_scores (Eq. 1): relative L2 <= 1e-5 against the fp64 oracle, bitwise
  reproducible, accumulating.
- si_merge_scores: relative error <= 1e-6; si_rank_neurons: exact, on the same float32 scores
  (ties, -0, NaN).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, say

pytestmark = pytest.mark.gpu


def _bf16(a):
    a = np.asarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)   # exact for small integers


def _int_problem(seed, N, d, L, T, wdtype):
    rng = np.random.default_rng(seed)
    # |g| is mostly large, where SiLU(g) = g in float32: the top activations are then exact
    # integers (equal or at least 1 apart), and bf16 holds every value exactly
    wg = rng.integers(-7, 8, (N, d)).astype(np.float32)
    wu = rng.integers(-7, 8, (N, d)).astype(np.float32)
    wd = rng.integers(-3, 4, (d, N)).astype(np.float32)
    x = rng.integers(-4, 5, (T, d)).astype(np.float32)
    if wdtype == "bf16":
        wg, wu, wd, x = _bf16(wg), _bf16(wu), _bf16(wd), _bf16(x)
    elif wdtype == "f16":
        wg, wu, wd, x = (a.astype(np.float16) for a in (wg, wu, wd, x))
    loaded = rng.permutation(N)[:L].astype(np.int32)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd), torch.from_numpy(loaded))
    return rng, x, ref, gpu


def _margins_ok(A32, alpha):
    """No near-tie at any token's alpha boundary of the float32 keys: the gap is 0 (equal keys,
    broken by index on both sides) or several float32 ulps, above the kernel's exp/divide
    error."""
    for row in np.abs(A32):
        v = np.sort(row)[::-1]
        if 0 < alpha < len(v):
            gap = v[alpha - 1] - v[alpha]
            if gap != 0.0 and gap <= 2e-6 * v[alpha - 1]:
                return False
    return True


@pytest.mark.parametrize("wdtype,T", [("bf16", 37), ("bf16", 300), ("f32", 23), ("f16", 300)])
def test_dynamic_set_exact(wdtype, T):
    N, d, L = 700, 64, 530
    say(f"dynamic set exact {wdtype} T={T}")
    rng, x, ref, gpu = _int_problem(T * 3 + len(wdtype), N, d, L, T, wdtype)
    static = np.sort(rng.permutation(L)[:60]).astype(np.int32)
    alpha, n_total = 75, 160
    A = oracle.activations(x, ref["gate_up_c"]).astype(np.float32).astype(np.float64)
    assert _margins_ok(A, alpha)
    want, want_counts = oracle.dynamic_set(x, ref["gate_up_c"], static, alpha, n_total)
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, n_total)
    assert np.array_equal(host_array(counts), want_counts)
    assert np.array_equal(host_array(got), want)
    # degenerate cases: no static slots; alpha = 0 (all counts 0: lowest slots fill);
    # n_total = n_static (the static set only)
    g2, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static[:0]), alpha, 50)
    assert np.array_equal(host_array(g2), oracle.select_dynamic(A, [], alpha, 50)[0])
    g3, c3 = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), 0, n_total)
    assert not host_array(c3).any()
    assert np.array_equal(host_array(g3), oracle.select_dynamic(A, static, 0, n_total)[0])
    g4, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, len(static))
    assert np.array_equal(host_array(g4), static)
    # every slot: the pick takes all non-static slots
    g5, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, L)
    assert np.array_equal(host_array(g5), np.arange(L, dtype=np.int32))


@pytest.mark.parametrize("L", [16384, 32768, 32769])
def test_dynamic_set_row_length_paths(L):
    """Up to 32768 loaded slots the tokens' choices travel as bitmaps and are counted per word;
    past it, as index lists counted with atomics. Both must give the oracle's result."""
    N, d, T = L + 300, 64, 40
    say(f"dynamic set L={L}")
    rng, x, ref, gpu = _int_problem(L, N, d, L, T, "bf16")
    static = rng.permutation(L)[:3000].astype(np.int32)   # unsorted on purpose
    alpha, n_total = 2500, 6000
    A = oracle.activations(x, ref["gate_up_c"]).astype(np.float32).astype(np.float64)
    assert _margins_ok(A, alpha)
    want, want_counts = oracle.dynamic_set(x, ref["gate_up_c"], np.sort(static), alpha, n_total)
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, n_total)
    assert np.array_equal(host_array(counts), want_counts)
    assert np.array_equal(host_array(got), want)


def test_dynamic_set_realistic_shape():
    """13B-like rows (d = 5120) with random N(0, 0.02) weights, 96 prompt tokens."""
    rng = np.random.default_rng(7)
    N, d, L, T = 2000, 5120, 1400, 96
    say("dynamic set, d=5120, L=1400, T=96")
    def draw(*shape, s):
        return _bf16((rng.standard_normal(shape) * s).astype(np.float32))
    wg, wu, wd = draw(N, d, s=0.02), draw(N, d, s=0.02), draw(d, N, s=0.02)
    x = draw(T, d, s=1.0)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd), torch.from_numpy(loaded))
    static = np.sort(rng.permutation(L)[:420]).astype(np.int32)
    alpha, n_total = 560, 560
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, n_total)
    got, counts = host_array(got), host_array(counts)
    # validity against the GPU's own counts
    assert len(got) == n_total and np.all(np.diff(got) > 0) and set(static) <= set(got)
    assert counts.sum() == T * alpha and counts.max() <= T
    dyn = [j for j in got if j not in set(static)]
    rest = [j for j in range(L) if j not in set(got)]
    worst_dyn = min((counts[j], -j) for j in dyn)
    best_rest = max((counts[j], -j) for j in rest)
    assert worst_dyn > best_rest
    # the counts against the oracle's, up to ranking near-ties at alpha
    _, want_counts = oracle.select_dynamic(oracle.activations(x, ref["gate_up_c"]), static,
                                           alpha, n_total)
    diff = np.abs(counts - want_counts)
    say(f"  counts differing: {int((diff > 0).sum())} of {L}, max {int(diff.max())}")
    assert (diff > 0).sum() <= L // 100 and diff.max() <= 2


@pytest.mark.parametrize("wdtype,T,d", [("bf16", 300, 256), ("bf16", 40, 264), ("f32", 50, 96),
                                        ("f16", 300, 256)])
def test_profile_scores(wdtype, T, d):
    N = 700
    say(f"profile scores {wdtype} T={T} d={d}")
    rng = np.random.default_rng(T + d)
    a = lambda *s: (rng.standard_normal(s) * 0.1).astype(np.float32)
    wg, wu, wd, x = a(N, d), a(N, d), a(d, N), (rng.standard_normal((T, d))).astype(np.float32)
    if wdtype == "bf16":
        wg, wu, wd, x = _bf16(wg), _bf16(wu), _bf16(wd), _bf16(x)
    elif wdtype == "f16":
        wg, wu, wd, x = (a.astype(np.float16) for a in (wg, wu, wd, x))
    full = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                          torch.arange(N, dtype=torch.int32))
    ref = oracle.compact(wg, wu, wd, np.arange(N))
    want, Tw = oracle.profile_scores(x, ref["gate_up_c"])
    assert Tw == T
    s1 = si.profile_scores(dev_tensor(x), full.gate_up_c)
    got = host_array(s1).astype(np.float64)
    err = np.linalg.norm(got - want) / np.linalg.norm(want)
    say(f"  rel L2 {err:.2e}")
    assert err <= 1e-5
    assert np.array_equal(host_array(si.profile_scores(dev_tensor(x), full.gate_up_c)),
                          host_array(s1))
    si.profile_scores(dev_tensor(x), full.gate_up_c, scores=s1)     # accumulates
    assert np.linalg.norm(host_array(s1) - 2 * want) / np.linalg.norm(2 * want) <= 1e-5


def test_merge_and_rank():
    rng = np.random.default_rng(3)
    F, N = 3, 5000
    s = (np.abs(rng.standard_normal((F, N))) * 10).astype(np.float32)
    toks = [7, 100, 33]
    got = host_array(si.merge_scores(dev_tensor(s), toks)).astype(np.float64)
    want = oracle.merge_scores([(s[f].astype(np.float64), toks[f]) for f in range(F)])
    assert np.max(np.abs(got - want) / np.maximum(np.abs(want), 1e-30)) <= 1e-6
    # ranking, on the same float32 values on both sides: ties, -0 / +0, NaN, negatives
    r = np.round(rng.standard_normal(N) * 4).astype(np.float32)
    r[:5] = [0.0, -0.0, np.nan, np.inf, -np.inf]
    r[100:110] = np.nan
    order = host_array(si.rank_neurons(dev_tensor(r)))
    assert np.array_equal(order, oracle.rank_neurons(r.astype(np.float64)))
    # one neuron
    assert host_array(si.rank_neurons(dev_tensor(np.array([2.5], np.float32)))).tolist() == [0]


def test_select_errors():
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    gu = torch.zeros((10, 2, 64), dtype=torch.bfloat16, device="cuda")
    st = torch.tensor([1, 2], dtype=torch.int32, device="cuda")
    for alpha, n_total in [(11, 5), (3, 11), (3, 1)]:
        with pytest.raises(si.SelectInferError):
            si.dynamic_set(x, gu, st, alpha, n_total)
    with pytest.raises(si.SelectInferError):
        si.merge_scores(torch.zeros((2, 5), device="cuda"), [1, 0])
