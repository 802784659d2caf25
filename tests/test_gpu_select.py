"""GPU parity of the neuron-selection entry points against the fp64 oracle.

- si_dynamic_set, exact: integer-valued weights and x make every gate and up product exact in
  float32, so the kernel's activations differ from the oracle's float64 ones only through
  SiLU and one product, a few parts in 10^6. Tokens repeat a few prototypes, and the data is
  drawn (seed search, deterministic) so that at every token's alpha boundary each activation
  key either equals the boundary key exactly in float64 (equal gate and up values: duplicated
  rows are planted there, so the lower-slot tie rule decides) or is at least 2e-5 away from it,
  ten times the kernel's error. Result and counts must then be identical to the oracle's, in
  both ranking modes (|a| and a).
- si_dynamic_set, realistic shape (d = 5120, N(0, 0.02) weights): compared with the oracle's
  float64 activations with an explicit near-tie allowance. A token's slot is "ambiguous" when
  its key lies within 1e-4 of the token's boundary key (relative); the GPU's counts must lie
  between the counts of sure picks and sure + ambiguous picks, equal the oracle's where no
  ambiguity is possible, and the GPU's dynamic pick may differ from the oracle's only by swaps
  that those intervals allow.
- si_profile_scores (Eq. 1): relative L2 <= 1e-5 against the fp64 oracle for one call, and
  <= 1e-6 after 1000 accumulating calls against the oracle over the concatenated tokens
  (float64 accumulation); bitwise reproducible.
- si_merge_scores: relative error <= 1e-15 (float64 division by the exact token count);
  si_rank_neurons: exact, on the same float64 scores (ties, -0, NaN).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, say

pytestmark = pytest.mark.gpu

MARGIN = 2e-5      # relative distance from the boundary key that float32 cannot reverse


def _bf16(a):
    a = np.asarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)   # exact for small integers


def _keys(A, mode):
    return np.abs(A) if mode == "abs" else A


def _boundary_clear(A, alpha, mode):
    """Every key of every row equals the row's alpha-th largest key exactly or lies at least
    MARGIN (relative) away from it."""
    for row in _keys(A, mode):
        if not 0 < alpha < len(row):
            continue
        v = np.sort(row)[::-1][alpha - 1]
        scale = max(abs(v), 1e-30)
        near = np.abs(row - v) < MARGIN * scale
        if np.any(near & (row != v)):
            return False
    return True


def _planted_problem(seed, N, d, L, T, wdtype, alpha, mode, n_proto=5):
    """Integer data, tokens drawn from n_proto prototypes, a duplicated row planted at each
    prototype's boundary; None when a boundary is not clear (the caller tries another seed)."""
    rng = np.random.default_rng(seed)
    # |g| <= 8: SiLU(g) / g then differs by at least 6e-4 between integer gates, so equal
    # products of different gates and ups stay far apart in float64 as well
    wg = rng.integers(-1, 2, (N, d)).astype(np.float32)
    wu = rng.integers(-7, 8, (N, d)).astype(np.float32)
    wd = rng.integers(-3, 4, (d, N)).astype(np.float32)
    proto = np.zeros((n_proto, d), np.float32)
    for p in range(n_proto):            # eight nonzero features per prototype, values +-1
        cols = rng.permutation(d)[:8]
        proto[p, cols] = rng.choice([-1.0, 1.0], 8)
    which = rng.integers(0, n_proto, T)
    which[:n_proto] = np.arange(n_proto)
    x = proto[which]
    loaded = rng.permutation(N)[:L].astype(np.int32)
    s2o = np.sort(loaded)
    # plant a tie at each prototype's boundary: the first left-out slot gets the rows of the
    # last taken one (its activation then equals it bitwise, on both sides)
    for p in range(n_proto):
        gu = np.stack([wg[s2o], wu[s2o]], axis=1)
        K = _keys(oracle.activations(proto[p:p + 1], gu)[0], mode)
        order = sorted(range(L), key=lambda j: (-K[j], j))
        j_in, j_out = order[alpha - 1], order[alpha]
        wg[s2o[j_out]] = wg[s2o[j_in]]
        wu[s2o[j_out]] = wu[s2o[j_in]]
    if wdtype == "bf16":
        wg, wu, wd, x = _bf16(wg), _bf16(wu), _bf16(wd), _bf16(x)
    elif wdtype == "f16":
        wg, wu, wd, x = (a.astype(np.float16) for a in (wg, wu, wd, x))
    ref = oracle.compact(wg, wu, wd, loaded)
    A = oracle.activations(x[:n_proto], ref["gate_up_c"])
    if not _boundary_clear(A, alpha, mode):
        return None
    return rng, x, ref, (wg, wu, wd, loaded)


def _find_problem(base, *args, **kw):
    for seed in range(base, base + 40):
        prob = _planted_problem(seed, *args, **kw)
        if prob is not None:
            return prob
    raise AssertionError("no seed with clear alpha boundaries")


def _gpu_layer(full):
    wg, wu, wd, loaded = full
    return si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                          torch.from_numpy(loaded))


@pytest.mark.parametrize("wdtype,T,mode", [("bf16", 37, "abs"), ("bf16", 300, "abs"),
                                           ("bf16", 300, "raw"), ("f32", 23, "abs"),
                                           ("f32", 40, "raw"), ("f16", 300, "abs")])
def test_dynamic_set_exact(wdtype, T, mode):
    N, d, L = 700, 64, 530
    alpha, n_total = 75, 160
    say(f"dynamic set exact {wdtype} T={T} mode={mode}")
    rng, x, ref, full = _find_problem(T * 7 + len(wdtype), N, d, L, T, wdtype, alpha, mode)
    gpu = _gpu_layer(full)
    static = np.sort(rng.permutation(L)[:60]).astype(np.int32)
    A = oracle.activations(x, ref["gate_up_c"])
    want, want_counts = oracle.dynamic_set(x, ref["gate_up_c"], static, alpha, n_total, mode)
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha,
                                 n_total, mode=mode)
    assert np.array_equal(host_array(counts), want_counts)
    assert np.array_equal(host_array(got), want)
    # degenerate cases: no static slots; alpha = 0 (all counts 0: lowest slots fill);
    # n_total = n_static (the static set only); n_total = L (every slot)
    g2, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static[:0]), alpha, 50,
                           mode=mode)
    assert np.array_equal(host_array(g2), oracle.select_dynamic(A, [], alpha, 50, mode)[0])
    g3, c3 = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), 0, n_total,
                            mode=mode)
    assert not host_array(c3).any()
    assert np.array_equal(host_array(g3), oracle.select_dynamic(A, static, 0, n_total, mode)[0])
    g4, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, len(static),
                           mode=mode)
    assert np.array_equal(host_array(g4), static)
    g5, _ = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, L,
                           mode=mode)
    assert np.array_equal(host_array(g5), np.arange(L, dtype=np.int32))


@pytest.mark.parametrize("L", [16384, 32768, 32769])
def test_dynamic_set_row_length_paths(L):
    """Up to 32768 loaded slots the tokens' choices travel as bitmaps and are counted per word;
    past it, as index lists counted with atomics. Both must give the oracle's result."""
    N, d, T = L + 300, 64, 40
    alpha, n_total = 2500, 6000
    say(f"dynamic set L={L}")
    rng, x, ref, full = _find_problem(L, N, d, L, T, "bf16", alpha, "abs")
    gpu = _gpu_layer(full)
    static = rng.permutation(L)[:3000].astype(np.int32)   # unsorted on purpose
    want, want_counts = oracle.dynamic_set(x, ref["gate_up_c"], np.sort(static), alpha, n_total)
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha, n_total)
    assert np.array_equal(host_array(counts), want_counts)
    assert np.array_equal(host_array(got), want)


def _tie_intervals(A, alpha, mode, delta):
    """Per slot: how many tokens surely take it (key above the token's boundary key by more
    than delta, relative, or equal-to-boundary impossible to move) and how many might."""
    K = _keys(A, mode)
    T, L = K.shape
    lo = np.zeros(L, np.int64)
    amb = np.zeros(L, np.int64)
    for row in K:
        v = np.sort(row)[::-1][alpha - 1]
        band = delta * max(abs(v), 1e-30)
        lo += row > v + band
        amb += np.abs(row - v) <= band
    return lo, lo + amb, int(amb.sum())


@pytest.mark.parametrize("mode", ["abs", "raw"])
def test_dynamic_set_realistic_shape(mode):
    """13B-like rows (d = 5120) with random N(0, 0.02) weights, 96 prompt tokens, against the
    float64 oracle with an explicit near-tie allowance."""
    rng = np.random.default_rng(7)
    N, d, L, T = 2000, 5120, 1400, 96
    say(f"dynamic set, d=5120, L=1400, T=96, mode={mode}")
    def draw(*shape, s):
        return _bf16((rng.standard_normal(shape) * s).astype(np.float32))
    wg, wu, wd = draw(N, d, s=0.02), draw(N, d, s=0.02), draw(d, N, s=0.02)
    x = draw(T, d, s=1.0)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd), torch.from_numpy(loaded))
    static = np.sort(rng.permutation(L)[:420]).astype(np.int32)
    alpha, n_total = 560, 700
    got, counts = si.dynamic_set(dev_tensor(x), gpu.gate_up_c, dev_tensor(static), alpha,
                                 n_total, mode=mode)
    got, counts = host_array(got), host_array(counts).astype(np.int64)
    A = oracle.activations(x, ref["gate_up_c"])
    want, want_counts = oracle.select_dynamic(A, static, alpha, n_total, mode)
    lo, hi, n_amb = _tie_intervals(A, alpha, mode, 1e-4)
    say(f"  ambiguous (token, slot) pairs: {n_amb}; counts differing from the oracle: "
        f"{int((counts != want_counts).sum())}")
    assert n_amb <= T * 4
    assert np.all(lo <= want_counts) and np.all(want_counts <= hi)      # the allowance holds
    assert np.all(lo <= counts) and np.all(counts <= hi)
    assert np.array_equal(counts[lo == hi], want_counts[lo == hi])
    assert counts.sum() == T * alpha
    # the set: size, order, static slots, and a dynamic pick that equals the oracle's up to
    # swaps the count intervals allow
    assert len(got) == n_total and np.all(np.diff(got) > 0) and set(static) <= set(got)
    only_gpu = sorted(set(got) - set(want))
    only_ref = sorted(set(want) - set(got))
    say(f"  dynamic slots differing: {len(only_gpu)}")
    assert len(only_gpu) == len(only_ref) <= 10
    for j in only_gpu:
        for i in only_ref:
            assert (hi[j], -j) > (lo[i], -i), (j, i)
    # and the GPU's pick is the top of its own counts (ties to the lower slot)
    st = set(static.tolist())
    dyn = [j for j in got if j not in st]
    rest = [j for j in range(L) if j not in set(got.tolist())]
    assert min((counts[j], -j) for j in dyn) > max((counts[j], -j) for j in rest)


def _score_problem(wdtype, N, d, T, seed):
    rng = np.random.default_rng(seed)
    a = lambda *s: (rng.standard_normal(s) * 0.1).astype(np.float32)
    wg, wu, wd = a(N, d), a(N, d), a(d, N)
    x = rng.standard_normal((T, d)).astype(np.float32)
    if wdtype == "bf16":
        wg, wu, wd, x = _bf16(wg), _bf16(wu), _bf16(wd), _bf16(x)
    elif wdtype == "f16":
        wg, wu, wd, x = (v.astype(np.float16) for v in (wg, wu, wd, x))
    full = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                          torch.arange(N, dtype=torch.int32))
    ref = oracle.compact(wg, wu, wd, np.arange(N))
    return x, full, ref


@pytest.mark.parametrize("wdtype,T,d", [("bf16", 300, 256), ("bf16", 40, 264), ("f32", 50, 96),
                                        ("f16", 300, 256)])
def test_profile_scores(wdtype, T, d):
    N = 700
    say(f"profile scores {wdtype} T={T} d={d}")
    x, full, ref = _score_problem(wdtype, N, d, T, T + d)
    want, Tw = oracle.profile_scores(x, ref["gate_up_c"])
    assert Tw == T
    s1 = si.profile_scores(dev_tensor(x), full.gate_up_c)
    assert s1.dtype == torch.float64
    got = host_array(s1)
    err = np.linalg.norm(got - want) / np.linalg.norm(want)
    say(f"  rel L2 {err:.2e}")
    assert err <= 1e-5
    assert np.array_equal(host_array(si.profile_scores(dev_tensor(x), full.gate_up_c)), got)
    si.profile_scores(dev_tensor(x), full.gate_up_c, scores=s1)     # accumulates
    assert np.linalg.norm(host_array(s1) - 2 * want) / np.linalg.norm(2 * want) <= 1e-5


@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_profile_scores_accumulate_1000_calls(wdtype):
    """A profile built from 1000 calls of 8 tokens: the float64 sums stay at the precision of
    the activations (a float32 accumulator drifts here), against the oracle's Eq. 1 over all
    8000 tokens at once. The merged and ranked result is then the oracle's."""
    N, d, T, calls = 256, 128, 8, 1000
    say(f"profile scores, {calls} accumulating calls of {T} tokens, {wdtype}")
    x, full, ref = _score_problem(wdtype, N, d, T * calls, 31)
    xd = dev_tensor(x)
    s = torch.zeros(N, dtype=torch.float64, device="cuda")
    for c in range(calls):
        si.profile_scores(xd[c * T:(c + 1) * T], full.gate_up_c, scores=s)
    torch.cuda.synchronize()
    want, Tw = oracle.profile_scores(x, ref["gate_up_c"])
    got = host_array(s)
    err = np.linalg.norm(got - want) / np.linalg.norm(want)
    say(f"  rel L2 after {calls} calls: {err:.2e}")
    assert Tw == T * calls and err <= 1e-6
    # two score files with their exact token counts, merged and ranked on the device
    half = T * calls // 2
    files = torch.stack([s, s.clone()])
    merged = si.merge_scores(files, [Tw, half])
    want_m = oracle.merge_scores([(got, Tw), (got, half)])
    assert np.max(np.abs(host_array(merged) - want_m) / want_m) <= 1e-15
    order = host_array(si.rank_neurons(merged))
    assert np.array_equal(order, oracle.rank_neurons(host_array(merged)))


def test_merge_and_rank():
    rng = np.random.default_rng(3)
    F, N = 3, 5000
    s = np.abs(rng.standard_normal((F, N))) * 10
    toks = [7, 100, (1 << 40) + 3]          # counts far above 2^24 stay exact
    got = host_array(si.merge_scores(dev_tensor(s), toks))
    want = oracle.merge_scores([(s[f], toks[f]) for f in range(F)])
    assert np.max(np.abs(got - want) / np.maximum(np.abs(want), 1e-300)) <= 1e-15
    # ranking, on the same float64 values on both sides: ties, -0 / +0, NaN, negatives, and
    # values float32 cannot tell apart
    r = np.round(rng.standard_normal(N) * 4)
    r[:5] = [0.0, -0.0, np.nan, np.inf, -np.inf]
    r[100:110] = np.nan
    r[200:204] = [1.0 + 2.0 ** -40, 1.0, 1.0 + 2.0 ** -41, 1.0]
    order = host_array(si.rank_neurons(dev_tensor(r)))
    assert np.array_equal(order, oracle.rank_neurons(r))
    # one neuron
    assert host_array(si.rank_neurons(dev_tensor(np.array([2.5])))).tolist() == [0]


def test_select_errors():
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    gu = torch.zeros((10, 2, 64), dtype=torch.bfloat16, device="cuda")
    st = torch.tensor([1, 2], dtype=torch.int32, device="cuda")
    for alpha, n_total in [(11, 5), (3, 11), (3, 1)]:
        with pytest.raises(si.SelectInferError):
            si.dynamic_set(x, gu, st, alpha, n_total)
    with pytest.raises(si.SelectInferError):
        si.merge_scores(torch.zeros((2, 5), dtype=torch.float64, device="cuda"), [1, 0])
    with pytest.raises(ValueError):
        si.merge_scores(torch.zeros((2, 5), dtype=torch.float32, device="cuda"), [1, 1])
