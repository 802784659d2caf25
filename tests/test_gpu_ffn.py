"""GPU parity of si_selective_ffn against the fp64 oracle, per token.

Tolerance (per token, relative L2, max over tokens): 1e-5 for f32 weights, 5e-3 for bf16
weights. The paths are held tighter where their arithmetic allows: the per-token path only
reassociates float32 sums, and below 128 tokens the union path feeds h to its MFMA GEMM as a
16-bit hi + lo pair (about 16 significant bits), so both are held to 1e-4 per token and to an
element-wise bound, max |y - y_ref| <= 1e-4 * max |y_ref| per token. From 128 tokens the tiled
union path feeds h as one 16-bit value by default (8 significant bits for bf16: a relative
rounding error of at most 2^-8 per h, about 1.5e-3 in rms), as does SI_FLAG_FAST_H at any
batch; these are held to the 5e-3 bar and to max |y - y_ref| <= 5e-3 * max |y_ref|, and
SI_FLAG_EXACT_H (the pair on the tiled path) to 1e-4.

With IEEE-half data the pair has a floor as well: once |h| < 2^-3 its low half is subnormal,
so h is carried to max(2^-22 |h|, 2^-25) absolutely rather than to 16 significant bits; the
cases here keep |h| where the 1e-4 bar measures the arithmetic rather than that floor (a token
whose every h is below 1e-3 can sit near 1e-4 on its own).
"""
import functools
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, max_rel_l2, rel_l2, say
from workloads import CONFIGS, active_sets, csr_from_sets, layer_weights, loaded_ids, tokens_x

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 5e-3}
ALARM_PER_TOKEN = 1e-4
ELEM = 1e-4
ELEM_ONE_H = 5e-3   # element-wise bound when h enters the second GEMM as one 16-bit value


def max_elem_err(got2d, ref2d) -> float:
    """max over tokens of max |got - ref| / max |ref| (0 / 0 counts as 0)."""
    worst = 0.0
    for g, r in zip(np.asarray(got2d, np.float64), np.asarray(ref2d, np.float64)):
        m = np.max(np.abs(r)) if r.size else 0.0
        e = np.max(np.abs(g - r)) if r.size else 0.0
        worst = max(worst, e / m if m > 0 else (0.0 if e == 0 else np.inf))
    return worst


@functools.lru_cache(maxsize=2)
def _layer(name, layer=0):
    cfg = CONFIGS[name]
    wg, wu, wd = layer_weights(cfg, layer)
    loaded = loaded_ids(cfg, layer)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                         torch.from_numpy(loaded))
    return cfg, ref, gpu


def _slots(ref, sets):
    return [oracle.remap(ref["orig_to_slot"], s) for s in sets]


def _run(x, slot_sets, gpu, flags=0):
    off, idx = csr_from_sets(slot_sets)
    y = si.selective_ffn(dev_tensor(x), dev_tensor(off), dev_tensor(idx), gpu.gate_up_c,
                         gpu.down_c, flags=flags)
    return host_array(y)


def _oracle(x, slot_sets, ref):
    return np.stack([oracle.selective_ffn(x[t], slot_sets[t], ref["gate_up_c"], ref["down_c"])
                     for t in range(len(slot_sets))])


def test_tiny_f32_all_tokens():
    cfg, ref, gpu = _layer("tiny_f32")
    say("tiny f32: 64 tokens, one call per token and one batched call")
    toks = range(cfg.steps)
    x = tokens_x(cfg, toks)
    slots = _slots(ref, active_sets(cfg, toks))
    want = _oracle(x, slots, ref)
    per_call = np.stack([_run(x[t:t + 1], [slots[t]], gpu)[0] for t in toks])
    assert max_rel_l2(per_call, want) <= TOL["f32"]
    batched = _run(x, slots, gpu)
    assert max_rel_l2(batched, want) <= TOL["f32"]


def test_llama2_7b_decode_sampled_tokens():
    cfg, ref, gpu = _layer("llama2_7b_decode")
    toks = [0, 1, 2, 3, 511, 1023]
    say(f"7B decode: tokens {toks}, B=1 calls as in the benchmark")
    x = tokens_x(cfg, toks)
    slots = _slots(ref, active_sets(cfg, toks))
    want = _oracle(x, slots, ref)
    got = np.stack([_run(x[i:i + 1], [slots[i]], gpu)[0] for i in range(len(toks))])
    err = max_rel_l2(got, want)
    say(f"7B decode max rel L2 {err:.3e}")
    assert err <= TOL["bf16"] and err <= ALARM_PER_TOKEN
    # bitwise reproducible
    again = np.stack([_run(x[i:i + 1], [slots[i]], gpu)[0] for i in range(len(toks))])
    assert np.array_equal(got, again)
    # order of the index list does not matter beyond float32 reassociation
    rev = np.stack([_run(x[i:i + 1], [slots[i][::-1].copy()], gpu)[0] for i in range(len(toks))])
    assert max_rel_l2(rev, got) <= 1e-6


def _rand_problem(seed, N, d, L, wdtype, wscale=0.02):
    rng = np.random.default_rng(seed)
    def draw(*shape, scale=wscale):
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
        if wdtype == "f16":
            return a.astype(np.float16)
        return (a.view(np.uint32) >> 16).astype(np.uint16) if wdtype == "bf16" else a
    wg, wu, wd = draw(N, d), draw(N, d), draw(d, N)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                         torch.from_numpy(loaded))
    return rng, draw, ref, gpu


@pytest.mark.parametrize("d,wdtype", [(8, "bf16"), (264, "bf16"), (1000, "bf16"),
                                      (4104, "bf16"), (5120, "bf16"), (12296, "bf16"),
                                      (16384, "bf16"), (12, "f32"), (1000, "f32"),
                                      (2052, "f32"), (6148, "f32"), (8192, "f32")])
def test_per_token_ragged_shapes(d, wdtype):
    """Each lane owns up to four 16-byte column groups of a row: d = 4104 / 2052 takes two,
    12296 / 6148 three and four with a ragged last group, 16384 / 8192 the largest d the
    per-token path supports (four full groups)."""
    N, L = 700, 530
    say(f"per-token ragged d={d} {wdtype}")
    rng, draw, ref, gpu = _rand_problem(d, N, d, L, wdtype)
    ks = [0, 1, 2, 7, 8, 9, 17, 130, 529, 530]
    sets = [rng.permutation(L)[:k].astype(np.int32) for k in ks]
    x = draw(len(ks), d, scale=1.0)
    want = _oracle(x, sets, ref)
    got = np.stack([_run(x[i:i + 1], [sets[i]], gpu)[0] for i in range(len(ks))])
    assert not np.any(got[0])                       # empty set -> exact zeros
    err = max_rel_l2(got, want)
    assert err <= TOL[wdtype] and (wdtype == "f32" or err <= ALARM_PER_TOKEN)
    got_b = _run(x, sets, gpu, flags=si.FLAG_PER_TOKEN)
    assert max_rel_l2(got_b, want) <= TOL[wdtype]


@pytest.mark.parametrize("B,d,L", [(2, 264, 613), (5, 1000, 613), (17, 264, 613),
                                   (32, 264, 613), (33, 512, 613), (64, 264, 613),
                                   (70, 1000, 613), (3, 72, 16500)])
def test_union_path_ragged(B, d, L):
    """Row-word GEMM path (SI_FLAG_UNION below 5 tokens); L = 16500 gives over 512 bitmap
    words, where a work-group takes both 16-row tiles of a word, and the smaller ones one tile
    each. Without the flag, 2 and 3 tokens take the per-token path, to the same result."""
    N = L + 287
    say(f"union ragged B={B} d={d} L={L}")
    rng, draw, ref, gpu = _rand_problem(B * 1000 + d, N, d, L, "bf16")
    sets = []
    for b in range(B):
        k = int(rng.integers(0, L + 1)) if b % 4 else (0 if b == 4 else int(rng.integers(1, 60)))
        sets.append(rng.permutation(L)[:k].astype(np.int32))
    x = draw(B, d, scale=1.0)
    want = _oracle(x, sets, ref)
    got = _run(x, sets, gpu, flags=si.FLAG_UNION)
    for b in range(B):
        if len(sets[b]) == 0:
            assert not np.any(got[b])
    assert max_rel_l2(got, want) <= TOL["bf16"]
    fast = _run(x, sets, gpu, flags=si.FLAG_FAST_H | si.FLAG_UNION)
    assert max_rel_l2(fast, want) <= TOL["bf16"]
    default = _run(x, sets, gpu)
    assert max_rel_l2(default, want) <= (ALARM_PER_TOKEN if B < 5 else TOL["bf16"])


@pytest.mark.parametrize("B,d,L,sparse", [(128, 264, 613, False), (257, 1000, 300, False),
                                           (300, 264, 613, True), (130, 64, 81, False),
                                           (300, 4088, 1000, False), (140, 5112, 1000, True),
                                           (160, 2048, 2100, False), (130, 6144, 700, False)])
def test_union_tiled_ragged(B, d, L, sparse):
    """Batches of 128 tokens and more take the LDS-tiled GEMMs: ragged token, slot and K tiles,
    a union much smaller than L (sparse), split-K tails, empty sets. The last four shapes run
    GEMM2 on its XCD grid (combo counts 8, 8, 16, 8) with 128-, 160-, 128- and 192-column
    tiles, the first two with a ragged last column tile."""
    N = L + 97
    say(f"union tiled B={B} d={d} L={L} sparse={sparse}")
    rng, draw, ref, gpu = _rand_problem(B * 7 + d + L, N, d, L, "bf16")
    pool = rng.permutation(L)[:max(1, L // 5)] if sparse else np.arange(L)
    sets = []
    for b in range(B):
        if b % 9 == 4:
            k = 0
        else:
            k = int(rng.integers(1, len(pool) + 1))
        sets.append(np.sort(rng.permutation(pool)[:k]).astype(np.int32))
    x = draw(B, d, scale=1.0)
    want = _oracle(x, sets, ref)
    got = _run(x, sets, gpu)
    for b in range(B):
        if len(sets[b]) == 0:
            assert not np.any(got[b])
    err = max_rel_l2(got, want)
    say(f"  default (h as one bf16 value) max rel L2 {err:.3e}")
    assert err <= TOL["bf16"] and max_elem_err(got, want) <= ELEM_ONE_H
    exact = _run(x, sets, gpu, flags=si.FLAG_EXACT_H)
    erre = max_rel_l2(exact, want)
    say(f"  SI_FLAG_EXACT_H (hi + lo) max rel L2 {erre:.3e}")
    assert erre <= 1e-4 and max_elem_err(exact, want) <= ELEM  # hi + lo pair: ~16 bits
    for b in range(B):
        if len(sets[b]) == 0:
            assert not np.any(exact[b])
    # SI_FLAG_FAST_H names the default here; with EXACT_H as well, FAST_H wins
    assert np.array_equal(_run(x, sets, gpu, flags=si.FLAG_FAST_H), got)
    assert np.array_equal(_run(x, sets, gpu, flags=si.FLAG_FAST_H | si.FLAG_EXACT_H), got)
    again = _run(x, sets, gpu)
    assert np.array_equal(got, again)   # fixed-order reductions: bitwise reproducible
    assert np.array_equal(_run(x, sets, gpu, flags=si.FLAG_EXACT_H), exact)


@pytest.mark.parametrize("d", [64, 128, 192, 256, 320, 384, 448])
def test_union_tiled_k_step_counts(d):
    """The 256-token GEMM1 keeps three K tiles in flight in rotating register sets and runs the
    one or two steps left over after its loop; GEMM2 keeps two or three. d = 64 .. 448 gives 1
    to 7 K steps in GEMM1, and union sizes around multiples of 64 give GEMM2 chunks of every
    remainder; each against the oracle and against the pair form of h."""
    B, L = 200, 700
    N = L + 50
    say(f"tiled K steps d={d}")
    rng, draw, ref, gpu = _rand_problem(9000 + d, N, d, L, "bf16", wscale=d ** -0.5)
    for nU in (64, 130, 191, 257, L):
        pool = rng.permutation(L)[:nU]
        sets = [np.sort(rng.permutation(pool)[:int(rng.integers(1, nU + 1))]).astype(np.int32)
                for _ in range(B)]
        sets[0] = np.sort(pool).astype(np.int32)          # the union is the whole pool
        x = draw(B, d, scale=1.0)
        want = _oracle(x, sets, ref)
        got = _run(x, sets, gpu)
        err = max_rel_l2(got, want)
        assert err <= TOL["bf16"] and max_elem_err(got, want) <= ELEM_ONE_H, (nU, err)
        exact = _run(x, sets, gpu, flags=si.FLAG_EXACT_H)
        assert max_rel_l2(exact, want) <= ALARM_PER_TOKEN, nU


@pytest.mark.parametrize("seed", range(24))
def test_random_shapes(seed):
    """Seeded random problems across the path boundaries: B from 1 to 300 (per-token below 5
    tokens, row-word union from 5, tiled union from 128 for 16-bit weights), d a multiple of 8
    from 8 to 3000, L from 1 to 1500, per-token sets of any size including empty ones, bf16 /
    f16 / f32 weights scaled by 1 / sqrt(d), so that gate and up products are of order one at
    every d, as in a trained layer. Each is held to its path's bar (one 16-bit h on the tiled
    path: 5e-3; otherwise 1e-4, and 1e-5 for f32 weights) and checked against the per-token
    path."""
    rng = np.random.default_rng(1000 + seed)
    wdtype = ["bf16", "f16", "f32"][seed % 3]
    B = int(rng.choice([1, 2, 3, 4, 5, 7, 16, 33, 64, 127, 128, 200, 300]))
    d = 8 * int(rng.integers(1, 376))
    L = int(rng.integers(1, 1501))
    N = L + int(rng.integers(0, 300))
    say(f"random shape seed={seed}: B={B} d={d} L={L} N={N} {wdtype}")
    _, draw, ref, gpu = _rand_problem(5000 + seed, N, d, L, wdtype, wscale=d ** -0.5)
    budget = max(1, 40000 // B)             # about 40k oracle rows per case in all
    sets = []
    for b in range(B):
        k = int(rng.integers(0, min(L, budget) + 1)) if b % 6 != 1 else 0
        sets.append(rng.permutation(L)[:k].astype(np.int32))
    x = draw(B, d, scale=1.0)
    want = _oracle(x, sets, ref)
    got = _run(x, sets, gpu)
    tiled = B >= 128 and wdtype != "f32"
    tol = TOL["f32"] if wdtype == "f32" else (TOL["bf16"] if tiled else ALARM_PER_TOKEN)
    err, elem = max_rel_l2(got, want), max_elem_err(got, want)
    say(f"  max rel L2 {err:.3e}, element-wise {elem:.3e} (bar {tol})")
    assert err <= tol and elem <= (ELEM_ONE_H if tiled else ELEM)
    for b in range(B):
        if len(sets[b]) == 0:
            assert not np.any(got[b])
    if B > 1:
        per = _run(x, sets, gpu, flags=si.FLAG_PER_TOKEN)
        assert max_rel_l2(per, want) <= (TOL["f32"] if wdtype == "f32" else ALARM_PER_TOKEN)


@pytest.mark.parametrize("B,d,xdt", [(1, 264, "f16"), (1, 4104, "f16"), (3, 1000, "f32"),
                                      (17, 264, "f16"), (70, 1000, "f16"), (130, 264, "f16")])
def test_fp16_weights(B, d, xdt):
    """IEEE-half weights (the paper's storage precision): per-token path with half or float32
    x, union paths (row-word below 128 tokens, tiled from 128) with half x."""
    N, L = 900, 613
    say(f"fp16 weights B={B} d={d} x={xdt}")
    rng, draw, ref, gpu = _rand_problem(B * 31 + d, N, d, L, "f16")
    sets = [rng.permutation(L)[:int(rng.integers(0, L + 1)) if b % 5 else 40].astype(np.int32)
            for b in range(B)]
    x = draw(B, d, scale=1.0)
    if xdt == "f32":
        x = x.astype(np.float32)
    want = _oracle(x, sets, ref)
    got = _run(x, sets, gpu)
    err = max_rel_l2(got, want)
    say(f"  rel L2 {err:.2e}")
    if B >= 128:
        # tiled: h as one half value by default (11 significant bits), the pair on request
        assert err <= TOL["bf16"]
        exact = _run(x, sets, gpu, flags=si.FLAG_EXACT_H)
        assert max_rel_l2(exact, want) <= ALARM_PER_TOKEN
    else:
        assert err <= ALARM_PER_TOKEN   # float32 sums; union: h as a half hi + lo pair
    if B > 1 and xdt == "f16":
        fast = _run(x, sets, gpu, flags=si.FLAG_FAST_H)
        assert max_rel_l2(fast, want) <= TOL["bf16"]
        per = _run(x, sets, gpu, flags=si.FLAG_PER_TOKEN)
        assert max_rel_l2(per, want) <= ALARM_PER_TOKEN


@pytest.mark.parametrize("B,d", [(1, 4096), (1, 5120), (3, 1000), (1, 12296), (2, 16384)])
def test_bf16_weights_f32_x(B, d):
    """bf16 weights with float32 x (the per-token path takes the pair at every batch size)."""
    N, L = 700, 530
    say(f"bf16 weights, f32 x: B={B} d={d}")
    rng, draw, ref, gpu = _rand_problem(B * 13 + d, N, d, L, "bf16")
    ks = [300, 0, 17][:B]
    sets = [rng.permutation(L)[:k].astype(np.int32) for k in ks]
    x = rng.standard_normal((B, d)).astype(np.float32)
    want = _oracle(x, sets, ref)
    got = _run(x, sets, gpu)
    assert max_rel_l2(got, want) <= ALARM_PER_TOKEN and max_elem_err(got, want) <= ELEM
    if B > 1:
        assert not np.any(got[1])


def test_invalid_slots_add_nothing():
    """Without SI_FLAG_CHECK an invalid slot id (negative or >= L) in a set is skipped: the result
    is the FFN over the valid slots, on the per-token and the union path."""
    N, d, L = 500, 256, 300
    rng, draw, ref, gpu = _rand_problem(77, N, d, L, "bf16")
    x = draw(3, d, scale=1.0)
    valid = [rng.permutation(L)[:k].astype(np.int32) for k in (9, 20, 5)]
    bad = [np.concatenate([v[:3], [L + 5, -1], v[3:]]).astype(np.int32) for v in valid]
    want = _oracle(x, valid, ref)
    one = np.stack([_run(x[b:b + 1], [bad[b]], gpu)[0] for b in range(3)])
    assert max_rel_l2(one, want) <= ALARM_PER_TOKEN
    assert max_rel_l2(_run(x, bad, gpu), want) <= TOL["bf16"]


def test_llama2_7b_batch16_union():
    cfg, ref, gpu = _layer("llama2_7b_b16")
    say("7B batch-16 union path: 2 steps of 16 tokens")
    for step in range(2):
        toks = range(step * 16, step * 16 + 16)
        x = tokens_x(cfg, toks)
        slots = _slots(ref, active_sets(cfg, toks))
        want = _oracle(x, slots, ref)
        got = _run(x, slots, gpu)
        err, elem = max_rel_l2(got, want), max_elem_err(got, want)
        say(f"union step {step} max rel L2 {err:.3e}, element-wise {elem:.3e}")
        assert err <= ALARM_PER_TOKEN and elem <= ELEM
        per_tok = _run(x, slots, gpu, flags=si.FLAG_PER_TOKEN)
        assert max_rel_l2(per_tok, want) <= ALARM_PER_TOKEN
        assert max_elem_err(per_tok, want) <= ELEM
        fast = _run(x, slots, gpu, flags=si.FLAG_FAST_H)
        errf = max_rel_l2(fast, want)
        say(f"union step {step} fast-h max rel L2 {errf:.3e}")
        assert errf <= TOL["bf16"]


def test_llama2_13b_prefill_union_all_tokens():
    """All 512 tokens of the union call against the per-token path, and 64 of them (every
    eighth) against the oracle directly, which also pins the per-token path at this shape.
    The default call (h as one bf16 value) is held to the 5e-3 bar; SI_FLAG_EXACT_H (hi + lo)
    to 1e-4."""
    cfg, ref, gpu = _layer("llama2_13b_prefill")
    say("13B prefill: 512 tokens in one union call; all against the per-token path, 64 "
        "against the oracle")
    toks = range(cfg.B)
    x = tokens_x(cfg, toks)
    slots = _slots(ref, active_sets(cfg, toks))
    got = _run(x, slots, gpu)
    exact = _run(x, slots, gpu, flags=si.FLAG_EXACT_H)
    per_tok = _run(x, slots, gpu, flags=si.FLAG_PER_TOKEN)
    sample = list(range(0, cfg.B, 8))
    want = _oracle(x[sample], [slots[t] for t in sample], ref)
    e_per = max_rel_l2(per_tok[sample], want)
    assert e_per <= ALARM_PER_TOKEN and max_elem_err(per_tok[sample], want) <= ELEM
    err, elem = max_rel_l2(got[sample], want), max_elem_err(got[sample], want)
    erx, elx = max_rel_l2(exact[sample], want), max_elem_err(exact[sample], want)
    say(f"13B prefill vs oracle ({len(sample)} tokens): union default {err:.3e} (element-wise "
        f"{elem:.3e}), EXACT_H {erx:.3e} ({elx:.3e}), per-token {e_per:.3e}")
    assert err <= TOL["bf16"] and elem <= ELEM_ONE_H
    assert erx <= ALARM_PER_TOKEN and elx <= ELEM
    err_all, elem_all = max_rel_l2(got, per_tok), max_elem_err(got, per_tok)
    erx_all, elx_all = max_rel_l2(exact, per_tok), max_elem_err(exact, per_tok)
    say(f"13B prefill vs per-token (512 tokens): default {err_all:.3e} (element-wise "
        f"{elem_all:.3e}), EXACT_H {erx_all:.3e} ({elx_all:.3e})")
    assert err_all <= TOL["bf16"] and elem_all <= ELEM_ONE_H
    assert erx_all <= ALARM_PER_TOKEN and elx_all <= ELEM


def test_llama3_8b_stack_teacher_forced():
    name = "llama3_8b_stack"
    cfg = CONFIGS[name]
    toks = [0, 1]
    say(f"8B stack: 2 layers teacher-forced, tokens {toks}")
    x = tokens_x(cfg, toks)
    for layer in range(2):
        c, ref, gpu = _layer(name, layer)
        slots = _slots(ref, active_sets(cfg, toks, layer))
        y = _run(x, slots, gpu, flags=si.FLAG_PER_TOKEN)
        want = _oracle(x, slots, ref)
        assert max_rel_l2(y, want) <= ALARM_PER_TOKEN
        xn = host_array(si.residual_rmsnorm(dev_tensor(x), dev_tensor(y.astype(np.float32))))
        for t in range(len(toks)):
            ref_next = oracle.residual_rmsnorm_bf16(x[t], want[t])
            assert rel_l2(oracle.decode(xn[t]), oracle.decode(ref_next)) <= TOL["bf16"]
        x = xn                                      # the oracle's next layer takes the GPU's x


def _resnorm_ref(xp, yp, xdtype):
    """The oracle's next-layer input: bf16 bits, or the exact float64 value for f32."""
    if xdtype == "bf16":
        return oracle.decode(oracle.residual_rmsnorm_bf16(xp, yp))
    r = np.asarray(xp, np.float64) + np.asarray(yp, np.float64)
    return r / math.sqrt(np.mean(r * r) + 1e-5)


def _check_resnorm(xp, yp, sets, ref, gpu, xdtype, wdtype, flags=0):
    """si_selective_ffn_resnorm against the oracle (x_out, then y teacher-forced on the GPU's
    x_out) and against the unfused pair si_residual_rmsnorm + si_selective_ffn."""
    off, idx = csr_from_sets(sets)
    xo, y = si.selective_ffn_resnorm(dev_tensor(xp), dev_tensor(yp), dev_tensor(off),
                                     dev_tensor(idx), gpu.gate_up_c, gpu.down_c, flags=flags)
    xo_h, y_h = host_array(xo), host_array(y)
    x_got = oracle.decode(xo_h) if xdtype == "bf16" else xo_h.astype(np.float64)
    for b in range(len(sets)):
        assert rel_l2(x_got[b], _resnorm_ref(xp[b], yp[b], xdtype)) <= (
            5e-3 if xdtype == "bf16" else 1e-6)
    # the pair of calls it replaces (equal up to the summation order of the mean square: a
    # bf16 x_out may differ by one unit where r / rms falls next to a rounding boundary)
    x_pair = host_array(si.residual_rmsnorm(dev_tensor(xp), dev_tensor(yp)))
    if xdtype == "bf16":
        assert np.mean(xo_h == x_pair) > 0.99
    else:
        assert max_rel_l2(xo_h, x_pair) <= 1e-6
    want = _oracle(xo_h, sets, ref)
    tol = ALARM_PER_TOKEN if wdtype == "bf16" else TOL["f32"]
    assert max_rel_l2(y_h, want) <= tol
    for b in range(len(sets)):
        if len(sets[b]) == 0:
            assert not np.any(y_h[b])
    return xo_h, y_h


def test_llama3_8b_stack_resnorm_fused():
    """Layer 1 of the 8B stack through the fused call, fed by layer 0's GPU output."""
    name = "llama3_8b_stack"
    cfg = CONFIGS[name]
    toks = [3]
    say(f"8B stack: fused residual RMSNorm into layer 1, token {toks}")
    x0 = tokens_x(cfg, toks)
    c, ref0, gpu0 = _layer(name, 0)
    y0 = _run(x0, _slots(ref0, active_sets(cfg, toks, 0)), gpu0)
    c, ref1, gpu1 = _layer(name, 1)
    _check_resnorm(x0, y0.astype(np.float32), _slots(ref1, active_sets(cfg, toks, 1)), ref1,
                   gpu1, "bf16", "bf16")


def test_llama3_8b_table1_dense_to_selective():
    """Table 1's layer range on the 8B stack: layer 4, the last whole layer (all 14336 neurons
    loaded and active), then layer 5, the first selective one, through the fused residual
    RMSNorm call; both teacher-forced against the oracle."""
    name = "llama3_8b_stack_table1"
    cfg = CONFIGS[name]
    assert not si.selective_layers(cfg.layers)[4] and si.selective_layers(cfg.layers)[5]
    toks = [5, 6]
    say(f"8B stack, Table 1 range: whole layer 4 into selective layer 5, tokens {toks}")
    x4 = tokens_x(cfg, toks)
    c, ref4, gpu4 = _layer(name, 4)
    sets4 = _slots(ref4, active_sets(cfg, toks, 4))
    assert all(len(s) == cfg.N for s in sets4)
    y4 = _run(x4, sets4, gpu4)
    want4 = _oracle(x4, sets4, ref4)
    assert max_rel_l2(y4, want4) <= ALARM_PER_TOKEN and max_elem_err(y4, want4) <= ELEM
    c, ref5, gpu5 = _layer(name, 5)
    sets5 = _slots(ref5, active_sets(cfg, toks, 5))
    assert all(len(s) == cfg.k for s in sets5)
    _check_resnorm(x4, y4.astype(np.float32), sets5, ref5, gpu5, "bf16", "bf16")


@pytest.mark.parametrize("B,d,wdtype,xdtype", [(1, 4104, "bf16", "bf16"), (2, 1000, "bf16", "bf16"),
                                               (3, 264, "f32", "f32"), (1, 8, "bf16", "bf16"),
                                               (2, 2052, "f32", "f32"), (2, 1000, "f32", "bf16"),
                                               (4, 512, "bf16", "bf16"), (1, 5120, "bf16", "bf16"),
                                               (2, 5120, "bf16", "f32"), (1, 8200, "bf16", "f32"),
                                               (1, 12296, "bf16", "bf16"),
                                               (1, 16384, "bf16", "bf16")])
def test_selective_ffn_resnorm(B, d, wdtype, xdtype):
    """Per-token path with the prologue (B < 5; f32 weights at any B; SI_FLAG_PER_TOKEN), a
    token with an empty set (its x_out is still written), ragged d, and the union path (bf16
    with SI_FLAG_UNION), which runs the two steps as separate kernels."""
    N, L = 700, 530
    say(f"resnorm B={B} d={d} w={wdtype} x={xdtype}")
    rng, draw, ref, gpu = _rand_problem(100 + d + B, N, d, L, wdtype)
    xp = rng.standard_normal((B, d)).astype(np.float32)
    if xdtype == "bf16":
        xp = (xp.view(np.uint32) >> 16).astype(np.uint16)
    yp = (rng.standard_normal((B, d)) * 0.3).astype(np.float32)
    ks = [0, 1, 130, 529, 17, 8][:B] if B > 1 else [130]
    sets = [rng.permutation(L)[:k].astype(np.int32) for k in ks]
    _check_resnorm(xp, yp, sets, ref, gpu, xdtype, wdtype)
    if B > 1 and wdtype == "bf16":
        _check_resnorm(xp, yp, sets, ref, gpu, xdtype, wdtype, flags=si.FLAG_PER_TOKEN)
        _check_resnorm(xp, yp, sets, ref, gpu, xdtype, wdtype, flags=si.FLAG_UNION)


def test_selective_ffn_resnorm_errors():
    rng, draw, ref, gpu = _rand_problem(7, 300, 64, 200, "bf16")
    xp = dev_tensor(draw(2, 64, scale=1.0))
    yp = torch.zeros((2, 64), dtype=torch.float32, device="cuda:0")
    off, idx = csr_from_sets([np.array([1, 2], np.int32), np.array([3], np.int32)])
    off, idx = dev_tensor(off), dev_tensor(idx)
    with pytest.raises(si.SelectInferError) as e:       # x_out aliases x_prev
        si.selective_ffn_resnorm(xp, yp, off, idx, gpu.gate_up_c, gpu.down_c, x_out=xp)
    assert e.value.status == 1
    with pytest.raises(si.SelectInferError) as e:       # negative eps
        si.selective_ffn_resnorm(xp, yp, off, idx, gpu.gate_up_c, gpu.down_c, eps=-1.0)
    assert e.value.status == 1
    xh = xp.view(torch.int16).to(torch.float16)         # half x: not a stack type here
    with pytest.raises(si.SelectInferError) as e:
        si.selective_ffn_resnorm(xh, yp, off, idx, gpu.gate_up_c, gpu.down_c)
    assert e.value.status == 5


def test_largest_d_and_refusal():
    """d past the supported width is refused before anything is enqueued."""
    say("d limits: 16392 (bf16) and 8196 (f32) are refused")
    for d, dt in ((16392, torch.bfloat16), (8196, torch.float32)):
        x = torch.zeros((1, d), dtype=dt, device="cuda:0")
        gu = torch.zeros((2, 2, d), dtype=dt, device="cuda:0")
        dn = torch.zeros((2, d), dtype=dt, device="cuda:0")
        off = torch.tensor([0, 1], dtype=torch.int32, device="cuda:0")
        idx = torch.tensor([1], dtype=torch.int32, device="cuda:0")
        with pytest.raises(si.SelectInferError) as e:
            si.selective_ffn(x, off, idx, gu, dn)
        assert e.value.status == 5


def test_check_flag_and_errors():
    say("check flag and error paths")
    rng, draw, ref, gpu = _rand_problem(5, 300, 64, 200, "bf16")
    x = dev_tensor(draw(2, 64, scale=1.0))
    good = [np.array([1, 5, 9], np.int32), np.array([0, 199], np.int32)]
    off, idx = csr_from_sets(good)
    y = si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c, gpu.down_c,
                         flags=si.FLAG_CHECK)
    assert max_rel_l2(host_array(y), _oracle(host_array(x), good, ref)) <= TOL["bf16"]
    cases = {
        3: [np.array([1, 5, 1], np.int32), np.array([2], np.int32)],      # duplicate
        2: [np.array([1, 200], np.int32), np.array([2], np.int32)],       # slot out of range
    }
    for code, sets in cases.items():
        off, idx = csr_from_sets(sets)
        with pytest.raises(si.SelectInferError) as e:
            si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c, gpu.down_c,
                             flags=si.FLAG_CHECK)
        assert e.value.status == code
    # SI_FLAG_SORTED: ascending lists pass the check, others are refused
    off, idx = csr_from_sets(good)
    y = si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c, gpu.down_c,
                         flags=si.FLAG_CHECK | si.FLAG_SORTED)
    assert max_rel_l2(host_array(y), _oracle(host_array(x), good, ref)) <= TOL["bf16"]
    for code, sets in {1: [np.array([1, 9, 5], np.int32), np.array([2], np.int32)],
                       3: [np.array([1, 5, 5], np.int32), np.array([2], np.int32)]}.items():
        off, idx = csr_from_sets(sets)
        with pytest.raises(si.SelectInferError) as e:
            si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c, gpu.down_c,
                             flags=si.FLAG_CHECK | si.FLAG_SORTED)
        assert e.value.status == code
    bad_off = dev_tensor(np.array([0, 3, 2], np.int32))
    with pytest.raises(si.SelectInferError) as e:
        si.selective_ffn(x, bad_off, dev_tensor(np.array([1, 2, 3], np.int32)), gpu.gate_up_c,
                         gpu.down_c, flags=si.FLAG_CHECK)
    assert e.value.status == 2
    # without the check, out-of-range slots are skipped (never read)
    off, idx = csr_from_sets([np.array([1, 100000, 5, -3], np.int32), np.array([7], np.int32)])
    y = host_array(si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c,
                                    gpu.down_c, flags=si.FLAG_PER_TOKEN))
    want = _oracle(host_array(x), [np.array([1, 5]), np.array([7])], ref)
    assert max_rel_l2(y, want) <= ALARM_PER_TOKEN
    # too small a workspace is refused
    off, idx = csr_from_sets(good)
    with pytest.raises(si.SelectInferError) as e:
        si.selective_ffn(x, dev_tensor(off), dev_tensor(idx), gpu.gate_up_c, gpu.down_c,
                         workspace=torch.empty(16, dtype=torch.uint8, device="cuda:0"))
    assert e.value.status == 7
    # B = 0 and nnz = 0
    e0 = si.selective_ffn(x[:0], dev_tensor(np.zeros(1, np.int32)), dev_tensor(np.zeros(0, np.int32)),
                          gpu.gate_up_c, gpu.down_c)
    assert e0.shape == (0, 64)
    z = si.selective_ffn(x, dev_tensor(np.zeros(3, np.int32)), dev_tensor(np.zeros(0, np.int32)),
                         gpu.gate_up_c, gpu.down_c)
    assert not torch.any(z)
