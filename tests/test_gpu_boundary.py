"""GPU parity of the boundary calls: compaction, remap, top-k, residual RMSNorm, errors.

Integer and copy results must match the oracle bit for bit.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, rel_l2, say
from workloads import CONFIGS, es_keys, layer_weights, loaded_ids

pytestmark = pytest.mark.gpu


def _rand_layer(seed, N, d, wdtype):
    rng = np.random.default_rng(seed)
    def draw(*shape):
        a = (rng.standard_normal(shape) * 0.02).astype(np.float32)
        return (a.view(np.uint32) >> 16).astype(np.uint16) if wdtype == "bf16" else a
    return draw(N, d), draw(N, d), draw(d, N)


def _compact_both(wg, wu, wd, loaded):
    c = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                       torch.from_numpy(np.asarray(loaded, np.int32)))
    ref = oracle.compact(wg, wu, wd, loaded)
    return c, ref


def _assert_compact_equal(c, ref):
    assert np.array_equal(host_array(c.slot_to_orig), ref["slot_to_orig"])
    assert np.array_equal(host_array(c.orig_to_slot), ref["orig_to_slot"])
    assert np.array_equal(host_array(c.gate_up_c), ref["gate_up_c"])
    assert np.array_equal(host_array(c.down_c), ref["down_c"])


@pytest.mark.parametrize("name", ["tiny_f32", "llama2_7b_decode"])
def test_compaction_matches_oracle_at_workload_size(name):
    cfg = CONFIGS[name]
    say(f"compaction {name}")
    wg, wu, wd = layer_weights(cfg)
    loaded = loaded_ids(cfg)
    c, ref = _compact_both(wg, wu, wd, loaded)
    _assert_compact_equal(c, ref)
    # the order of the loaded list does not matter
    c2 = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd),
                        torch.from_numpy(loaded[::-1].copy()))
    assert torch.equal(c2.gate_up_c, c.gate_up_c) and torch.equal(c2.down_c, c.down_c)
    # Eq. 2: the compacted layer holds 3*d*L*s bytes
    s = 2 if cfg.wdtype == "bf16" else 4
    nbytes = c.gate_up_c.numel() * s + c.down_c.numel() * s
    assert nbytes == oracle.compacted_bytes(cfg.d, cfg.L, s)


@pytest.mark.parametrize("N,d,L,wdtype", [(1000, 264, 333, "bf16"), (130, 8, 130, "bf16"),
                                          (77, 4, 1, "f32"), (300, 100, 299, "f32")])
def test_compaction_ragged_shapes(N, d, L, wdtype):
    say(f"compaction ragged N={N} d={d} L={L} {wdtype}")
    wg, wu, wd = _rand_layer(N + d, N, d, wdtype)
    loaded = np.random.default_rng(L).permutation(N)[:L].astype(np.int32)
    c, ref = _compact_both(wg, wu, wd, loaded)
    _assert_compact_equal(c, ref)


def test_compaction_errors():
    say("compaction errors")
    wg, wu, wd = _rand_layer(1, 50, 16, "bf16")
    g, u, dn = dev_tensor(wg), dev_tensor(wu), dev_tensor(wd)
    with pytest.raises(si.SelectInferError) as e:
        si.compact_ffn(g, u, dn, torch.tensor([3, 9, 3], dtype=torch.int32))
    assert e.value.status == 3
    with pytest.raises(si.SelectInferError) as e:
        si.compact_ffn(g, u, dn, torch.tensor([3, 50], dtype=torch.int32))
    assert e.value.status == 2
    with pytest.raises(si.SelectInferError) as e:
        si.compact_ffn(g, u, dn, torch.tensor([-1], dtype=torch.int32))
    assert e.value.status == 2
    # a good call afterwards is unaffected by the earlier errors
    c, ref = _compact_both(wg, wu, wd, [5, 1, 30])
    _assert_compact_equal(c, ref)


def test_remap_matches_oracle():
    say("remap")
    N = 5000
    rng = np.random.default_rng(3)
    loaded = rng.permutation(N)[:3100].astype(np.int32)
    ref = oracle.compact(np.zeros((N, 8), np.float32), np.zeros((N, 8), np.float32),
                         np.zeros((8, N), np.float32), loaded)
    o2s = dev_tensor(ref["orig_to_slot"])
    ids = rng.permutation(loaded)[:2000]
    got = host_array(si.remap_ids(o2s, torch.from_numpy(ids)))
    assert np.array_equal(got, oracle.remap(ref["orig_to_slot"], ids))
    got_c = host_array(si.remap_ids(o2s, torch.from_numpy(ids), check=True))
    assert np.array_equal(got_c, got)
    # not loaded / out of range -> -1, and errors under check
    not_loaded = np.setdiff1d(np.arange(N), loaded)[:3].astype(np.int32)
    bad = np.concatenate([ids[:5], not_loaded, np.array([N, -7], np.int32)])
    out = host_array(si.remap_ids(o2s, torch.from_numpy(bad)))
    assert list(out[5:]) == [-1] * 5
    with pytest.raises(si.SelectInferError) as e:
        si.remap_ids(o2s, torch.from_numpy(np.concatenate([ids[:5], not_loaded])), check=True)
    assert e.value.status == 4
    with pytest.raises(si.SelectInferError) as e:
        si.remap_ids(o2s, torch.tensor([int(ids[0]), N + 3], dtype=torch.int32), check=True)
    assert e.value.status == 2
    assert si.remap_ids(o2s, torch.zeros(0, dtype=torch.int32)).numel() == 0


@pytest.mark.parametrize("name", ["tiny_f32", "llama2_7b_decode", "llama2_13b_prefill"])
def test_topk_matches_oracle_on_sampling_keys(name):
    cfg = CONFIGS[name]
    say(f"topk keys {name}")
    keys = es_keys(cfg, range(6))
    got = host_array(si.select_topk(dev_tensor(keys), cfg.k, "raw"))
    for t in range(6):
        assert np.array_equal(got[t], oracle.select_topk(keys[t], cfg.k, "raw"))
    got_abs = host_array(si.select_topk(dev_tensor(keys), cfg.k, "abs"))
    for t in range(2):
        assert np.array_equal(got_abs[t], oracle.select_topk(keys[t], cfg.k, "abs"))


@pytest.mark.parametrize("L", [1, 7, 1000, 1024, 1025, 5000, 16384, 16385, 32768, 32769, 40000])
def test_topk_ties_zeros_nan(L):
    """Rows held in registers (up to 32768 keys, 1 to 32 per thread) and longer rows, which the
    kernel reads again in each radix pass."""
    say(f"topk adversarial L={L}")
    rng = np.random.default_rng(L)
    pool = np.array([0.0, -0.0, 1.0, -1.0, 2.5, -2.5, np.inf, -np.inf, np.nan, 0.125,
                     3e-39, -3e-39], dtype=np.float32)
    rows = np.stack([pool[rng.integers(0, len(pool), L)],
                     rng.standard_normal(L).astype(np.float32).round(1),
                     np.full(L, 5.0, np.float32),
                     np.where(rng.random(L) < 0.5, np.float32(np.nan), np.float32(-0.0))])
    scores = dev_tensor(rows)
    for k in sorted({0, 1, L // 2, max(L - 1, 0), L}):
        for mode in ("abs", "raw"):
            got = host_array(si.select_topk(scores, k, mode))
            for b in range(rows.shape[0]):
                assert np.array_equal(got[b], oracle.select_topk(rows[b], k, mode)), (k, mode, b)
    with pytest.raises(si.SelectInferError):
        si.select_topk(scores, L + 1)


@pytest.mark.parametrize("seed", range(16))
def test_topk_random_shapes(seed):
    """Seeded random rows, lengths and k (including 0 and L), in both modes: integer-valued,
    coarsely rounded (many ties), normal, and tiny (subnormal) keys, exact against the oracle."""
    rng = np.random.default_rng(300 + seed)
    B = int(rng.integers(1, 41))
    L = int(rng.choice([int(rng.integers(1, 2000)), int(rng.integers(2000, 50000))]))
    kind = seed % 4
    if kind == 0:
        rows = rng.integers(-20, 21, (B, L)).astype(np.float32)
    elif kind == 1:
        rows = rng.standard_normal((B, L)).astype(np.float32).round(2)
    elif kind == 2:
        rows = rng.standard_normal((B, L)).astype(np.float32)
    else:
        rows = (rng.standard_normal((B, L)) * 1e-39).astype(np.float32)
    k = int(rng.choice([0, L, int(rng.integers(0, L + 1)), min(L, int(rng.integers(1, 64)))]))
    mode = ("abs", "raw")[seed % 2]
    say(f"topk random seed={seed}: B={B} L={L} k={k} {mode} kind={kind}")
    got = host_array(si.select_topk(dev_tensor(rows), k, mode))
    assert got.shape == (B, k)
    for b in range(B):
        assert np.array_equal(got[b], oracle.select_topk(rows[b], k, mode)), b


@pytest.mark.parametrize("xdt,d", [("bf16", 4096), ("f32", 4096), ("bf16", 20000),
                                   ("f32", 100), ("bf16", 102), ("f32", 4098)])
def test_residual_rmsnorm(xdt, d):
    """d = 4096: one chunk held in registers; 20000: past the register-held size, the second
    pass reads again; 102 and 4098 (not multiples of 4): the generic kernel."""
    say(f"rmsnorm {xdt} d={d}")
    rng = np.random.default_rng(9 + d)
    B = 5
    x32 = rng.standard_normal((B, d)).astype(np.float32)
    x = (x32.view(np.uint32) >> 16).astype(np.uint16) if xdt == "bf16" else x32
    y = (rng.standard_normal((B, d)) * 0.3).astype(np.float32)
    got = host_array(si.residual_rmsnorm(dev_tensor(x), dev_tensor(y)))
    for b in range(B):
        ref_bits = oracle.residual_rmsnorm_bf16(x[b], y[b])
        ref = oracle.decode(ref_bits)
        if xdt == "bf16":
            assert rel_l2(oracle.decode(got[b]), ref) <= 5e-3
            assert np.mean(got[b] == ref_bits) > 0.99
        else:
            r = oracle.decode(x[b]) + y[b].astype(np.float64)
            exact = r / math.sqrt(np.mean(r * r) + 1e-5)
            assert rel_l2(got[b], exact) <= 1e-6
    # in place
    xt = dev_tensor(x)
    out = si.residual_rmsnorm(xt, dev_tensor(y), out=xt)
    assert np.array_equal(host_array(out), got)
