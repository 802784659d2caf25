"""The seeded input generator: determinism, shapes and the statistics each workload states."""
import numpy as np

import oracle
from workloads import CONFIGS, active_sets, csr_from_sets, es_keys, layer_weights, loaded_ids, \
    popularity, storage_from_f32, tokens_x


def test_config_counts():
    c = CONFIGS
    assert (c["tiny_f32"].L, c["tiny_f32"].k) == (512, 128)
    assert (c["llama2_7b_decode"].L, c["llama2_7b_decode"].k) == (7706, 2202)
    assert c["llama2_7b_b16"].hot == 1101
    assert (c["llama3_8b_stack"].L, c["llama3_8b_stack"].k) == (8602, 2150)
    assert (c["llama2_13b_prefill"].L, c["llama2_13b_prefill"].k) == (9677, 3456)


def test_deterministic_and_layer_dependent():
    cfg = CONFIGS["tiny_f32"]
    a = layer_weights(cfg, 0)
    b = layer_weights(cfg, 0)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    c = layer_weights(cfg, 1)
    assert not np.array_equal(a[0], c[0])
    assert a[0].shape == (1024, 256) and a[2].shape == (256, 1024) and a[0].dtype == np.float32
    assert abs(float(a[0].std()) - 0.02) < 1e-3
    assert np.array_equal(tokens_x(cfg, [3, 5]), tokens_x(cfg, [3, 5]))


def test_bf16_storage_rounding():
    v = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.0], dtype=np.float32)
    got = storage_from_f32(v, "bf16")
    assert list(got) == [0x3F80, 0x3F80, 0x3F82, 0xC000]


def test_loaded_is_top_popularity():
    cfg = CONFIGS["llama2_7b_decode"]
    pi, w = popularity(cfg)
    ld = loaded_ids(cfg)
    assert len(set(ld.tolist())) == cfg.L
    assert np.array_equal(ld, pi[: cfg.L])
    assert w[pi[0]] == 1.0 and np.all(np.diff(w[pi]) < 0)


def test_active_sets_are_topk_of_keys():
    cfg = CONFIGS["tiny_f32"]
    keys = es_keys(cfg, range(4))
    sets = active_sets(cfg, range(4))
    slots_of = np.sort(loaded_ids(cfg))
    for t in range(4):
        want = slots_of[oracle.select_topk(keys[t], cfg.k, "raw")]
        assert np.array_equal(np.sort(want), sets[t])
        assert len(sets[t]) == cfg.k and np.all(np.diff(sets[t]) > 0)


def test_hot_core_overlap_statistics():
    cfg = CONFIGS["llama2_7b_b16"]
    sets = active_sets(cfg, range(16))
    pi, _ = popularity(cfg)
    core = set(pi[: cfg.hot].tolist())
    inter = []
    for i in range(16):
        assert core <= set(sets[i].tolist())
        for j in range(i + 1, 16):
            inter.append(len(np.intersect1d(sets[i], sets[j])) / cfg.k)
    union = len(np.unique(np.concatenate(sets)))
    assert 0.55 < float(np.mean(inter)) < 0.67        # "~60% overlap"
    assert 6500 < union < 7300                         # about 0.9 L


def test_csr():
    off, ids = csr_from_sets([np.array([1, 2]), np.array([], np.int32), np.array([7])])
    assert off.tolist() == [0, 2, 2, 3] and ids.tolist() == [1, 2, 7]


def test_table1_stack_dense_layers():
    """The Table 1 stack: its selective layers are the 8B stack's own (same seeds); a dense
    layer loads and activates every neuron."""
    a, b = CONFIGS["llama3_8b_stack"], CONFIGS["llama3_8b_stack_table1"]
    small = dict(d=64, N=300, L=180, k=45)
    a, b = a.with_(**small), b.with_(**small)
    assert np.array_equal(loaded_ids(a, 7), loaded_ids(b, 7))
    for x, y in zip(active_sets(a, range(3), 7), active_sets(b, range(3), 7)):
        assert np.array_equal(x, y)
    assert b.L_of(0) == b.k_of(31) == 300 and b.L_of(5) == 180 and b.k_of(29) == 45
    assert np.array_equal(np.sort(loaded_ids(b, 0)), np.arange(300))
    for s in active_sets(b, range(2), 31):
        assert np.array_equal(s, np.arange(300))
