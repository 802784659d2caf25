"""GPU parity of si_load_selected: bit-identical to the oracle's compaction, whether the full
layer sits in ordinary host memory or in a memory-mapped file."""
import os
import tempfile

import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import host_array, say
from workloads import CONFIGS, layer_weights, loaded_ids

pytestmark = pytest.mark.gpu


def _same(layer, ref):
    assert np.array_equal(host_array(layer.gate_up_c), ref["gate_up_c"])
    assert np.array_equal(host_array(layer.down_c), ref["down_c"])
    assert np.array_equal(host_array(layer.slot_to_orig), ref["slot_to_orig"])
    assert np.array_equal(host_array(layer.orig_to_slot), ref["orig_to_slot"])


@pytest.mark.parametrize("wdtype,N,d,L", [("bf16", 900, 264, 613), ("f32", 300, 100, 1),
                                          ("f32", 257, 12, 257), ("f16", 500, 72, 333),
                                          ("f32", 20001, 1000, 20000)])
def test_load_selected_ragged(wdtype, N, d, L):
    """Ragged d and L; the last case needs two staging buffers of W_down rows cut to the loaded
    columns (20000 * 4 bytes a row, 838 rows a buffer) and three of gate/up rows."""
    say(f"load_selected {wdtype} N={N} d={d} L={L}")
    rng = np.random.default_rng(N + d)
    def draw(*s):
        a = rng.standard_normal(s).astype(np.float32)
        if wdtype == "f16":
            return a.astype(np.float16)
        return (a.view(np.uint32) >> 16).astype(np.uint16) if wdtype == "bf16" else a
    wg, wu, wd = draw(N, d), draw(N, d), draw(d, N)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    _same(si.load_selected(wg, wu, wd, loaded), oracle.compact(wg, wu, wd, loaded))


def test_load_selected_7b_from_mapped_file():
    cfg = CONFIGS["llama2_7b_decode"]
    say("load_selected: 7B-shape layer from a memory-mapped file")
    wg, wu, wd = layer_weights(cfg, 0)
    loaded = loaded_ids(cfg, 0)
    ref = oracle.compact(wg, wu, wd, loaded)
    with tempfile.TemporaryDirectory() as tmp:
        maps = []
        for name, a in (("gate", wg), ("up", wu), ("down", wd)):
            path = os.path.join(tmp, name + ".bin")
            a.tofile(path)
            maps.append(np.memmap(path, dtype=a.dtype, mode="r", shape=a.shape))
        layer = si.load_selected(*maps, loaded)
        torch.cuda.synchronize()
        del maps
    _same(layer, ref)


def test_load_selected_errors():
    w = np.zeros((8, 16), np.float32)
    wd = np.zeros((16, 8), np.float32)
    with pytest.raises(si.SelectInferError):
        si.load_selected(w, w, wd, np.array([1, 1], np.int32))
    with pytest.raises(si.SelectInferError):
        si.load_selected(w, w, wd, np.array([3, 8], np.int32))
