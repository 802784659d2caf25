"""si_build_loaded_set runs on the host only: checked here through the C ABI, without a GPU,
against the oracle's loaded-set construction (exact)."""
import numpy as np
import pytest

import oracle
import paper_2607_18081_amd as si


@pytest.mark.parametrize("seed", range(6))
def test_build_loaded_set_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 3000))
    t, m = rng.permutation(N).astype(np.int32), rng.permutation(N).astype(np.int32)
    nb = int(rng.integers(0, N + 1))
    nl = int(rng.integers(nb, N + 1))
    got = si.build_loaded_set(t, m, nb, nl)
    assert np.array_equal(got, oracle.build_loaded_set(t, m, nb, nl))


def test_build_loaded_set_table1_fractions():
    # Table 1: 30% base (task-specific) neurons, 70% loaded, on a 7B-shape layer
    N = 11008
    rng = np.random.default_rng(1)
    t, m = rng.permutation(N).astype(np.int32), rng.permutation(N).astype(np.int32)
    nb, nl = round(0.3 * N), round(0.7 * N)
    got = si.build_loaded_set(t, m, nb, nl)
    assert len(got) == nl == len(set(got.tolist()))
    assert np.array_equal(got[:nb], t[:nb])


def test_build_loaded_set_errors():
    t = np.arange(5, dtype=np.int32)
    with pytest.raises(si.SelectInferError):
        si.build_loaded_set(t, np.array([0, 1, 2, 3, 3], np.int32), 1, 2)   # not a permutation
    with pytest.raises(si.SelectInferError):
        si.build_loaded_set(t, t, 3, 2)                                     # n_loaded < n_base
    with pytest.raises(si.SelectInferError):
        si.build_loaded_set(t, t, 0, 6)                                     # n_loaded > N


def test_selective_layers_table1():
    """si_selective_layers against the oracle's layer range and Table 1's counts: layers 5 to
    the second-last (exclusive) of 28 and of 16 layers (21 and 9, the Memory Footprint
    section's 9 of 16 for the 1B model)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "table1_parameters.json")))
    first, last = g["first_layer"], g["last_layer"]
    for n in (0, 1, 5, 6, 7, 8, 16, 28, 32, 80):
        got = si.selective_layers(n, first, last)
        assert np.flatnonzero(got).tolist() == oracle.selective_layers(n, first, last)
    assert int(si.selective_layers(g["n_layers_llama32_1b"], first, last).sum()) == \
        g["selected_layers_llama32_1b"]
    assert int(si.selective_layers(g["n_layers_llama32_3b"], first, last).sum()) == 21
    m32 = si.selective_layers(32)                      # the defaults are Table 1's
    assert np.flatnonzero(~m32).tolist() == [0, 1, 2, 3, 4, 30, 31]


def test_selective_layers_errors():
    for args in ((-1, 5, -2), (8, -1, -2), (8, 5, 1)):
        with pytest.raises(si.SelectInferError):
            si.selective_layers(*args)
    assert not si.selective_layers(4, 5, -2).any()      # range past the end: no layer
