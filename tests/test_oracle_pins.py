"""The oracle against its pins (CPU only)."""
import json
import os

import numpy as np
import pytest

import oracle
from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle)


def test_table1_fractions_add_up():
    with open(os.path.join(pins.GOLDEN, "table1_parameters.json")) as f:
        t = json.load(f)
    assert t["base_static_pct"] + t["secondary_pct"] == t["loaded_pct"]
    assert t["base_static_pct"] + t["dynamic_pct"] == t["computed_pct"]
    # layers [5, n-2): 21 of 28 (r_layer = 0.75 in Eq. 2) and 9 of 16
    n3, n1 = t["n_layers_llama32_3b"], t["n_layers_llama32_1b"]
    assert (n3 + t["last_layer"]) - t["first_layer"] == 21 == 0.75 * n3
    assert (n1 + t["last_layer"]) - t["first_layer"] == t["selected_layers_llama32_1b"]


def test_dense_helper_matches_pin_reference():
    wg, wu, wd, x = pins._problem(1, 17, 9)
    mask = (np.arange(17) % 3 == 0).astype(float)
    a = oracle.dense_swiglu(x, wg, wu, wd, mask)
    b = pins._masked_dense(x, wg, wu, wd, mask)
    assert pins._rel(a, b) <= 1e-14


def test_stack_step_consistent():
    wg, wu, wd, x = pins._problem(2, 20, 16, "bf16")
    c = oracle.compact(wg, wu, wd, range(20))
    y, xn = oracle.stack_step(x, [1, 5, 7], c["gate_up_c"], c["down_c"])
    assert np.array_equal(xn, oracle.residual_rmsnorm_bf16(x, y))
    assert xn.dtype == np.uint16 and xn.shape == (16,)
