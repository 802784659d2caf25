"""The C-ABI library loads and exports what include/selectinfer.h declares (no GPU needed).

Only host-side paths run here: nothing below launches a kernel or initialises a device.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "selectinfer.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(si_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_18081_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2607_18081_amd import build
        build.build()
    return _lib.load()


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("si_compact_ffn", "si_select_topk", "si_selective_ffn", "si_remap_ids",
              "si_selective_ffn_workspace", "si_residual_rmsnorm", "si_status_string",
              "si_version"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for n in _declared():
        assert hasattr(lib, n), n


def test_binding_signatures_cover_header():
    from paper_2607_18081_amd._lib import SIGNATURES
    assert sorted(SIGNATURES) == _declared()


def test_status_strings(lib):
    assert lib.si_status_string(0) == b"ok"
    assert b"range" in lib.si_status_string(2)
    assert lib.si_status_string(999) == b"unknown status"
    assert lib.si_version() == 100


def test_host_side_argument_errors(lib):
    # each of these returns before any HIP call
    assert lib.si_select_topk(None, 1, 4, 5, 0, None, None) == 1          # k > L
    assert lib.si_select_topk(None, 1, 4, 2, 7, None, None) == 1          # bad mode
    assert lib.si_select_topk(None, 0, 4, 2, 0, None, None) == 0          # B = 0: no-op
    assert lib.si_select_topk(None, 3, 4, 0, 0, None, None) == 0          # k = 0: no-op
    assert lib.si_selective_ffn(None, 1, 1, 0, None, None, 0, None, None, 4, 1, None, None,
                                0, 0, None) == 1                          # d < 1
    assert lib.si_selective_ffn(None, 3, 1, 8, None, None, 0, None, None, 4, 1, None, None,
                                0, 0, None) == 5                          # bad dtype
    assert lib.si_selective_ffn(None, 1, 1, 12, None, None, 0, None, None, 4, 1, None, None,
                                0, 0, None) == 5                          # bf16 needs d % 8
    assert lib.si_selective_ffn(None, 1, 0, 8, None, None, 0, None, None, 4, 1, None, None,
                                0, 0, None) == 0                          # B = 0: no-op
    assert lib.si_compact_ffn(None, None, None, 4, 8, 1, None, 2, None, None, None, None,
                              None) == 1                                  # NULL pointers
    assert lib.si_remap_ids(None, 4, None, 0, None, 0, None) == 0         # n = 0: no-op
    assert lib.si_residual_rmsnorm(None, 1, None, 1, 8, ctypes.c_float(-1.0), None,
                                   None) == 1                             # eps < 0


def test_path_choice_by_batch(lib):
    """The workspace query follows the path the call takes: per-token below 5 tokens (unless
    SI_FLAG_UNION), the union path from 5 (unless SI_FLAG_PER_TOKEN), per-token for f32."""
    ws = lambda B, flags, dt=1: lib.si_selective_ffn_workspace(B, 2202 * B, 7706, 4096, dt, dt,
                                                               flags)
    PER, UNION = 2, 8
    for B in (2, 3, 4):
        assert ws(B, 0) == ws(B, PER)
        assert ws(B, UNION) != ws(B, PER)
    for B in (5, 16):
        assert ws(B, 0) == ws(B, UNION)
        assert ws(B, 0) != ws(B, PER)
    assert ws(16, 0, dt=0) == ws(16, PER, dt=0)                          # f32: per-token


def test_lib_exports_resnorm_entry(lib):
    # x_out overlapping x_prev is refused before anything is enqueued
    buf = ctypes.create_string_buffer(1024)
    p = ctypes.addressof(buf)
    p16 = (p + 15) & ~15
    assert lib.si_selective_ffn_resnorm(p16, p16 + 256, ctypes.c_float(1e-5), p16 + 16, 1, 1, 64,
                                        None, None, 0, None, None, 4, 1, None, None, 0, 0,
                                        None) == 1
    assert lib.si_selective_ffn_resnorm(None, None, ctypes.c_float(1e-5), None, 2, 1, 64, None,
                                        None, 0, None, None, 4, 2, None, None, 0, 0,
                                        None) == 5                        # half x


def test_product_path_fails_without_library(monkeypatch, tmp_path):
    from paper_2607_18081_amd import _lib
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(_lib.LibraryMissing):
        _lib.load()
