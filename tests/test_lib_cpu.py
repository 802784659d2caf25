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


def _enum_values():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return {k: int(v) for k, v in re.findall(r"\b(SI_[A-Z0-9_]+)\s*=\s*(\d+)", text)}


def _prototype(name):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    m = re.search(r"\b" + name + r"\s*\(([^)]*)\)", text)
    assert m, name
    return [a.strip() for a in " ".join(m.group(1).split()).split(",")]


def test_header_declares_the_boundary():
    """The calls, argument lists and enum values of the boundary the hot path is specified
    with: compaction, per-token top-k (with its workspace query), the selective FFN."""
    names = _declared()
    for n in ("si_compact_ffn", "si_select_topk", "si_select_topk_workspace",
              "si_selective_ffn", "si_selective_ffn_workspace", "si_status_string",
              "si_remap_ids", "si_residual_rmsnorm", "si_version"):
        assert n in names
    ev = _enum_values()
    want = dict(SI_F32=0, SI_BF16=1, SI_OK=0, SI_ERR_INVALID=1, SI_ERR_RANGE=2,
                SI_ERR_DUPLICATE=3, SI_ERR_NOT_LOADED=4, SI_ERR_UNSUPPORTED=5, SI_ERR_HIP=6,
                SI_TOPK_ABS=1, SI_TOPK_RAW=2, SI_FLAG_CHECK=4, SI_FLAG_SORTED=8)
    for k, v in want.items():
        assert ev.get(k) == v, k
    assert _prototype("si_compact_ffn") == [
        "const void* w_gate", "const void* w_up", "const void* w_down", "int64_t N",
        "int64_t d", "si_dtype wdt", "const int32_t* loaded", "int64_t L", "void* gate_up_c",
        "void* down_c", "int32_t* slot_to_orig", "int32_t* orig_to_slot", "void* hip_stream"]
    assert _prototype("si_select_topk_workspace") == ["int64_t B", "int64_t L", "int64_t k"]
    assert _prototype("si_select_topk") == [
        "const float* scores", "int64_t B", "int64_t L", "int64_t k", "int mode",
        "int32_t* out_idx", "void* ws", "size_t ws_bytes", "void* hip_stream"]
    assert _prototype("si_selective_ffn") == [
        "const void* x", "si_dtype xdt", "int64_t B", "int64_t d", "const int32_t* offsets",
        "const int32_t* idx", "int64_t nnz", "const void* gate_up_c", "const void* down_c",
        "int64_t L", "si_dtype wdt", "float* y", "void* ws", "size_t ws_bytes", "int flags",
        "void* hip_stream"]
    # the workspace query also takes the dtypes and flags, which choose the path
    assert _prototype("si_selective_ffn_workspace")[:4] == [
        "int64_t B", "int64_t nnz", "int64_t L", "int64_t d"]


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
    assert lib.si_version() == 200


def test_host_side_argument_errors(lib):
    # each of these returns before any HIP call
    ABS, RAW, SORTED = 1, 2, 8
    assert lib.si_select_topk_workspace(64, 11008, 2202) == 0
    assert lib.si_select_topk(None, 1, 4, 5, ABS, None, None, 0, None) == 1     # k > L
    assert lib.si_select_topk(None, 1, 4, 2, 0, None, None, 0, None) == 1       # no ranking key
    assert lib.si_select_topk(None, 1, 4, 2, ABS | RAW, None, None, 0, None) == 1   # two keys
    assert lib.si_select_topk(None, 1, 4, 2, 4, None, None, 0, None) == 1       # not a key
    assert lib.si_select_topk(None, 1, 4, 2, ABS, None, None, 16, None) == 7    # ws size, no ws
    assert lib.si_select_topk(None, 0, 4, 2, RAW | SORTED, None, None, 0, None) == 0  # B = 0: no-op
    assert lib.si_select_topk(None, 3, 4, 0, ABS, None, None, 0, None) == 0     # k = 0: no-op
    assert lib.si_dynamic_set(None, 1, 4, 64, None, 10, 1, None, 0, 2, 3, 0, None, None, None,
                              0, None) == 1                              # no ranking key
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
    PER, UNION = 16, 64
    for B in (2, 3, 4):
        assert ws(B, 0) == ws(B, PER)
        assert ws(B, UNION) != ws(B, PER)
    for B in (5, 16):
        assert ws(B, 0) == ws(B, UNION)
        assert ws(B, 0) != ws(B, PER)
    assert ws(16, 0, dt=0) == ws(16, PER, dt=0)                          # f32: per-token


def test_h_form_workspace(lib):
    """From 128 tokens (the tiled GEMMs) h is one 16-bit value unless SI_FLAG_EXACT_H, whose
    workspace adds the lo plane of H; FAST_H names the default and wins over EXACT_H; below
    128 tokens the H flags do not change the workspace. The 13B-shape 512-token prefill fits
    the no-allocation entry point's scratch either way."""
    ws = lambda B, flags, L=9677, d=5120: lib.si_selective_ffn_workspace(
        B, 3456 * B, L, d, 1, 1, flags)
    EXACT, FAST = 128, 32
    up = (9677 + 63) // 64 * 64
    assert ws(512, EXACT) - ws(512, 0) == (512 * up * 2 + 255) // 256 * 256
    assert ws(512, FAST) == ws(512, 0) == ws(512, FAST | EXACT)
    assert ws(16, EXACT) == ws(16, 0) == ws(16, FAST)
    assert ws(512, EXACT) <= 64 << 20


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


def test_no_kernel_spills():
    """Every kernel instance in the library keeps its state in registers: no scratch (register
    spill) memory, by the compiler's per-kernel resource remarks recorded at build time."""
    import json
    import os
    from paper_2607_18081_amd import build as b
    if not os.path.exists(b.USAGE):
        pytest.skip("the library was not built by build() in this tree (no resource record)")
    usage = json.load(open(b.USAGE))
    assert len(usage) > 50                   # every source's kernels were recorded
    spilled = [(u["kernel"], u.get("scratch_bytes_per_lane")) for u in usage
               if u.get("scratch_bytes_per_lane", 0) != 0]
    assert not spilled, spilled
