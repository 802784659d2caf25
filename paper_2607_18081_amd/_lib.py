"""ctypes view of libselectinfer.so (the C ABI declared in include/selectinfer.h).

Loading fails loudly when the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libselectinfer.so")

c_i64 = ctypes.c_int64
c_int = ctypes.c_int
c_vp = ctypes.c_void_p
c_size = ctypes.c_size_t

# name -> (restype, argtypes); must match include/selectinfer.h
SIGNATURES = {
    "si_version": (c_int, []),
    "si_status_string": (ctypes.c_char_p, [c_int]),
    "si_compact_ffn": (c_int, [c_vp, c_vp, c_vp, c_i64, c_i64, c_int, c_vp, c_i64,
                               c_vp, c_vp, c_vp, c_vp, c_vp]),
    "si_remap_ids": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_int, c_vp]),
    "si_select_topk_workspace": (c_size, [c_i64, c_i64, c_i64]),
    "si_select_topk": (c_int, [c_vp, c_i64, c_i64, c_i64, c_int, c_vp, c_vp, c_size, c_vp]),
    "si_selective_ffn_workspace": (c_size, [c_i64, c_i64, c_i64, c_i64, c_int, c_int, c_int]),
    "si_selective_ffn": (c_int, [c_vp, c_int, c_i64, c_i64, c_vp, c_vp, c_i64, c_vp, c_vp,
                                 c_i64, c_int, c_vp, c_vp, c_size, c_int, c_vp]),
    "si_selective_ffn_noalloc": (c_int, [c_vp, c_int, c_i64, c_i64, c_vp, c_vp, c_i64, c_vp, c_vp,
                                         c_i64, c_int, c_vp, c_int, c_vp]),
    "si_selective_ffn_resnorm": (c_int, [c_vp, c_vp, ctypes.c_float, c_vp, c_int, c_i64, c_i64,
                                         c_vp, c_vp, c_i64, c_vp, c_vp, c_i64, c_int, c_vp, c_vp,
                                         c_size, c_int, c_vp]),
    "si_set_timing_events": (c_int, [c_vp, c_vp]),
    "si_ceiling_stream": (c_int, [c_vp, c_i64, c_int, c_vp, c_vp]),
    "si_ceiling_gather": (c_int, [c_vp, c_vp, c_i64, c_i64, c_int, c_vp, c_i64, c_int, c_vp,
                                  c_vp]),
    "si_residual_rmsnorm": (c_int, [c_vp, c_int, c_vp, c_i64, c_i64, ctypes.c_float, c_vp,
                                    c_vp]),
    "si_dynamic_set_workspace": (c_size, [c_i64, c_i64, c_i64, c_i64]),
    "si_dynamic_set": (c_int, [c_vp, c_int, c_i64, c_i64, c_vp, c_i64, c_int, c_vp, c_i64, c_i64,
                               c_i64, c_int, c_vp, c_vp, c_vp, c_size, c_vp]),
    "si_profile_scores_workspace": (c_size, [c_i64, c_i64, c_i64, c_int, c_int]),
    "si_profile_scores": (c_int, [c_vp, c_int, c_i64, c_i64, c_vp, c_i64, c_int, c_vp, c_vp,
                                  c_size, c_vp]),
    "si_merge_scores": (c_int, [c_vp, c_vp, c_i64, c_i64, c_vp, c_vp]),
    "si_rank_neurons": (c_int, [c_vp, c_i64, c_vp, c_vp]),
    "si_build_loaded_set": (c_int, [c_vp, c_vp, c_i64, c_i64, c_i64, c_vp]),
    "si_selective_layers": (c_int, [c_i64, c_i64, c_i64, c_vp, c_vp]),
    "si_load_selected": (c_int, [c_vp, c_vp, c_vp, c_i64, c_i64, c_int, c_vp, c_i64, c_vp, c_vp,
                                 c_vp, c_vp, c_vp]),
}

_lib = None


class LibraryMissing(RuntimeError):
    pass


def load() -> ctypes.CDLL:
    """The loaded library; raises LibraryMissing if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(
                f"{LIB_PATH} is missing: build it with `python -m paper_2607_18081_amd.build` "
                "(the selective FFN has no non-HIP implementation)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib
