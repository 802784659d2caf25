"""Python binding of the selective-FFN C ABI (argument marshalling only).

Tensors are PyTorch tensors on a ROCm device; they supply device memory and the current HIP
stream. Every computation happens in the HIP kernels of libselectinfer.so. Function names
follow the C entry points without their ``si_`` prefix.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import torch

from ._lib import load

F32, BF16, F16 = 0, 1, 2
TOPK_ABS, TOPK_RAW = 1, 2
FLAG_CHECK, FLAG_SORTED, FLAG_PER_TOKEN, FLAG_FAST_H, FLAG_UNION = 4, 8, 16, 32, 64
FLAG_EXACT_H = 128
_MODES = {"abs": TOPK_ABS, "raw": TOPK_RAW}

_DT = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}


class SelectInferError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = load().si_status_string(status).decode()
        super().__init__(f"{where}: {msg} (status {status})")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != 0:
        raise SelectInferError(status, where)


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}") from None


def _dev(t: torch.Tensor) -> torch.device:
    if t.device.type != "cuda":
        raise ValueError("tensors must live on a ROCm GPU device")
    return t.device


def _ptr(t):
    if t is None or t.numel() == 0:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def version() -> int:
    return load().si_version()


@dataclass
class CompactLayer:
    """A compacted FFN layer: only the loaded neurons, neuron-major."""
    gate_up_c: torch.Tensor      # [L][2][d]
    down_c: torch.Tensor         # [L][d]
    slot_to_orig: torch.Tensor   # [L] int32, ascending
    orig_to_slot: torch.Tensor   # [N] int32, -1 = not loaded

    @property
    def L(self) -> int:
        return self.gate_up_c.shape[0]

    @property
    def d(self) -> int:
        return self.gate_up_c.shape[2]


def compact_ffn(w_gate: torch.Tensor, w_up: torch.Tensor, w_down: torch.Tensor,
                loaded: torch.Tensor) -> CompactLayer:
    """si_compact_ffn: W_gate/W_up [N][d], W_down [d][N], loaded ids [L] -> CompactLayer."""
    dev = _dev(w_gate)
    N, d = w_gate.shape
    if w_up.shape != (N, d) or w_down.shape != (d, N):
        raise ValueError("weight shapes must be [N][d], [N][d], [d][N]")
    if not (w_gate.dtype == w_up.dtype == w_down.dtype):
        raise ValueError("weights must share one dtype")
    loaded = loaded.to(device=dev, dtype=torch.int32).contiguous()
    L = loaded.numel()
    gu = torch.empty((L, 2, d), dtype=w_gate.dtype, device=dev)
    dc = torch.empty((L, d), dtype=w_gate.dtype, device=dev)
    s2o = torch.empty(L, dtype=torch.int32, device=dev)
    o2s = torch.empty(N, dtype=torch.int32, device=dev)
    st = load().si_compact_ffn(_ptr(w_gate), _ptr(w_up), _ptr(w_down), N, d, _dt(w_gate),
                               _ptr(loaded), L, _ptr(gu), _ptr(dc), _ptr(s2o), _ptr(o2s),
                               _stream(dev))
    _check(st, "si_compact_ffn")
    return CompactLayer(gu, dc, s2o, o2s)


def remap_ids(orig_to_slot: torch.Tensor, ids: torch.Tensor, check: bool = False,
              out: torch.Tensor | None = None) -> torch.Tensor:
    """si_remap_ids: original ids -> slots (-1 where not loaded)."""
    dev = _dev(orig_to_slot)
    ids = ids.to(device=dev, dtype=torch.int32).contiguous()
    if out is None:
        out = torch.empty_like(ids)
    st = load().si_remap_ids(_ptr(orig_to_slot), orig_to_slot.numel(), _ptr(ids), ids.numel(),
                             _ptr(out), FLAG_CHECK if check else 0, _stream(dev))
    _check(st, "si_remap_ids")
    return out


def select_topk(scores: torch.Tensor, k: int, mode: str = "abs",
                out: torch.Tensor | None = None) -> torch.Tensor:
    """si_select_topk: scores [B][L] float32 -> [B][k] int32, rows ascending."""
    dev = _dev(scores)
    if scores.dtype != torch.float32 or scores.dim() != 2:
        raise ValueError("scores must be a 2-D float32 tensor")
    B, L = scores.shape
    if out is None:
        out = torch.empty((B, k), dtype=torch.int32, device=dev)
    lib = load()
    need = int(lib.si_select_topk_workspace(B, L, k))
    ws = _workspace(dev, need) if need > 0 else None
    st = lib.si_select_topk(_ptr(scores), B, L, k, _MODES[mode], _ptr(out), _ptr(ws),
                            ws.numel() if ws is not None else 0, _stream(dev))
    _check(st, "si_select_topk")
    return out


def selective_ffn_workspace(B: int, nnz: int, L: int, d: int, xdt=BF16, wdt=BF16,
                            flags: int = 0) -> int:
    return int(load().si_selective_ffn_workspace(B, nnz, L, d, xdt, wdt, flags))


_WS: dict = {}


def _workspace(dev: torch.device, nbytes: int) -> torch.Tensor:
    """A per-device workspace that only grows. Calls sharing it must not overlap in time
    (pass ``workspace=`` explicitly when using several streams)."""
    key = (dev.type, dev.index)
    ws = _WS.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        _WS[key] = ws
    return ws


def selective_ffn(x: torch.Tensor, offsets: torch.Tensor, idx: torch.Tensor,
                  gate_up_c: torch.Tensor, down_c: torch.Tensor, flags: int = 0,
                  y: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None) -> torch.Tensor:
    """si_selective_ffn: x [B][d], CSR active slots (offsets [B+1], idx [nnz]) -> y [B][d] f32."""
    dev = _dev(x)
    if x.dim() != 2:
        raise ValueError("x must be [B][d]")
    B, d = x.shape
    L = gate_up_c.shape[0]
    if gate_up_c.shape != (L, 2, d) or down_c.shape != (L, d):
        raise ValueError("compacted weights must be [L][2][d] and [L][d]")
    if offsets.dtype != torch.int32 or idx.dtype != torch.int32:
        raise ValueError("offsets and idx must be int32")
    if offsets.numel() < B + 1:
        raise ValueError("offsets needs B + 1 entries")
    nnz = idx.numel()
    if y is None:
        y = torch.empty((B, d), dtype=torch.float32, device=dev)
    need = selective_ffn_workspace(B, nnz, L, d, _dt(x), _dt(gate_up_c), flags)
    if workspace is None:
        workspace = _workspace(dev, need)
    st = load().si_selective_ffn(_ptr(x), _dt(x), B, d, _ptr(offsets), _ptr(idx), nnz,
                                 _ptr(gate_up_c), _ptr(down_c), L, _dt(gate_up_c), _ptr(y),
                                 _ptr(workspace), workspace.numel(), flags, _stream(dev))
    _check(st, "si_selective_ffn")
    return y


NOALLOC_SCRATCH_BYTES = 64 << 20


def selective_ffn_noalloc(x: torch.Tensor, offsets: torch.Tensor, idx: torch.Tensor,
                          gate_up_c: torch.Tensor, down_c: torch.Tensor, y: torch.Tensor,
                          flags: int = 0) -> torch.Tensor:
    """si_selective_ffn_noalloc: as selective_ffn, with the library's static device scratch as
    the workspace; y [B][d] float32 is the caller's. Nothing is allocated."""
    dev = _dev(x)
    if x.dim() != 2:
        raise ValueError("x must be [B][d]")
    B, d = x.shape
    L = gate_up_c.shape[0]
    if gate_up_c.shape != (L, 2, d) or down_c.shape != (L, d):
        raise ValueError("compacted weights must be [L][2][d] and [L][d]")
    if offsets.dtype != torch.int32 or idx.dtype != torch.int32:
        raise ValueError("offsets and idx must be int32")
    if offsets.numel() < B + 1:
        raise ValueError("offsets needs B + 1 entries")
    if y.shape != (B, d) or y.dtype != torch.float32:
        raise ValueError("y must be [B][d] float32")
    st = load().si_selective_ffn_noalloc(_ptr(x), _dt(x), B, d, _ptr(offsets), _ptr(idx),
                                         idx.numel(), _ptr(gate_up_c), _ptr(down_c), L,
                                         _dt(gate_up_c), _ptr(y), flags, _stream(dev))
    _check(st, "si_selective_ffn_noalloc")
    return y


def selective_ffn_resnorm(x_prev: torch.Tensor, y_prev: torch.Tensor, offsets: torch.Tensor,
                          idx: torch.Tensor, gate_up_c: torch.Tensor, down_c: torch.Tensor,
                          eps: float = 1e-5, flags: int = 0, x_out: torch.Tensor | None = None,
                          y: torch.Tensor | None = None,
                          workspace: torch.Tensor | None = None):
    """si_selective_ffn_resnorm: x = RMSNorm(x_prev + y_prev) -> x_out, then the selective FFN
    of x -> y. Returns (x_out, y)."""
    dev = _dev(x_prev)
    if x_prev.dim() != 2 or y_prev.shape != x_prev.shape or y_prev.dtype != torch.float32:
        raise ValueError("x_prev must be [B][d] and y_prev [B][d] float32")
    B, d = x_prev.shape
    L = gate_up_c.shape[0]
    if gate_up_c.shape != (L, 2, d) or down_c.shape != (L, d):
        raise ValueError("compacted weights must be [L][2][d] and [L][d]")
    if offsets.dtype != torch.int32 or idx.dtype != torch.int32:
        raise ValueError("offsets and idx must be int32")
    if offsets.numel() < B + 1:
        raise ValueError("offsets needs B + 1 entries")
    nnz = idx.numel()
    if x_out is None:
        x_out = torch.empty_like(x_prev)
    if y is None:
        y = torch.empty((B, d), dtype=torch.float32, device=dev)
    need = selective_ffn_workspace(B, nnz, L, d, _dt(x_prev), _dt(gate_up_c), flags)
    if workspace is None:
        workspace = _workspace(dev, need)
    st = load().si_selective_ffn_resnorm(_ptr(x_prev), _ptr(y_prev), float(eps), _ptr(x_out),
                                         _dt(x_prev), B, d, _ptr(offsets), _ptr(idx), nnz,
                                         _ptr(gate_up_c), _ptr(down_c), L, _dt(gate_up_c),
                                         _ptr(y), _ptr(workspace), workspace.numel(), flags,
                                         _stream(dev))
    _check(st, "si_selective_ffn_resnorm")
    return x_out, y


def set_timing_events(start: "torch.cuda.Event | None", stop: "torch.cuda.Event | None") -> None:
    """si_set_timing_events: bracket the main kernel of later selective_ffn calls on this thread.

    Events must have timing enabled and must already exist on the device (torch creates them
    lazily: record each once before passing it). Pass None, None to stop.
    """
    h0 = None if start is None else start.cuda_event
    h1 = None if stop is None else stop.cuda_event
    _check(load().si_set_timing_events(h0, h1), "si_set_timing_events")


def ceiling_stream(buf: torch.Tensor, blocks: int, sink: torch.Tensor) -> None:
    """si_ceiling_stream (measurement only): read the whole of buf contiguously."""
    dev = _dev(buf)
    if sink.dtype != torch.int32 or sink.numel() < blocks * 512:
        raise ValueError("sink must hold blocks * 512 int32 words")
    st = load().si_ceiling_stream(_ptr(buf), buf.numel() * buf.element_size(), blocks,
                                  _ptr(sink), _stream(dev))
    _check(st, "si_ceiling_stream")


def ceiling_gather(gate_up_c: torch.Tensor, down_c: torch.Tensor, idx: torch.Tensor, P: int,
                   sink: torch.Tensor) -> None:
    """si_ceiling_gather (measurement only): load the gate, up and down rows of the slots idx
    in the per-token path's pattern, without its arithmetic."""
    dev = _dev(gate_up_c)
    L, _, d = gate_up_c.shape
    if down_c.shape != (L, d) or idx.dtype != torch.int32:
        raise ValueError("compacted weights [L][2][d], [L][d] and int32 slots expected")
    if sink.dtype != torch.int32 or sink.numel() < P * 512:
        raise ValueError("sink must hold P * 512 int32 words")
    st = load().si_ceiling_gather(_ptr(gate_up_c), _ptr(down_c), L, d, _dt(gate_up_c),
                                  _ptr(idx), idx.numel(), P, _ptr(sink), _stream(dev))
    _check(st, "si_ceiling_gather")


def residual_rmsnorm(x: torch.Tensor, y: torch.Tensor, eps: float = 1e-5,
                     out: torch.Tensor | None = None) -> torch.Tensor:
    """si_residual_rmsnorm: RMSNorm(x + y), unit gain, stored in x's dtype."""
    dev = _dev(x)
    B, d = x.shape
    if out is None:
        out = torch.empty_like(x)
    st = load().si_residual_rmsnorm(_ptr(x), _dt(x), _ptr(y), B, d, float(eps), _ptr(out),
                                    _stream(dev))
    _check(st, "si_residual_rmsnorm")
    return out


def dynamic_set(x: torch.Tensor, gate_up_c: torch.Tensor, static_slots: torch.Tensor,
                alpha: int, n_total: int, workspace: torch.Tensor | None = None,
                out: torch.Tensor | None = None, counts: torch.Tensor | None = None,
                mode: str = "abs"):
    """si_dynamic_set: a prompt x [T][d] over a compacted layer -> (active slots [n_total]
    ascending, counts [L]: how many of the T per-token top-alpha lists hold each slot). The
    per-token ranking key is |a| (mode "abs") or a ("raw")."""
    dev = _dev(gate_up_c)
    T, d = x.shape
    L = gate_up_c.shape[0]
    if gate_up_c.shape != (L, 2, d):
        raise ValueError("gate_up_c must be [L][2][d]")
    if static_slots.dtype != torch.int32:
        raise ValueError("static_slots must be int32")
    if out is None:
        out = torch.empty(n_total, dtype=torch.int32, device=dev)
    if counts is None:
        counts = torch.empty(L, dtype=torch.int32, device=dev)
    if out.numel() < n_total or counts.numel() < L:
        raise ValueError("out needs n_total entries and counts L")
    lib = load()
    need = int(lib.si_dynamic_set_workspace(T, L, alpha, n_total))
    if workspace is None:
        workspace = _workspace(dev, need)
    st = lib.si_dynamic_set(_ptr(x), _dt(x), T, d, _ptr(gate_up_c), L, _dt(gate_up_c),
                            _ptr(static_slots), static_slots.numel(), alpha, n_total,
                            _MODES[mode], _ptr(out), _ptr(counts), _ptr(workspace),
                            workspace.numel(), _stream(dev))
    _check(st, "si_dynamic_set")
    return out, counts


def profile_scores(x: torch.Tensor, gate_up: torch.Tensor, scores: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None) -> torch.Tensor:
    """si_profile_scores: scores [N] float64 += sum over the tokens x [T][d] of |a_n| (Eq. 1);
    a new zeroed scores tensor when none is given."""
    dev = _dev(gate_up)
    T, d = x.shape
    N = gate_up.shape[0]
    if gate_up.shape != (N, 2, d):
        raise ValueError("gate_up must be [N][2][d]")
    if scores is None:
        scores = torch.zeros(N, dtype=torch.float64, device=dev)
    if scores.dtype != torch.float64 or scores.numel() != N:
        raise ValueError("scores must be a float64 tensor of N entries")
    lib = load()
    need = int(lib.si_profile_scores_workspace(T, N, d, _dt(x), _dt(gate_up)))
    if workspace is None:
        workspace = _workspace(dev, need)
    st = lib.si_profile_scores(_ptr(x), _dt(x), T, d, _ptr(gate_up), N, _dt(gate_up),
                               _ptr(scores), _ptr(workspace), workspace.numel(), _stream(dev))
    _check(st, "si_profile_scores")
    return scores


def merge_scores(scores: torch.Tensor, tokens) -> torch.Tensor:
    """si_merge_scores: float64 scores [F][N] with token counts [F] (host ints) -> sum of
    s_f / T_f (float64)."""
    import ctypes

    dev = _dev(scores)
    if scores.dtype != torch.float64 or scores.dim() != 2:
        raise ValueError("scores must be a 2-D float64 tensor")
    F, N = scores.shape
    if len(tokens) != F:
        raise ValueError("one token count per score file")
    toks = (ctypes.c_int64 * F)(*[int(t) for t in tokens])
    out = torch.empty(N, dtype=torch.float64, device=dev)
    st = load().si_merge_scores(_ptr(scores), ctypes.cast(toks, ctypes.c_void_p), F, N,
                                _ptr(out), _stream(dev))
    _check(st, "si_merge_scores")
    return out


def rank_neurons(scores: torch.Tensor) -> torch.Tensor:
    """si_rank_neurons: neuron indices by decreasing float64 score (ties to the lower index)."""
    dev = _dev(scores)
    if scores.dtype != torch.float64:
        raise ValueError("scores must be float64")
    order = torch.empty(scores.numel(), dtype=torch.int32, device=dev)
    st = load().si_rank_neurons(_ptr(scores), scores.numel(), _ptr(order), _stream(dev))
    _check(st, "si_rank_neurons")
    return order


def build_loaded_set(task_rank, model_rank, n_base: int, n_loaded: int):
    """si_build_loaded_set (host only): base = task_rank[:n_base], then model-ranked neurons
    not yet chosen, until n_loaded. Rankings and result are int32 NumPy arrays."""
    import numpy as np

    t = np.ascontiguousarray(task_rank, dtype=np.int32)
    m = np.ascontiguousarray(model_rank, dtype=np.int32)
    if t.shape != m.shape or t.ndim != 1:
        raise ValueError("rankings must be 1-D and of one length")
    out = np.empty(max(int(n_loaded), 0), dtype=np.int32)
    st = load().si_build_loaded_set(t.ctypes.data, m.ctypes.data, t.size, n_base, n_loaded,
                                    out.ctypes.data if out.size else None)
    _check(st, "si_build_loaded_set")
    return out


def selective_layers(n_layers: int, first: int = 5, last: int = -2):
    """si_selective_layers (host only): boolean mask of the layers whose FFN is loaded and
    computed selectively, first <= i < n_layers + last (Table 1: 5 and -2)."""
    import numpy as np

    mask = np.zeros(max(int(n_layers), 0), dtype=np.uint8)
    cnt = ctypes.c_int64(0)
    st = load().si_selective_layers(n_layers, first, last,
                                    mask.ctypes.data if mask.size else None, ctypes.byref(cnt))
    _check(st, "si_selective_layers")
    assert int(cnt.value) == int(mask.sum())
    return mask.astype(bool)


def load_selected(w_gate, w_up, w_down, loaded, device=None) -> CompactLayer:
    """si_load_selected: full layer in HOST memory (NumPy arrays or memory maps; bf16 as uint16
    bit patterns or float32) -> compacted layer on the device, moving only the loaded slices."""
    import numpy as np

    dev = torch.device(device or "cuda")
    wg, wu, wd = (np.asarray(w) for w in (w_gate, w_up, w_down))
    for w in (wg, wu, wd):
        if not w.flags.c_contiguous:
            raise ValueError("weights must be C-contiguous")
    N, d = wg.shape
    if wu.shape != (N, d) or wd.shape != (d, N) or wg.dtype != wu.dtype or wg.dtype != wd.dtype:
        raise ValueError("expect W_gate, W_up [N][d] and W_down [d][N] of one dtype")
    if wg.dtype == np.uint16:
        wdt, tdt = BF16, torch.bfloat16
    elif wg.dtype == np.float16:
        wdt, tdt = F16, torch.float16
    elif wg.dtype == np.float32:
        wdt, tdt = F32, torch.float32
    else:
        raise TypeError(f"unsupported dtype {wg.dtype}")
    ids = np.ascontiguousarray(loaded, dtype=np.int32).reshape(-1)
    L = ids.size
    gu = torch.empty((L, 2, d), dtype=tdt, device=dev)
    dc = torch.empty((L, d), dtype=tdt, device=dev)
    s2o = torch.empty(L, dtype=torch.int32, device=dev)
    o2s = torch.empty(N, dtype=torch.int32, device=dev)
    st = load().si_load_selected(wg.ctypes.data, wu.ctypes.data, wd.ctypes.data, N, d, wdt,
                                 ids.ctypes.data, L, _ptr(gu), _ptr(dc), _ptr(s2o), _ptr(o2s),
                                 _stream(dev))
    _check(st, "si_load_selected")
    return CompactLayer(gu, dc, s2o, o2s)
