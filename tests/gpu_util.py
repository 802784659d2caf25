"""Helpers for GPU tests: storage arrays <-> device tensors, error metrics, progress lines."""
from __future__ import annotations

import sys

import numpy as np
import torch


def dev_tensor(a: np.ndarray, device="cuda:0") -> torch.Tensor:
    """uint16 (bf16 bits) -> bfloat16 tensor; float32 / int32 as is."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def host_array(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    n = np.linalg.norm(ref)
    if n == 0.0:
        return float(np.linalg.norm(got))
    return float(np.linalg.norm(got - ref) / n)


def max_rel_l2(got2d, ref2d) -> float:
    return max(rel_l2(g, r) for g, r in zip(got2d, ref2d)) if len(ref2d) else 0.0


def say(msg: str) -> None:
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()
