"""Helpers shared by the GPU tests: host arrays -> device tensors, and the
parity metric.  Inputs come only from paper_2407_00066_amd.workloads; expected
values only from the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch


def dev(a: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 arrays are bf16 bit patterns; float32/int32 copy as they are."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def host(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return (t.view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return t.numpy().astype(np.float64)


def row_rel_err(y: np.ndarray, ref: np.ndarray) -> float:
    """max over tokens of  max_o |y - ref| / max_o |ref|  (per-token inf-norm
    relative error)."""
    if y.size == 0:
        return 0.0
    num = np.abs(y - ref).max(axis=1)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return float((num / den).max())


TOL = {"f32": 1e-5, "bf16": 2e-2}


def say(msg: str):
    """Name the case before a GPU step (flushed, so it survives a crash)."""
    print(msg, file=sys.stderr, flush=True)
