"""Copies seeded workloads to a torch device (data movement only)."""
from __future__ import annotations

import numpy as np
import torch

from . import Workload


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns -> torch.bfloat16 tensor on `device`."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def upload_layers(w: Workload, layers, device, keep_host: bool = False, threads: int | None = None):
    """Generate K, V (bf16 [rows, d]) and Q (fp32 [B, Hq, W, d]) for `layers`.

    Returns (dev, host): dev maps 'K', 'V', 'Q' to {layer: tensor}; host holds
    the numpy arrays when keep_host is set (else None)."""
    dev = {"K": {}, "V": {}, "Q": {}}
    host = {"K": {}, "V": {}, "Q": {}} if keep_host else None
    for l in layers:
        K = w.kv_layer("K", l, threads=threads)
        V = w.kv_layer("V", l, threads=threads)
        Q = w.q_layer(l)
        dev["K"][l] = bf16_tensor(K, device)
        dev["V"][l] = bf16_tensor(V, device)
        dev["Q"][l] = torch.from_numpy(Q).to(device)
        if keep_host:
            host["K"][l], host["V"][l], host["Q"][l] = K, V, Q
    return dev, host


def to_host_bf16(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 device tensor -> uint16 bit patterns on the host."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
