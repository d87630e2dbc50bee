"""Copies seeded workloads to a torch device (data movement only)."""
from __future__ import annotations

import numpy as np
import torch

from . import Workload


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns -> torch.bfloat16 tensor on `device`."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def upload_layers(w: Workload, layers, device, keep_host: bool = False, threads: int | None = None,
                  prefill: bool = False, host_only: bool = False):
    """Generate K, V (bf16 [rows, d]) and Q (fp32 [B, Hq, W, d]) for `layers`;
    with `prefill`, Q is the query of every prefill token (fp32
    [sum_b Hq*(n_b+W), d]) and 'KT' holds the text keys (bf16 [B, Hkv, W, d]).

    Returns (dev, host): dev maps 'K', 'V', 'Q' (and 'KT') to {layer: tensor};
    host holds the numpy arrays when keep_host is set (else None).  With
    host_only nothing is copied to a device (dev maps to empty dicts)."""
    roles = ("K", "V", "Q", "KT") if prefill else ("K", "V", "Q")
    dev = {r: {} for r in roles}
    host = {r: {} for r in roles} if keep_host else None
    for l in layers:
        arrs = {"K": w.kv_layer("K", l, threads=threads), "V": w.kv_layer("V", l, threads=threads),
                "Q": w.qall_layer(l) if prefill else w.q_layer(l)}
        if prefill:
            arrs["KT"] = w.ktext_layer(l)
        for r, a in arrs.items():
            if not host_only:
                dev[r][l] = torch.from_numpy(a).to(device) if r == "Q" else bf16_tensor(a, device)
            if keep_host:
                host[r][l] = a
    return dev, host


def to_host_bf16(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 device tensor -> uint16 bit patterns on the host."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
