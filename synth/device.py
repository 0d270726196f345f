"""Copy synthetic workloads to device memory as torch tensors (no computation)."""
from __future__ import annotations

import numpy as np


def to_device(a: np.ndarray, device="cuda"):
    """numpy -> torch on ``device``; uint16 arrays (bf16 bit patterns) become bfloat16."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def state_tensors(w, device="cuda"):
    """Token-state arrays of a workload: dict of device tensors."""
    return {n: to_device(getattr(w, n), device) for n in
            ("block_idx", "masked", "hist_len", "conf_prev1", "conf_prev2", "seq_offsets",
             "active_block")}


def weight_tensors(w, layer: int = 0, device="cuda"):
    """Expert, router and shared-expert weights of one layer: dict of device tensors."""
    d = {"w_gate": to_device(w.w_gate(layer), device), "w_up": to_device(w.w_up(layer), device),
         "w_down": to_device(w.w_down(layer), device), "w_router": to_device(w.w_router(layer), device),
         "router_bias": None if w.router_bias is None else to_device(w.router_bias, device)}
    sh = w.shared_weights(layer)
    if sh is not None:
        d["ws_gate"], d["ws_up"], d["ws_down"] = (to_device(x, device) for x in sh)
    return d


def bf16_bits(t) -> np.ndarray:
    """Device bfloat16 tensor -> numpy uint16 bit patterns."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
