"""A multi-forward decoding run on the GPU: each denoising forward runs the fused
variable-count MoE layer(s) on the current decoding state, then the state kernel
commits positions by the confidence threshold (Eq. (1)), shifts the confidence
history and advances blocks.  The confidences are inputs (in a real model they
come from the LM head of the same forward).

This is bookkeeping around the library's entry points; every step runs in HIP
kernels.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

from . import _lib
from .layer import MoELayer, TokenState


@dataclass
class TrajectoryStats:
    forwards: int = 0
    pairs: List[int] = field(default_factory=list)      # P of each forward
    masked_left: List[int] = field(default_factory=list)

    @property
    def total_pairs(self) -> int:
        return int(sum(self.pairs))


def run_trajectory(layer: MoELayer, h, state: TokenState, confidence: Callable[[int], object],
                   theta: float, min_commit: int = 0, max_forwards: int = 10_000,
                   on_forward: Optional[Callable[[int, TokenState], None]] = None,
                   stream=None) -> TrajectoryStats:
    """Run forwards until every target position is committed (or max_forwards).

    confidence(t) returns the [T] float32 device tensor of forward t's
    confidences.  on_forward(t, state), if given, is called after each layer
    forward and before the state update (the state still describes forward t)."""
    import torch
    stats = TrajectoryStats()
    remaining = torch.empty(state.active_block.shape[0], dtype=torch.int32,
                            device=state.active_block.device)
    for t in range(max_forwards):
        layer.forward(h, state, stream=stream)
        if on_forward is not None:
            on_forward(t, state)
        conf_t = confidence(t)
        _lib.reflex_advance_state(conf_t, state.block_idx, state.seq_offsets, theta, min_commit,
                                  state.masked, state.hist_len, state.conf_prev1, state.conf_prev2,
                                  state.active_block, remaining, stream=stream)
        stats.forwards += 1
        stats.pairs.append(int(layer.pairs.item()))
        left = int(remaining.sum().item())
        stats.masked_left.append(left)
        if left == 0:
            break
    return stats
