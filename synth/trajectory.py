"""Seeded inputs of a synthetic multi-forward decoding trajectory.

A trajectory starts with every target position masked and block 1 active in
every sequence.  The confidence the model would report at each position on
forward t is drawn here, independently of the decoding state: every position has
a seeded starting confidence and growth rate, so its confidence rises over
forwards (with small per-forward noise) until it crosses the commitment
threshold.  Nothing here computes any step of the method.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .workloads import Workload

_TAG_TRAJ = 21


def generation_start(w: Workload) -> Dict[str, np.ndarray]:
    """The decoding state before the first forward: prompt committed (block 0),
    all target positions masked, no confidence history, block 1 active."""
    T = len(w.block_idx)
    return {
        "block_idx": w.block_idx.copy(),
        "masked": (w.block_idx > 0).astype(np.uint8),
        "hist_len": np.zeros(T, np.int8),
        "conf_prev1": np.zeros(T, np.float32),
        "conf_prev2": np.zeros(T, np.float32),
        "seq_offsets": w.seq_offsets.copy(),
        "active_block": np.ones(len(w.active_block), np.int32),
    }


def forward_confidence(seed: int, t: int, T: int) -> np.ndarray:
    """c_i^t for every position i on forward t (float32; only masked positions
    are read): clip(base_i + rate_i * t + noise_{i,t}, 0, 1), base ~ Beta(2, 5),
    rate ~ U(0.03, 0.2), noise ~ N(0, 0.02^2)."""
    rng = np.random.default_rng([seed, _TAG_TRAJ])
    base = rng.beta(2.0, 5.0, T)
    rate = rng.uniform(0.03, 0.2, T)
    noise = np.random.default_rng([seed, _TAG_TRAJ, t]).normal(0.0, 0.02, T)
    return np.clip(base + rate * t + noise, 0.0, 1.0).astype(np.float32)
