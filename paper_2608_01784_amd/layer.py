"""The fused variable-K MoE layer (``reflex_moe_forward``) from torch tensors.

This module only allocates device buffers with torch and fills the C argument
struct; every step of the layer runs in the HIP kernels of libreflex.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import torch

from . import _lib


@dataclass
class TokenState:
    """Per-token decoding state of one denoising forward (device tensors).

    block_idx int32 [T] (prompt = 0), masked uint8 [T], hist_len int8 [T],
    conf_prev1 / conf_prev2 float32 [T], seq_offsets int32 [B+1], active_block int32 [B].
    """
    block_idx: torch.Tensor
    masked: torch.Tensor
    hist_len: torch.Tensor
    conf_prev1: torch.Tensor
    conf_prev2: torch.Tensor
    seq_offsets: torch.Tensor
    active_block: torch.Tensor


@dataclass
class ExpertWeights:
    """bf16 expert weights: w_gate, w_up [E, f, d]; w_down [E, d, f]; router fp32 [E, d];
    optional shared expert (ws_gate, ws_up [fs, d], ws_down [d, fs])."""
    w_gate: torch.Tensor
    w_up: torch.Tensor
    w_down: torch.Tensor
    w_router: torch.Tensor
    router_bias: Optional[torch.Tensor] = None
    ws_gate: Optional[torch.Tensor] = None
    ws_up: Optional[torch.Tensor] = None
    ws_down: Optional[torch.Tensor] = None

    @property
    def E(self):
        return self.w_router.shape[0]

    @property
    def f(self):
        return self.w_gate.shape[1]

    @property
    def f_shared(self):
        return 0 if self.ws_gate is None else self.ws_gate.shape[0]


class MoELayer:
    """Holds the workspace and output buffers for repeated fused forwards of one shape."""

    def __init__(self, T: int, d: int, weights: ExpertWeights, params, uniform_k: int = 0,
                 norm_topk: int = 1, k_rule: int = 0, k_threshold: float = 0.0, device="cuda"):
        """k_rule: 0 = REFLEX budget; 1 = Top-p, 2 = Expert-Threshold with k_threshold
        (counts bounded by params.k_min, params.k_max)."""
        self.T, self.d, self.w = T, d, weights
        self.params = params
        self.uniform_k = int(uniform_k)
        self.norm_topk = int(norm_topk)
        self.k_rule, self.k_threshold = int(k_rule), float(k_threshold)
        self.kcap = self.uniform_k if self.uniform_k > 0 else int(params.k_max)
        nbytes = _lib.reflex_workspace_size(T, weights.E, d, weights.f, weights.f_shared, self.kcap)
        if nbytes == 0 and T > 0:
            raise ValueError("unsupported layer shape")
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.out = torch.empty((T, d), dtype=torch.bfloat16, device=device)
        self.k = torch.empty(T, dtype=torch.int32, device=device)
        self.pairs = torch.empty(1, dtype=torch.int32, device=device)
        self.logits = torch.empty((T, weights.E), dtype=torch.float32, device=device)

    def args(self, h: torch.Tensor, state: Optional[TokenState] = None,
             k_in: Optional[torch.Tensor] = None, residual_a=None, residual_b=None,
             out: Optional[torch.Tensor] = None) -> _lib.MoeArgsC:
        w = self.w
        a = _lib.MoeArgsC()
        a.T, a.d, a.E, a.f, a.f_shared = self.T, self.d, w.E, w.f, w.f_shared
        a.norm_topk, a.uniform_k = self.norm_topk, self.uniform_k
        a.k_rule, a.k_threshold = self.k_rule, self.k_threshold
        P = _lib.ptr
        a.h, a.w_gate, a.w_up, a.w_down = P(h), P(w.w_gate), P(w.w_up), P(w.w_down)
        a.ws_gate, a.ws_up, a.ws_down = P(w.ws_gate), P(w.ws_up), P(w.ws_down)
        a.w_router, a.router_bias = P(w.w_router), P(w.router_bias)
        if state is not None:
            a.B = state.active_block.shape[0]
            a.block_idx, a.seq_offsets, a.active_block = (P(state.block_idx), P(state.seq_offsets),
                                                          P(state.active_block))
            a.masked, a.hist_len = P(state.masked), P(state.hist_len)
            a.conf_prev1, a.conf_prev2 = P(state.conf_prev1), P(state.conf_prev2)
        a.k_in = P(k_in)
        a.residual_a, a.residual_b = P(residual_a), P(residual_b)
        a.params = _lib.alloc_params(self.params)
        a.out = P(self.out if out is None else out)
        a.k_out, a.pairs_out, a.logits_out = P(self.k), P(self.pairs), P(self.logits)
        return a

    def forward(self, h, state=None, k_in=None, residual_a=None, residual_b=None, out=None,
                stream=None) -> torch.Tensor:
        args = self.args(h, state, k_in, residual_a, residual_b, out)
        _lib.reflex_moe_forward(args, self.ws, stream)
        return self.out if out is None else out
