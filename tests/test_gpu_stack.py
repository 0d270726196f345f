"""GPU parity of the 16-layer LLaDA-MoE stack (8 x 1024 tokens) against the oracle,
layer by layer with teacher forcing.

One count vector is computed by the first layer's budget and reused by every layer
(k shared across the forward's MoE layers, Section 3.3); between layers a fixed
random residual stands in for attention: h_{l+1} = bf16(h_l + MoE_l(h_l) + rho_l).
Each checked layer is compared on sampled tokens, given the GPU's own input h_l
and the GPU's fp32 router scores (selection pinned), so errors do not compound.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from gpu_common import layer_tolerance_check, note, oracle_budget, require_gpu
from synth import make_fuzz_workload, make_workload
from synth.device import bf16_bits, state_tensors, to_device

pytestmark = pytest.mark.gpu

NAME = "lladamoe_stack16_t8192"
CHECKED = (0, 1, 7, 15)
N_SAMPLE = 128


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def test_stack16_teacher_forced(torch):
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    w = make_workload(NAME)
    L = w.n_layers
    assert L == 16 and w.T == 8192
    layers = []
    for l in range(L):
        layers.append(ExpertWeights(w_gate=to_device(w.w_gate(l)), w_up=to_device(w.w_up(l)),
                                    w_down=to_device(w.w_down(l)),
                                    w_router=to_device(w.w_router(l))))
        w.release(l)
    res = [to_device(w.residual(l)) for l in range(L)]
    lay = MoELayer(w.T, w.d, layers[0], w.params)
    state = TokenState(**state_tensors(w))
    h = [to_device(w.h)]
    k0 = None
    saved = {}
    for l in range(L):
        lay.w = layers[l]
        out = torch.empty_like(h[0])
        lay.forward(h[l], state if l == 0 else None, k_in=k0, residual_a=h[l], residual_b=res[l],
                    out=out)
        if l == 0:
            k0 = lay.k.clone()
            pairs0 = int(lay.pairs.item())
        if l in CHECKED:
            saved[l] = lay.logits.cpu().numpy().astype(np.float64)
        h.append(out)
    torch.cuda.synchronize()
    note(f"{NAME}: 16 layers run")

    k = k0.cpu().numpy()
    ref_b = oracle_budget(w)
    assert np.array_equal(k, ref_b.k)
    assert pairs0 == ref_b.pairs
    toks = np.sort(np.random.default_rng(3).choice(w.T, N_SAMPLE, replace=False))
    for l in CHECKED:
        h_in = bf16_bits(h[l])
        got = oracle.bf16_to_f64(bf16_bits(h[l + 1])[toks])
        r = oracle.router_scores(h_in[toks], w.w_router(l))
        assert np.all(np.abs(saved[l][toks] - r).max(axis=1) <= 1e-4 * np.abs(r).max(axis=1))
        route = oracle.topk_route(saved[l], k, w.norm_topk)
        moe = oracle.moe_layer(h_in, route, lambda e, l=l: w.expert_weights(l, e), w.E,
                               tokens=toks)
        ref = moe + oracle.bf16_to_f64(h_in[toks]) + oracle.bf16_to_f64(w.residual(l)[toks])
        layer_tolerance_check(got, ref, f"{NAME} layer {l} (teacher forced)")
    # end-to-end drift is reported, not asserted: the stack compounds 16 roundings
    h_last = oracle.bf16_to_f64(bf16_bits(h[L])[toks])
    note(f"{NAME}: |h_16| rms {np.sqrt((h_last ** 2).mean()):.3f}")


def test_per_layer_counts(torch):
    # counts given per layer as rows of an [L, T] array (a per-layer allocation,
    # Section 3.3's generalisation); each layer is checked against the oracle with
    # its own row, teacher forced
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer
    w = make_fuzz_workload(321, T=700, d=256, E=16, f=128, k_max=6)
    L = 3
    k_rows = np.random.default_rng(9).integers(0, w.params.k_max + 1, (L, w.T)).astype(np.int32)
    k_dev = to_device(k_rows)
    lay = None
    h = [to_device(w.h)]
    logits = []
    res = [to_device(w.residual(l)) for l in range(L)]
    for l in range(L):
        ew = ExpertWeights(w_gate=to_device(w.w_gate(l)), w_up=to_device(w.w_up(l)),
                           w_down=to_device(w.w_down(l)), w_router=to_device(w.w_router(l)))
        if lay is None:
            lay = MoELayer(w.T, w.d, ew, w.params)
        lay.w = ew
        out = torch.empty_like(h[0])
        lay.forward(h[l], k_in=k_dev[l], residual_a=h[l], residual_b=res[l], out=out)
        assert int(lay.pairs.item()) == int(k_rows[l].sum())
        logits.append(lay.logits.cpu().numpy().astype(np.float64))
        h.append(out)
    torch.cuda.synchronize()
    for l in range(L):
        h_in = bf16_bits(h[l])
        route = oracle.topk_route(logits[l], k_rows[l])
        wg, wu, wd = w.w_gate(l), w.w_up(l), w.w_down(l)
        ref = (oracle.moe_layer(h_in, route, lambda e: (wg[e], wu[e], wd[e]), w.E)
               + oracle.bf16_to_f64(h_in) + oracle.bf16_to_f64(w.residual(l)))
        layer_tolerance_check(oracle.bf16_to_f64(bf16_bits(h[l + 1])), ref, f"per-layer counts, layer {l}")
