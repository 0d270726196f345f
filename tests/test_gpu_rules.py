"""GPU parity of the score-derived count rules (Top-p and Expert-Threshold
Routing, Appendix B) against the oracle, alone and inside the fused layer.

Both sides decide in fp64 from the same fp32 scores; they may differ only where
the routing mass sits within a relative 1e-12 of the threshold (exp and the softmax
sum are not bitwise alike).  Such tokens are counted; for them the GPU's count must
be one of the two counts the boundary allows."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from gpu_common import layer_tolerance_check, note, require_gpu
from synth import make_fuzz_workload, make_workload
from synth.device import bf16_bits, state_tensors, to_device

pytestmark = pytest.mark.gpu

MARGIN = 1e-12
# thresholds the paper calibrates (low / high compute) for the two model families
PAPER_P = [0.15, 0.20, 0.25, 0.325]
PAPER_TAU = [0.0215, 0.0190, 0.0270, 0.0220]


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _ranked(r):
    E = r.shape[1]
    prob = oracle.router_probs(r)
    order = np.lexsort((np.broadcast_to(np.arange(E), r.shape), -(r + 0.0)), axis=1)
    return np.take_along_axis(prob, order, axis=1)


def _fragile_topp(r, p, k_min, k_max):
    """Tokens whose Top-p count could flip under a last-ulp change of the mass: a
    prefix of at most k_max experts whose mass is within a relative 1e-12 of p."""
    pp = float(np.float32(p))
    cum = np.cumsum(_ranked(r), axis=1)[:, :max(k_max, 1)]
    return np.any(np.abs(cum - pp) <= MARGIN * pp, axis=1)


def _fragile_thr(r, tau):
    prob = oracle.router_probs(r)
    t = float(np.float32(tau))
    return np.any(np.abs(prob - t) <= MARGIN * np.maximum(prob, t), axis=1)


def _check_counts(got, ref, fragile, what):
    assert np.array_equal(got[~fragile], ref[~fragile]), what
    # at a boundary the count may land on either side of it
    assert np.all(np.abs(got[fragile] - ref[fragile]) <= 1), what
    note(f"{what}: {int(fragile.sum())} boundary token(s)")


def _gpu_rule(torch, r32, rule, thr, k_min, k_max):
    from paper_2608_01784_amd import _lib
    logits = torch.from_numpy(r32).cuda()
    k = torch.empty(r32.shape[0], dtype=torch.int32, device="cuda")
    pairs = torch.empty(1, dtype=torch.int32, device="cuda")
    _lib.reflex_count_rule(logits, rule, thr, k_min, k_max, k, pairs)
    torch.cuda.synchronize()
    return k.cpu().numpy(), int(pairs.item())


def _logits(seed, T, E, scale, ties=False):
    rng = np.random.default_rng(seed)
    r = (rng.standard_normal((T, E)) * scale).astype(np.float32)
    if ties:
        r = np.round(r * 4) / 4          # many exactly equal scores
        r[:, :2] = 0.0
        r[0] = -0.0
    return r


CASES = [(0, 777, 64, 0.9, False), (1, 512, 256, 1.2, False), (2, 300, 8, 2.0, True),
         (3, 129, 1, 1.0, False), (4, 1000, 255, 0.3, False), (5, 64, 64, 6.0, True)]


@pytest.mark.parametrize("seed,T,E,scale,ties", CASES)
@pytest.mark.parametrize("p", PAPER_P + [1.0])
def test_top_p_counts_bit_exact(torch, seed, T, E, scale, ties, p):
    from paper_2608_01784_amd import _lib
    r = _logits(seed, T, E, scale, ties)
    k_min, k_max = (1, min(12, E)) if E > 1 else (0, 1)
    got, pairs = _gpu_rule(torch, r, _lib.RULE_TOP_P, p, k_min, k_max)
    ref, _ = oracle.topp_counts(r.astype(np.float64), p, k_min, k_max)
    fragile = _fragile_topp(r.astype(np.float64), p, k_min, k_max)
    _check_counts(got, ref, fragile, f"top-p {p} E={E}")
    assert pairs == int(got.sum())


@pytest.mark.parametrize("seed,T,E,scale,ties", CASES)
@pytest.mark.parametrize("tau", PAPER_TAU + [0.0, 0.5])
def test_threshold_counts_bit_exact(torch, seed, T, E, scale, ties, tau):
    from paper_2608_01784_amd import _lib
    r = _logits(seed, T, E, scale, ties)
    k_min, k_max = (1, min(12, E)) if E > 1 else (0, 1)
    got, pairs = _gpu_rule(torch, r, _lib.RULE_THRESHOLD, tau, k_min, k_max)
    ref = oracle.threshold_counts(r.astype(np.float64), tau, k_min, k_max)
    fragile = _fragile_thr(r.astype(np.float64), tau)
    _check_counts(got, ref, fragile, f"threshold {tau} E={E}")
    assert pairs == int(got.sum())


def test_rule_bounds_from_k_min_zero(torch):
    # k_min = 0 keeps a 0 count possible for the threshold rule (no expert above tau)
    from paper_2608_01784_amd import _lib
    r = np.zeros((10, 16), np.float32)               # masses 1/16 = 0.0625
    got, pairs = _gpu_rule(torch, r, _lib.RULE_THRESHOLD, 0.1, 0, 8)
    assert np.all(got == 0) and pairs == 0
    got, _ = _gpu_rule(torch, r, _lib.RULE_THRESHOLD, 0.05, 0, 8)
    assert np.all(got == 8)
    got, _ = _gpu_rule(torch, r, _lib.RULE_TOP_P, 0.25, 0, 8)       # 4 x 1/16 = 0.25
    assert np.all(got == 4)


@pytest.mark.parametrize("name,rule,thr", [("tiny_t128_e8", 1, 0.5), ("tiny_t128_e8", 2, 0.1),
                                           ("lladamoe_t1024_e64", 1, 0.20),
                                           ("lladamoe_t1024_e64", 2, 0.0190),
                                           ("llada2mini_t4096_e256", 1, 0.325),
                                           ("llada2mini_t4096_e256", 2, 0.0220)])
def test_fused_layer_with_count_rule(torch, name, rule, thr):
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    w = make_workload(name)
    params = w.params.replace(k_min=1, k_max=min(12, w.E))
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()),
          "router_bias": None if w.router_bias is None else to_device(w.router_bias)}
    sh = w.shared_weights()
    if sh is not None:
        dw["ws_gate"], dw["ws_up"], dw["ws_down"] = (to_device(x) for x in sh)
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), params, k_rule=rule, k_threshold=thr)
    out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), TokenState(**state_tensors(w)))))
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    logits = lay.logits.cpu().numpy().astype(np.float64)
    if rule == 1:
        ref_k, _ = oracle.topp_counts(logits, thr, params.k_min, params.k_max)
        fragile = _fragile_topp(logits, thr, params.k_min, params.k_max)
    else:
        ref_k = oracle.threshold_counts(logits, thr, params.k_min, params.k_max)
        fragile = _fragile_thr(logits, thr)
    _check_counts(k, ref_k, fragile, f"{name} rule {rule}")
    assert int(lay.pairs.item()) == int(k.sum())
    note(f"{name} rule {rule} thr {thr}: AvgK {k.mean():.3f}")
    toks = None if w.T <= 1200 else np.sort(np.random.default_rng(1).choice(w.T, 256, replace=False))
    route = oracle.topk_route(logits, k)
    wg, wu, wd = w.w_gate(), w.w_up(), w.w_down()
    ref = oracle.moe_layer(w.h, route, lambda e: (wg[e], wu[e], wd[e]), w.E, shared=sh, tokens=toks)
    layer_tolerance_check(out if toks is None else out[toks], ref, f"{name} rule {rule}")
