"""reflex_moe_forward_noalloc (the entry point for callers that cannot allocate) against
reflex_moe_forward on the same inputs, through the C ABI.  Both run the same kernels on
the same data, so every output must match bit for bit; two calls in a row, the second on
a smaller layer, check that the shared scratch carries nothing from one call to the next."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_common import note, require_gpu
from synth import make_workload
from synth.device import bf16_bits, state_tensors, to_device, weight_tensors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _both(torch, w, T, state, h, weights, uniform_k=0):
    """Outputs (out bits, k, P, logits) of the allocating and the allocation-free entry
    points for the first T tokens of workload w."""
    from paper_2608_01784_amd import _lib
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    lay = MoELayer(T, w.d, ExpertWeights(**weights), w.params, uniform_k=uniform_k)
    st = TokenState(**state)
    res = []
    for noalloc in (False, True):
        # fresh outputs filled with garbage, so nothing is inherited from the other run
        out = torch.full((T, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lay.k.fill_(-7)
        lay.pairs.fill_(-7)
        lay.logits.fill_(float("nan"))
        args = lay.args(h, st, out=out)
        if noalloc:
            _lib.reflex_moe_forward_noalloc(args)
        else:
            _lib.reflex_moe_forward(args, lay.ws)
        torch.cuda.synchronize()
        res.append((bf16_bits(out), lay.k.cpu().numpy().copy(), int(lay.pairs.item()),
                    lay.logits.cpu().numpy().copy()))
    return res


def _assert_same(a, b, what):
    assert a[2] == b[2], f"{what}: pairs {a[2]} vs {b[2]}"
    assert np.array_equal(a[1], b[1]), f"{what}: counts differ"
    assert np.array_equal(a[3].view(np.uint32), b[3].view(np.uint32)), f"{what}: scores differ"
    assert np.array_equal(a[0], b[0]), f"{what}: layer outputs differ"
    note(f"{what}: P={a[2]} identical")


def test_noalloc_matches_forward_then_a_smaller_layer(torch):
    big = make_workload("lladamoe_t1024_e64")
    wt = weight_tensors(big)
    a, b = _both(torch, big, big.T, state_tensors(big), to_device(big.h), wt)
    _assert_same(a, b, "lladamoe_t1024_e64")
    small = make_workload("tiny_t128_e8")
    a, b = _both(torch, small, small.T, state_tensors(small), to_device(small.h), weight_tensors(small))
    _assert_same(a, b, "tiny_t128_e8 after the larger layer")
    # the fixed-count path on the same scratch
    a, b = _both(torch, small, small.T, state_tensors(small), to_device(small.h), weight_tensors(small),
                 uniform_k=small.params.k_base)
    _assert_same(a, b, "tiny_t128_e8 uniform")


def test_noalloc_shared_expert_inline(torch):
    # the first sequence (1024 tokens) of the LLaDA2.0-mini-shaped layer, with its shared
    # expert, which the allocation-free call runs on the caller's stream
    w = make_workload("llada2mini_t4096_e256")
    T = int(w.seq_offsets[1])
    st = {"block_idx": to_device(w.block_idx[:T]), "masked": to_device(w.masked[:T]),
          "hist_len": to_device(w.hist_len[:T]), "conf_prev1": to_device(w.conf_prev1[:T]),
          "conf_prev2": to_device(w.conf_prev2[:T]),
          "seq_offsets": to_device(np.array([0, T], np.int32)),
          "active_block": to_device(w.active_block[:1])}
    a, b = _both(torch, w, T, st, to_device(w.h[:T]), weight_tensors(w))
    _assert_same(a, b, "llada2mini first sequence + shared expert")


def test_noalloc_rejects_layers_beyond_the_scratch(torch):
    from paper_2608_01784_amd import _lib
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    w = make_workload("llada2mini_t4096_e256")
    assert _lib.lib().reflex_workspace_size(w.T, w.E, w.d, w.f, w.f_shared, w.params.k_max) > \
        _lib.NOALLOC_SCRATCH_BYTES
    lay = MoELayer(w.T, w.d, ExpertWeights(**weight_tensors(w)), w.params)
    args = lay.args(to_device(w.h), TokenState(**state_tensors(w)))
    with pytest.raises(_lib.ReflexError) as e:
        _lib.reflex_moe_forward_noalloc(args)
    assert e.value.status == -4      # REFLEX_ERR_WORKSPACE, nothing launched


def test_noalloc_block_sort_layer(torch):
    # a layer above the route launch's in-kernel sort (275 blocks of 16 tokens x 64
    # experts), so the pairs are sorted by the block-sort launches, on the shared scratch;
    # then the small layer again
    from synth import make_fuzz_workload
    w = make_fuzz_workload(140, T=4400, d=256, E=64, f=128, k_max=6)
    a, b = _both(torch, w, w.T, state_tensors(w), to_device(w.h), weight_tensors(w))
    _assert_same(a, b, "T=4400 E=64 (block sort)")
    small = make_workload("tiny_t128_e8")
    a, b = _both(torch, small, small.T, state_tensors(small), to_device(small.h), weight_tensors(small))
    _assert_same(a, b, "tiny_t128_e8 after the block-sort layer")
