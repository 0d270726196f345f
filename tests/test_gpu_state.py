"""GPU parity of the cross-forward decoding state update and of a whole synthetic
multi-forward trajectory against the oracle.

Every state array after every forward must equal the oracle's bit for bit (the
kernel only compares fp32 confidences with fp32 theta and copies values), and the
counts each forward's budget assigns must equal the oracle's on the same state."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from gpu_common import note, require_gpu
from synth import forward_confidence, generation_start, make_fuzz_workload, make_workload
from synth.device import state_tensors, to_device

pytestmark = pytest.mark.gpu

THETA = 0.9


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


def _host(state):
    return {k: getattr(state, k).cpu().numpy() for k in
            ("block_idx", "masked", "hist_len", "conf_prev1", "conf_prev2", "seq_offsets",
             "active_block")}


def _check_advance(before, after, conf_t, min_commit, remaining=None):
    ref = oracle.advance_state(before["block_idx"], before["masked"], before["hist_len"],
                               before["conf_prev1"], before["conf_prev2"], before["seq_offsets"],
                               before["active_block"], conf_t, THETA, min_commit)
    assert np.array_equal(after["masked"], ref.masked)
    assert np.array_equal(after["hist_len"], ref.hist_len)
    assert np.array_equal(after["conf_prev1"].view(np.uint32), ref.conf_prev1.view(np.uint32))
    assert np.array_equal(after["conf_prev2"].view(np.uint32), ref.conf_prev2.view(np.uint32))
    assert np.array_equal(after["active_block"], ref.active_block)
    if remaining is not None:
        assert np.array_equal(remaining, ref.remaining)
    return ref


@pytest.mark.parametrize("min_commit", [0, 1])
@pytest.mark.parametrize("name", ["tiny_t128_e8", "tiny_roles_t128_e8", "lladamoe_t1024_e64",
                                  "llada2mini_t4096_e256", "skewed_t16384_e256", "fuzz3", "fuzz9"])
def test_advance_state_one_forward(torch, name, min_commit):
    from paper_2608_01784_amd import _lib
    from paper_2608_01784_amd.layer import TokenState
    w = make_fuzz_workload(int(name[4:])) if name.startswith("fuzz") else make_workload(name)
    st = TokenState(**state_tensors(w))
    before = _host(st)
    # low confidences exercise the progress guard; the usual ones the threshold
    conf = forward_confidence(11, 0 if min_commit else 4, w.T)
    rem = torch.empty(w.B, dtype=torch.int32, device="cuda")
    _lib.reflex_advance_state(to_device(conf), st.block_idx, st.seq_offsets, THETA, min_commit,
                              st.masked, st.hist_len, st.conf_prev1, st.conf_prev2, st.active_block,
                              rem)
    torch.cuda.synchronize()
    ref = _check_advance(before, _host(st), conf, min_commit, rem.cpu().numpy())
    note(f"{name}: committed {int(ref.committed.sum())}, advanced "
         f"{int((ref.active_block != before['active_block']).sum())} sequence(s)")


@pytest.mark.parametrize("name,min_commit", [("lladamoe_t1024_e64", 0), ("tiny_t128_e8", 1),
                                             ("llada2mini_t4096_e256", 0)])
def test_trajectory_matches_oracle(torch, name, min_commit):
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    from paper_2608_01784_amd.trajectory import run_trajectory
    w = make_workload(name)
    start = generation_start(w)
    st = TokenState(**{k: to_device(v) for k, v in start.items()})
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()),
          "router_bias": None if w.router_bias is None else to_device(w.router_bias)}
    sh = w.shared_weights()
    if sh is not None:
        dw["ws_gate"], dw["ws_up"], dw["ws_down"] = (to_device(x) for x in sh)
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params)
    h = to_device(w.h)
    confs = {}
    ref_state = dict(start)
    n_checked = [0]

    def conf_fn(t):
        confs[t] = forward_confidence(5, t, w.T)
        return to_device(confs[t])

    def on_forward(t, state):
        k = lay.k.cpu().numpy()
        b = oracle.assign_budget(ref_state["block_idx"], ref_state["masked"], ref_state["hist_len"],
                                 ref_state["conf_prev1"], ref_state["conf_prev2"],
                                 ref_state["seq_offsets"], ref_state["active_block"], w.params)
        assert np.array_equal(k, b.k), t
        assert np.array_equal(_host(state)["masked"], ref_state["masked"]), t
        n_checked[0] += 1

    def advance_ref(t):
        r = oracle.advance_state(ref_state["block_idx"], ref_state["masked"], ref_state["hist_len"],
                                 ref_state["conf_prev1"], ref_state["conf_prev2"],
                                 ref_state["seq_offsets"], ref_state["active_block"], confs[t], THETA,
                                 min_commit)
        ref_state.update(masked=r.masked, hist_len=r.hist_len, conf_prev1=r.conf_prev1,
                         conf_prev2=r.conf_prev2, active_block=r.active_block)
        return r

    # step the oracle in lockstep: each callback checks forward t, then the oracle advances
    def on_forward_and_advance(t, state):
        if t > 0:
            advance_ref(t - 1)
        on_forward(t, state)

    stats = run_trajectory(lay, h, st, conf_fn, THETA, min_commit, max_forwards=400,
                           on_forward=on_forward_and_advance)
    r = advance_ref(stats.forwards - 1)
    torch.cuda.synchronize()
    final = _host(st)
    assert np.array_equal(final["masked"], r.masked) and r.masked.sum() == 0
    assert np.array_equal(final["active_block"], r.active_block)
    assert n_checked[0] == stats.forwards
    note(f"{name}: {stats.forwards} forwards, {stats.total_pairs} pairs, "
         f"AvgK {stats.total_pairs / (stats.forwards * w.T):.3f}")
