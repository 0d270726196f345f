"""Pins of the oracle's cross-forward state update (Section 3.1, Eq. (1)):
the committed set is exactly the masked active-block positions at or above the
threshold, masks only shrink, the confidence history shifts by one forward,
blocks advance only when emptied, the optional progress guard commits the single
most confident position, and a rising-confidence trajectory terminates."""
import numpy as np
import pytest

import oracle
from synth import forward_confidence, generation_start, make_workload

TH = 0.9


def _one_seq(b, masked, a, conf_t, c1=None, hist=None, min_commit=0):
    T = len(b)
    c1 = np.zeros(T, np.float32) if c1 is None else np.asarray(c1, np.float32)
    hist = np.zeros(T, np.int8) if hist is None else np.asarray(hist, np.int8)
    return oracle.advance_state(np.asarray(b, np.int32), np.asarray(masked, np.uint8), hist, c1,
                                np.full(T, 0.5, np.float32), np.array([0, T], np.int32),
                                np.array([a], np.int32), np.asarray(conf_t, np.float32), TH,
                                min_commit)


def test_commits_exactly_the_confident_active_positions():
    b = [0, 0, 1, 1, 1, 1, 2, 2]
    m = [0, 0, 1, 1, 1, 0, 1, 1]
    ct = [0.99, 0.99, 0.95, 0.5, np.float32(0.9), 0.99, 0.99, 0.2]
    r = _one_seq(b, m, 1, ct)
    # positions 2 (0.95) and 4 (exactly fp32 0.9) commit; 3 stays; block 2 is untouched
    assert r.committed.tolist() == [False, False, True, False, True, False, False, False]
    assert r.masked.tolist() == [0, 0, 0, 1, 0, 0, 1, 1]
    assert r.active_block.tolist() == [1]           # position 3 still masked
    assert r.remaining.tolist() == [3]


def test_history_shifts_for_every_masked_position():
    b = [1, 1, 2, 2]
    m = [1, 0, 1, 1]
    c1 = [0.3, 0.4, 0.5, 0.6]
    hist = [0, 1, 1, 2]
    ct = [0.7, 0.8, 0.1, 0.2]
    r = _one_seq(b, m, 1, ct, c1=c1, hist=hist)
    assert r.conf_prev1.tolist() == pytest.approx([0.7, 0.4, 0.1, 0.2])
    assert r.conf_prev2.tolist() == pytest.approx([0.3, 0.5, 0.5, 0.6])    # 0.5 = old c^{t-2}
    assert r.hist_len.tolist() == [1, 1, 2, 2]


def test_block_advances_only_when_emptied_and_stops_at_the_last():
    b = [1, 1, 2, 2]
    r = _one_seq(b, [1, 1, 1, 1], 1, [0.95, 0.91, 0.0, 0.0])
    assert r.active_block.tolist() == [2]
    r = _one_seq(b, [0, 0, 1, 1], 2, [0.0, 0.0, 0.95, 0.99])
    assert r.active_block.tolist() == [2] and r.remaining.tolist() == [0]


@pytest.mark.parametrize("min_commit", [0, 1])
def test_progress_guard(min_commit):
    b = [1, 1, 1, 1]
    ct = [0.3, 0.7, 0.7, 0.1]
    r = _one_seq(b, [1, 1, 1, 1], 1, ct, min_commit=min_commit)
    if min_commit:
        assert r.committed.tolist() == [False, True, False, False]   # tie -> lower position
    else:
        assert not r.committed.any()


def test_trajectory_terminates_and_masks_only_shrink():
    w = make_workload("lladamoe_t1024_e64")
    st = generation_start(w)
    n_blocks = int(w.block_idx.max())
    for t in range(200):
        prev = st["masked"].copy()
        r = oracle.advance_state(st["block_idx"], st["masked"], st["hist_len"], st["conf_prev1"],
                                 st["conf_prev2"], st["seq_offsets"], st["active_block"],
                                 forward_confidence(7, t, len(prev)), TH)
        assert np.all(r.masked <= prev)
        assert np.all(r.committed == ((prev == 1) & (r.masked == 0)))
        st.update(masked=r.masked, hist_len=r.hist_len, conf_prev1=r.conf_prev1,
                  conf_prev2=r.conf_prev2, active_block=r.active_block)
        if r.remaining.sum() == 0:
            break
    assert r.remaining.sum() == 0
    assert t + 1 >= n_blocks                  # at least one forward per block
    assert st["active_block"].tolist() == [n_blocks]
