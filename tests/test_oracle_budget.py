"""Pins of the oracle's allocator (RRB, forecast, FPS, FGER, clamp) against what the
paper fixes: hand-derived budgets, closed-form points of the logistic gates,
stated invariants, and brute-force optimality on tiny inputs."""
import itertools
import math

import numpy as np
import pytest

import oracle
from conftest import read_golden
from synth import AllocParams, make_workload, make_fuzz_workload


def logistic(x):
    # closed form independent of the oracle's exp-based sigmoid
    return 0.5 * (1.0 + math.tanh(0.5 * x))


def f32(x):
    return float(np.float32(x))


# ---------------------------------------------------------------- RRB (Eq. (5))
def test_rrb_budget_matches_hand_derivation_for_every_active_block():
    rows = read_golden("rrb_budget_lladamoe_t1024.txt")
    for a_str, ks_str in rows:
        w = make_workload("lladamoe_t1024_e64", seed=0, active=int(a_str))
        p = w.params
        d = oracle.block_distance(w.block_idx, w.seq_offsets, w.active_block)
        H = oracle.role_budget(d, p.k_base, p.delta_role)
        assert int(H.sum()) == int(ks_str), a_str
        res = oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1,
                                   w.conf_prev2, w.seq_offsets, w.active_block, p)
        assert res.k_sigma == int(ks_str)
        # FGER keeps the total before the clamp (Section 4.3)
        assert int(res.k_unclamped.sum()) == int(ks_str)
        # the clamp at K_max = 12 removes delta_cur from each high-group member
        n_high = int((res.group == 1).sum())
        assert res.pairs == int(ks_str) - n_high * (p.k_base + p.delta_role + p.delta_cur - p.k_max)


def test_rrb_three_levels_on_role_relabelled_tiny():
    w = make_workload("tiny_roles_t128_e8")
    res = oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1, w.conf_prev2,
                               w.seq_offsets, w.active_block, w.params)
    # prompt: d = 3 -> K_base - delta_role = 1; active block d = 0 -> 3; block 5 d = 2 -> 2
    assert set(res.k_rrb[:64]) == {1}
    assert set(res.k_rrb[64:96]) == {3}
    assert set(res.k_rrb[96:]) == {2}
    assert res.k_sigma == 64 * 1 + 32 * 3 + 32 * 2 == 224
    assert res.pairs == 224  # FGER on m = 16 preserves the total, clamp [1, 4] inactive


def test_tiny_counts_and_pairs():
    w = make_workload("tiny_t128_e8")
    res = oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1, w.conf_prev2,
                               w.seq_offsets, w.active_block, w.params)
    # every token has d <= 1: H = 3; FGER on m = 16, n_q = 4 -> {4 x 4, 8 x 3, 4 x 2}
    J = (w.masked == 1) & (w.block_idx == 1)
    vals, cnt = np.unique(res.k[J], return_counts=True)
    assert dict(zip(vals.tolist(), cnt.tolist())) == {2: 4, 3: 8, 4: 4}
    assert set(res.k[~J]) == {3}
    assert res.pairs == 384


def test_distance_uses_each_sequences_active_block():
    b = np.array([0, 1, 2, 3, 0, 1, 2, 3], np.int32)
    so = np.array([0, 4, 8], np.int32)
    act = np.array([1, 3], np.int32)
    assert oracle.block_distance(b, so, act).tolist() == [1, 0, 1, 2, 3, 2, 1, 0]


# ------------------------------------------------------- forecast and FPS (Eqs. (6)-(8))
@pytest.mark.parametrize("w", [0.30, 0.25])
def test_frontier_factor_closed_form_points(w):
    th, wf, ta = f32(0.9), f32(w), f32(0.05)
    # at the centre of the frontier interval both gates see w/(2 tau)
    c = th - wf / 2
    assert oracle.frontier_factor(c, th, wf, ta) == pytest.approx(logistic(wf / (2 * ta)) ** 2, rel=1e-13)
    # at either end one gate is sigma(0) = 1/2 and the other sigma(w/tau)
    for c in (th, th - wf):
        assert oracle.frontier_factor(c, th, wf, ta) == pytest.approx(0.5 * logistic(wf / ta), rel=1e-13)
    # symmetric about the centre, and maximal there
    xs = np.linspace(-0.5, 0.5, 101)
    left = oracle.frontier_factor(th - wf / 2 - xs, th, wf, ta)
    right = oracle.frontier_factor(th - wf / 2 + xs, th, wf, ta)
    np.testing.assert_allclose(left, right, rtol=1e-12, atol=1e-300)
    assert np.argmax(right) == 50


def test_frontier_factor_paper_default_values():
    # sigma(3)^2 and sigma(2.5)^2 for w = 0.30 / 0.25, tau = 0.05 at the interval centre.
    # The hyper-parameters are float32 values (w/(2 tau) = 3 + 4.5e-8), so the decimal
    # closed form holds to ~1e-8; the exact-float32 form is pinned tightly above.
    assert oracle.frontier_factor(f32(0.9) - f32(0.3) / 2, 0.9, 0.30, 0.05) == pytest.approx(
        0.9073974670915, abs=2e-8)
    assert oracle.frontier_factor(f32(0.9) - f32(0.25) / 2, 0.9, 0.25, 0.05) == pytest.approx(
        0.8540381034336, abs=2e-8)


def test_progress_factor_closed_form_points():
    vr, ta = f32(0.01), f32(0.05)
    assert oracle.progress_factor(vr, 0.01, 0.05) == pytest.approx(0.5, abs=1e-15)
    assert oracle.progress_factor(0.0, 0.01, 0.05) == pytest.approx(logistic(vr / ta), rel=1e-13)
    # logistic symmetry about v_ref, and monotone decreasing in v_bar
    v = np.linspace(-0.2, 0.2, 41)
    p1 = oracle.progress_factor(v, 0.01, 0.05)
    p2 = oracle.progress_factor(2 * vr - v, 0.01, 0.05)
    np.testing.assert_allclose(p1 + p2, 1.0, rtol=1e-13)
    assert np.all(np.diff(p1) < 0)
    # clipped extremes for w = 0.30
    assert oracle.progress_factor(f32(0.3) / 2, 0.01, 0.05) == pytest.approx(0.0573241758989, abs=2e-8)
    assert oracle.progress_factor(-f32(0.3) / 2, 0.01, 0.05) == pytest.approx(0.9608342772032, abs=2e-8)


def test_forecast_clips_and_history_rules():
    w = f32(0.30)
    c1 = np.array([0.5, 0.5, 0.95, 0.02, 0.4, 0.4], np.float32)
    c2 = np.array([0.1, 0.9, 0.50, 0.40, 0.4, 0.0], np.float32)
    hist = np.array([2, 2, 2, 2, 1, 0], np.int8)
    vb, ch = oracle.confidence_forecast(c1, c2, hist, 0.30)
    c1d = c1.astype(np.float64)
    assert vb[0] == w / 2 and ch[0] == c1d[0] + w / 2          # +0.4 clipped to +w/2
    assert vb[1] == -w / 2 and ch[1] == c1d[1] - w / 2         # -0.4 clipped to -w/2
    assert ch[2] == 1.0                                        # forecast clipped at 1
    assert ch[3] == 0.0                                        # forecast clipped at 0
    assert vb[4] == 0.0 and ch[4] == c1d[4]                    # one observation: zero velocity
    S, F, P, _, _ = oracle.frontier_progress_score(c1, c2, hist, 0.9, 0.30, 0.01, 0.05)
    assert P[4] == 1.0 and S[4] == F[4]                        # P = 1 without c^{t-2}
    np.testing.assert_array_equal(S, F * P)


def test_fps_prefers_frontier_and_slow_progress():
    # the multiplicative score suppresses tokens meeting only one condition
    th = 0.9
    c_front = np.float32(0.75)
    S = oracle.frontier_progress_score(
        np.array([c_front, c_front, 0.2, 0.2], np.float32),
        np.array([c_front, c_front - np.float32(0.15), 0.2, 0.05], np.float32),
        np.array([2, 2, 2, 2], np.int8), th, 0.30, 0.01, 0.05)[0]
    # near the frontier and stalled beats near-the-frontier-but-rising, and both beat
    # far-from-frontier tokens
    assert S[0] > S[1] > max(S[2], S[3])


# ------------------------------------------------------------------ FGER (Eq. (9))
@pytest.mark.parametrize("m,q", [(m, q) for m in range(0, 9) for q in (0.125, 0.25, 0.3, 0.5)])
def test_fger_groups_brute_force_optimal(m, q):
    rng = np.random.default_rng(1000 + m)
    S = rng.random(m)
    tok = np.arange(m) + 7
    g = oracle.fger_groups(S, tok, q)
    n_q = int(math.floor(f32(q) * m))
    assert (g == 1).sum() == n_q and (g == -1).sum() == n_q
    # rearrangement: among all assignments with these group sizes, ours maximises sum g*S
    best = -np.inf
    for hi in itertools.combinations(range(m), n_q):
        rest = [i for i in range(m) if i not in hi]
        for lo in itertools.combinations(rest, n_q):
            gg = np.zeros(m)
            gg[list(hi)] = 1
            gg[list(lo)] = -1
            best = max(best, float(gg @ S))
    assert float(g @ S) == pytest.approx(best, abs=1e-12)


def test_fger_ties_go_to_lower_token_index():
    S = np.array([0.5, 0.7, 0.5, 0.5, 0.7, 0.1, 0.5, 0.5])
    tok = np.array([10, 11, 12, 13, 14, 15, 16, 17])
    g = oracle.fger_groups(S, tok, 0.25)        # n_q = 2
    assert g.tolist() == [0, 1, 0, 0, 1, -1, 0, -1]
    g = oracle.fger_groups(np.full(8, 0.3), tok, 0.25)
    assert g.tolist() == [1, 1, 0, 0, 0, 0, -1, -1]


def _budget(w, p):
    return oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1, w.conf_prev2,
                                w.seq_offsets, w.active_block, p)


@pytest.mark.parametrize("seed", range(12))
def test_fger_preserves_active_block_budget_when_clamp_inactive(seed):
    w = make_fuzz_workload(seed, k_max=32)
    p = w.params.replace(k_min=0, k_max=1000)
    res = _budget(w, p)
    # J total equals |J| K_cur per sequence; total equals K^Sigma
    assert res.pairs == res.k_sigma
    k_cur = p.k_base + p.delta_role
    for s in range(w.B):
        lo, hi = w.seq_offsets[s], w.seq_offsets[s + 1]
        J = np.arange(lo, hi)[(w.masked[lo:hi] == 1) & (w.block_idx[lo:hi] == w.active_block[s])]
        assert int(res.k[J].sum()) == len(J) * k_cur
        assert np.all(res.k[J] <= k_cur + p.delta_cur) and np.all(res.k[J] >= k_cur - p.delta_cur)
        # tokens of J without history keep K_cur
        assert np.all(res.k[J][w.hist_len[J] == 0] == k_cur)


def test_fger_only_keeps_avgk_at_k_base_as_in_table_2():
    avgk = float([r for r in read_golden("table_pairs_avgk.txt") if r[0] == "fger_only_avgk"][0][1])
    for name in ("lladamoe_t1024_e64", "llada2mini_t4096_e256"):
        w = make_workload(name)
        p = w.params.replace(delta_role=0, k_max=16)   # FGER Only: no role offset
        res = _budget(w, p)
        assert res.pairs / w.T == avgk == p.k_base


def test_rrb_only_equals_role_prior_and_uniform_equals_k_base():
    w = make_workload("lladamoe_t1024_e64")
    res = _budget(w, w.params.replace(delta_cur=0))
    np.testing.assert_array_equal(res.k, res.k_rrb)
    res = _budget(w, w.params.replace(delta_cur=0, delta_role=0))
    assert np.all(res.k == w.params.k_base)


@pytest.mark.parametrize("field,values", [
    ("w_cf", [0.20, 0.25, 0.30, 0.35, 0.40]),      # Appendix D sweeps
    ("v_ref", [0.0, 0.005, 0.01, 0.025, 0.05]),
    ("tau", [0.01, 0.025, 0.05, 0.10, 0.20]),
    ("q", [0.125, 0.25, 0.375]),
    ("signal", [0, 1, 2, 3, 4]),
])
def test_ranking_only_parameters_leave_the_budget_unchanged(field, values):
    w = make_workload("llada2mini_t4096_e256")
    base = w.params.replace(k_max=16)
    totals = {_budget(w, base.replace(**{field: v})).pairs for v in values}
    assert totals == {_budget(w, base).pairs}


def test_clamp_keeps_counts_in_bounds():
    for seed in range(20):
        w = make_fuzz_workload(seed)
        res = _budget(w, w.params)
        assert res.k.min() >= w.params.k_min and res.k.max() <= w.params.k_max


def test_signal_variants_rank_by_their_key():
    c1 = np.array([0.1, 0.8, 0.5, 0.95, 0.3, 0.6, 0.7, 0.2], np.float32)
    c2 = c1 - np.float32(0.05)
    hist = np.full(8, 2, np.int8)
    b = np.ones(8, np.int32)
    so = np.array([0, 8], np.int32)
    act = np.array([1], np.int32)
    m = np.ones(8, np.uint8)
    p = AllocParams.make(8, 4, 2, 1, 16, q=0.25)
    k = oracle.assign_budget(b, m, hist, c1, c2, so, act, p.replace(signal=3)).k
    assert k.tolist() == [10, 14, 12, 14, 12, 12, 12, 10]      # highest c^{t-1} get +2
    k = oracle.assign_budget(b, m, hist, c1, c2, so, act, p.replace(signal=4)).k
    assert k.tolist() == [14, 10, 12, 10, 12, 12, 12, 14]      # lowest c^{t-1} get +2


def test_frontier_only_and_progress_only_rank_by_their_own_factor():
    """Appendix C's single-signal rankings: Frontier Only orders J by F of Eq. (6),
    Progress Only by P of Eq. (7).  The eight tokens decouple the two factors: F
    depends only on the forecast c_hat and, being sigma(w/2 + x) sigma(w/2 - x) over
    tau with x = c_hat - (theta - w/2), falls strictly with |x|; P depends only on the
    clipped velocity v_bar and falls strictly with it.  Every c is a multiple of 1/32
    (exact in fp32, and c1 - c2, c1 + v_bar exact in fp64) and no velocity reaches the
    w/2 clip, so v_bar = c1 - c2 and c_hat = c1 + v_bar."""
    #           t0     t1      t2     t3      t4       t5       t6       t7
    c_hat = [0.75, 0.6875, 0.25, 0.5, 0.875, 0.59375, 0.375, 0.71875]
    v_bar = [0.125, 0.0625, -0.125, -0.0625, 0.09375, 0.0, -0.09375, 0.03125]
    c1 = np.array([c - v for c, v in zip(c_hat, v_bar)], np.float32)
    c2 = np.array([a - v for a, v in zip(c1.tolist(), v_bar)], np.float32)
    hist = np.full(8, 2, np.int8)
    b = np.ones(8, np.int32)
    so = np.array([0, 8], np.int32)
    act = np.array([1], np.int32)
    m = np.ones(8, np.uint8)
    # K_cur = 12, delta_cur = 2, q = 0.25 -> outer groups of 2, clamp [1, 16] inactive
    p = AllocParams.make(8, 4, 2, 1, 16, q=0.25, w_cf=0.30)
    # by |c_hat - 0.75|: t0 < t7 < t1 < t4 < t5 < t3 < t6 < t2
    k_f = oracle.assign_budget(b, m, hist, c1, c2, so, act, p.replace(signal=1)).k
    assert k_f.tolist() == [14, 12, 10, 12, 12, 12, 10, 14]
    # by v_bar ascending (larger P first): t2 < t6 < t3 < t5 < t7 < t1 < t4 < t0
    k_p = oracle.assign_budget(b, m, hist, c1, c2, so, act, p.replace(signal=2)).k
    assert k_p.tolist() == [10, 12, 14, 12, 10, 12, 14, 12]
    # the keys themselves at t0 (c_hat at the frontier centre, v_bar = 1/8) and t2,
    # against the logistic evaluated here in tanh form on the fp32 hyper-parameters
    th, w, tau, vr = f32(0.9), f32(0.30), f32(0.05), f32(0.01)
    for t in (0, 2):
        F = logistic((c_hat[t] - th + w) / tau) * logistic((th - c_hat[t]) / tau)
        P = logistic((vr - v_bar[t]) / tau)
        kf = oracle.ranking_key(1, c1[t:t + 1], c2[t:t + 1], hist[t:t + 1], th, w, vr, tau)[0]
        kp = oracle.ranking_key(2, c1[t:t + 1], c2[t:t + 1], hist[t:t + 1], th, w, vr, tau)[0]
        assert kf == pytest.approx(F, rel=1e-12) and kp == pytest.approx(P, rel=1e-12)
    # t0 sits at the frontier centre: F = sigma(w / 2 tau)^2 = sigma(3)^2 (w = 0.30)
    k0 = oracle.ranking_key(1, c1[:1], c2[:1], hist[:1], th, w, vr, tau)[0]
    assert k0 == pytest.approx(0.9073974670915, abs=2e-7)
