"""Pins of the oracle's score-derived count rules (Top-p and Expert-Threshold
Routing, Appendix B): closed forms on uniform and one-hot routing mass, the
defining minimality of the Top-p prefix checked as a property, monotonicity in
the threshold, and agreement with the TopK prefix order."""
import numpy as np
import pytest

import oracle


def _f32(x):
    return float(np.float32(x))


def test_router_probs_closed_forms():
    r = np.zeros((1, 8))
    assert np.array_equal(oracle.router_probs(r), np.full((1, 8), 0.125))
    r = np.array([[np.log(3.0), 0.0]])            # masses 3/4, 1/4
    assert np.allclose(oracle.router_probs(r), [[0.75, 0.25]], rtol=0, atol=1e-15)


@pytest.mark.parametrize("p,expect", [(0.3, 3), (0.25, 2), (0.125, 1), (0.126, 2), (1.0, 8)])
def test_topp_uniform_mass(p, expect):
    # 8 equal masses of 1/8 (exact): the prefix of n experts holds n/8
    r = np.zeros((3, 8))
    k, cum = oracle.topp_counts(r, p, 1, 12)
    assert np.all(k == expect)
    assert np.all(cum == expect / 8)


@pytest.mark.parametrize("tau,expect", [(0.1, 8), (0.124, 8), (0.125, 1), (0.2, 1)])
def test_threshold_uniform_mass(tau, expect):
    # 1/8 > tau keeps all 8; otherwise none, raised to k_min = 1
    r = np.zeros((2, 8))
    assert np.all(oracle.threshold_counts(r, tau, 1, 12) == expect)


def test_one_dominant_expert():
    r = np.zeros((4, 64))
    r[:, 5] = 50.0
    k, _ = oracle.topp_counts(r, 0.99, 1, 12)
    assert np.all(k == 1)
    assert np.all(oracle.threshold_counts(r, 0.02, 1, 12) == 1)
    # bounds: the clamp raises to k_min
    k, _ = oracle.topp_counts(r, 0.5, 3, 12)
    assert np.all(k == 3)


def _ranked_mass(r):
    prob = oracle.router_probs(r)
    out = []
    for i in range(r.shape[0]):
        order = sorted(range(r.shape[1]), key=lambda e: (-r[i, e], e))
        out.append(prob[i, order])
    return np.array(out)


@pytest.mark.parametrize("seed", range(6))
def test_topp_is_the_shortest_prefix_reaching_p(seed):
    rng = np.random.default_rng(seed)
    E = int(rng.choice([8, 64, 256]))
    r = rng.standard_normal((40, E)) * rng.uniform(0.3, 3.0)
    p = _f32(rng.uniform(0.05, 0.6))
    k, _ = oracle.topp_counts(r, p, 1, E)
    ranked = _ranked_mass(r)
    for i in range(r.shape[0]):
        n = int(k[i])
        assert ranked[i, :n].sum() >= p - 1e-12
        assert n == 1 or ranked[i, :n - 1].sum() < p + 1e-12


@pytest.mark.parametrize("seed", range(4))
def test_rules_monotone_and_threshold_is_a_prefix(seed):
    rng = np.random.default_rng(100 + seed)
    r = rng.standard_normal((50, 64)) * 1.5
    ks = [oracle.topp_counts(r, _f32(p), 1, 64)[0] for p in (0.1, 0.2, 0.4, 0.8)]
    for a, b in zip(ks, ks[1:]):
        assert np.all(a <= b)
    ts = [oracle.threshold_counts(r, _f32(t), 0, 64) for t in (0.005, 0.01, 0.02, 0.05)]
    for a, b in zip(ts, ts[1:]):
        assert np.all(a >= b)
    # the experts above the threshold are the first ones in TopK order
    prob = oracle.router_probs(r)
    n = oracle.threshold_counts(r, _f32(0.02), 0, 64)
    route = oracle.topk_route(r, n)
    for i in range(r.shape[0]):
        sel = set(route.expert[route.offsets[i]:route.offsets[i + 1]].tolist())
        assert sel == set(np.nonzero(prob[i] > _f32(0.02))[0].tolist())


def test_bounds_paper_setting():
    # the compared rules use counts in [1, 12]
    rng = np.random.default_rng(7)
    r = rng.standard_normal((200, 64)) * 0.9
    k, _ = oracle.topp_counts(r, 0.20, 1, 12)
    assert k.min() >= 1 and k.max() <= 12
    t = oracle.threshold_counts(r, 0.0190, 1, 12)
    assert t.min() >= 1 and t.max() <= 12
