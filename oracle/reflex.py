"""fp64 oracle of the REFLEX MoE layer (test infrastructure only).

Notation follows the paper: T_i the selected expert set of token i, k_i its
count, r_{i,e} router scores, alpha_{i,e} the normalised router weight,
b(i) the block index (prompt = 0), a the active block, J the masked positions
of the active block, c^{t-1}, c^{t-2} the two latest confidences.

Every real computation is fp64.  bf16 inputs are widened exactly; float32
inputs and hyper-parameters are widened exactly (so theta is float32(0.9)).

Readings where the paper is silent or leaves a choice (each also listed in
the design notes of the repository):
  * counts are clamped to [K_min, K_max] after reallocation (Eq. (3) bounds);
  * the outer FGER groups both have floor(q * m) members, m = |J'|;
  * J' = J restricted to tokens with at least one confidence observation;
    tokens of J without history keep K_cur;
  * ranking ties (equal scores) go to the lower token index; TopK ties go to
    the lower expert index; -0.0 compares equal to +0.0;
  * alpha is the softmax of the router scores renormalised over T_i
    (``norm_topk=1``), or the full softmax over all E experts (``norm_topk=0``);
  * each expert is a bias-free SwiGLU: W_d (SiLU(W_g x) * (W_u x)).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

__all__ = [
    "bf16_to_f64", "f64_to_bf16_bits", "sigmoid",
    "router_scores", "block_distance", "role_budget", "confidence_forecast",
    "frontier_factor", "progress_factor", "frontier_progress_score", "ranking_key",
    "fger_groups", "assign_budget", "BudgetResult", "advance_state", "StateResult",
    "topk_route", "RouteResult", "pair_permutation", "PermResult",
    "router_probs", "topp_counts", "threshold_counts",
    "swiglu_expert", "moe_layer", "dense_masked_moe", "fixed_topk_moe",
    "routed_expert_flops", "SIGNAL_FPS", "SIGNAL_FRONTIER", "SIGNAL_PROGRESS",
    "SIGNAL_CONFIDENCE", "SIGNAL_UNCERTAINTY",
]

SIGNAL_FPS, SIGNAL_FRONTIER, SIGNAL_PROGRESS, SIGNAL_CONFIDENCE, SIGNAL_UNCERTAINTY = 0, 1, 2, 3, 4


# ---------------------------------------------------------------------------------------
# number formats
# ---------------------------------------------------------------------------------------
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns: the bits are the high half of a float32."""
    b = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to bfloat16 (8 significant bits, nearest, ties to even)
    in one step, and return the bit patterns.  Finite, normal-range inputs only."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2**e, 0.5 <= |m| < 1
    r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)   # keep 8 significant bits
    return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def sigmoid(x):
    """The logistic function 1 / (1 + e^{-x})."""
    return 1.0 / (1.0 + np.exp(-np.asarray(x, dtype=np.float64)))


def _p64(v) -> float:
    return float(np.float64(np.float32(v)))


# ---------------------------------------------------------------------------------------
# router scores (Section 3.2)
# ---------------------------------------------------------------------------------------
def router_scores(h_bits: np.ndarray, w_router: np.ndarray,
                  bias: Optional[np.ndarray] = None) -> np.ndarray:
    """r_{i,e} = sum_k h_{i,k} W_r[e,k] (+ bias_e), in fp64.  h: bf16 bits [T,d];
    W_r: float32 [E,d]; result [T,E]."""
    h = bf16_to_f64(h_bits)
    r = h @ np.asarray(w_router, dtype=np.float64).T
    if bias is not None:
        r = r + np.asarray(bias, dtype=np.float64)[None, :]
    return r


# ---------------------------------------------------------------------------------------
# Refinement-Role Budgeting (Section 4.2, Eq. (5))
# ---------------------------------------------------------------------------------------
def block_distance(block_idx, seq_offsets, active_block) -> np.ndarray:
    """d_t(i) = |b(i) - a_t| with a_t the active block of the token's sequence."""
    b = np.asarray(block_idx, dtype=np.int64)
    d = np.empty_like(b)
    so = np.asarray(seq_offsets)
    for s in range(len(so) - 1):
        lo, hi = int(so[s]), int(so[s + 1])
        d[lo:hi] = np.abs(b[lo:hi] - int(active_block[s]))
    return d


def role_budget(dist: np.ndarray, k_base: int, delta_role: int) -> np.ndarray:
    """H(d): K_base + delta_role for d <= 1, K_base for d == 2, K_base - delta_role
    for d >= 3 (Eq. (5))."""
    dist = np.asarray(dist)
    return np.where(dist <= 1, k_base + delta_role,
                    np.where(dist == 2, k_base, k_base - delta_role)).astype(np.int64)


# ---------------------------------------------------------------------------------------
# Frontier-Guided Expert Reallocation (Section 4.3, Eqs. (6)-(9))
# ---------------------------------------------------------------------------------------
def confidence_forecast(c1, c2, hist, w_cf):
    """First-order forecast of the unobserved confidence.

    With both observations (hist == 2): v = c^{t-1} - c^{t-2}, clipped to
    [-w_cf/2, w_cf/2] giving v_bar, and c_hat = clip(c^{t-1} + v_bar, 0, 1).
    With one (hist == 1): v_bar = 0 and c_hat = c^{t-1}.  Returns (v_bar, c_hat)."""
    c1 = np.asarray(c1, dtype=np.float64)
    c2 = np.asarray(c2, dtype=np.float64)
    w = _p64(w_cf)
    two = np.asarray(hist) >= 2
    v = np.where(two, c1 - c2, 0.0)
    v_bar = np.minimum(np.maximum(v, -w / 2.0), w / 2.0)
    c_hat = np.where(two, np.minimum(np.maximum(c1 + v_bar, 0.0), 1.0), c1)
    return v_bar, c_hat


def frontier_factor(c_hat, theta, w_cf, tau):
    """F = sigma((c_hat - theta + w_cf)/tau) * sigma((theta - c_hat)/tau)  (Eq. (6))."""
    th, w, ta = _p64(theta), _p64(w_cf), _p64(tau)
    c_hat = np.asarray(c_hat, dtype=np.float64)
    return sigmoid((c_hat - th + w) / ta) * sigmoid((th - c_hat) / ta)


def progress_factor(v_bar, v_ref, tau):
    """P = sigma((v_ref - v_bar)/tau)  (Eq. (7))."""
    return sigmoid((_p64(v_ref) - np.asarray(v_bar, dtype=np.float64)) / _p64(tau))


def frontier_progress_score(c1, c2, hist, theta, w_cf, v_ref, tau):
    """S = F * P (Eq. (8)); P is taken as 1 when c^{t-2} is missing (hist < 2).
    Returns (S, F, P, v_bar, c_hat)."""
    v_bar, c_hat = confidence_forecast(c1, c2, hist, w_cf)
    F = frontier_factor(c_hat, theta, w_cf, tau)
    P = np.where(np.asarray(hist) >= 2, progress_factor(v_bar, v_ref, tau), 1.0)
    return F * P, F, P, v_bar, c_hat


def ranking_key(signal: int, c1, c2, hist, theta, w_cf, v_ref, tau):
    """Active-block priority key: the Frontier-Progress Score (signal 0), or one of
    the single-signal rankings compared in Appendix C: frontier factor alone (1),
    progress factor alone (2), lagged confidence c^{t-1} (3), its complement (4)."""
    S, F, P, _, _ = frontier_progress_score(c1, c2, hist, theta, w_cf, v_ref, tau)
    c1 = np.asarray(c1, dtype=np.float64)
    return {SIGNAL_FPS: S, SIGNAL_FRONTIER: F, SIGNAL_PROGRESS: P,
            SIGNAL_CONFIDENCE: c1, SIGNAL_UNCERTAINTY: 1.0 - c1}[int(signal)]


def fger_groups(score: np.ndarray, token: np.ndarray, q: float):
    """Eq. (9) grouping.  Rank the candidates by (score descending, token index
    ascending); the first floor(q*m) form G_high, the last floor(q*m) form G_low,
    the rest G_mid.  Returns +1 / 0 / -1 per candidate (in input order)."""
    m = len(score)
    n_q = int(np.floor(_p64(q) * m))
    order = np.lexsort((np.asarray(token), -np.asarray(score, dtype=np.float64)))
    g = np.zeros(m, dtype=np.int64)
    g[order[:n_q]] = 1
    if n_q:
        g[order[m - n_q:]] = -1
    return g


@dataclass
class BudgetResult:
    k: np.ndarray            # final counts, int64 [T]
    k_unclamped: np.ndarray  # after RRB + FGER, before the [K_min, K_max] clamp
    k_rrb: np.ndarray        # RRB prior H(d)
    score: np.ndarray        # ranking key per token (NaN where not ranked)
    group: np.ndarray        # +1 / 0 / -1 / 0 per token (0 also for unranked)
    ranked: np.ndarray       # bool: token was in J' (ranked by FGER)

    @property
    def pairs(self) -> int:
        return int(self.k.sum())

    @property
    def k_sigma(self) -> int:
        """Per-forward budget K^Sigma = sum_i H(d_t(i)) (Section 4.2)."""
        return int(self.k_rrb.sum())


def assign_budget(block_idx, masked, hist_len, conf_prev1, conf_prev2, seq_offsets,
                  active_block, params) -> BudgetResult:
    """The REFLEX allocator Pi (Eq. (3)) for one denoising forward.

    Per sequence s with active block a_s:
      1. RRB prior k_i = H(|b(i) - a_s|) for every token (Eq. (5)).
      2. J = masked tokens of the active block (Section 3.1); J' = those with
         confidence history.  K_cur = K_base + delta_role.
      3. Rank J' by the score (Eq. (8)) and give the groups K_cur + delta_cur /
         K_cur / K_cur - delta_cur (Eq. (9)).  Tokens of J without history keep
         K_cur; every other token keeps its RRB count.
      4. Clamp every count to [K_min, K_max].
    """
    p = params
    dist = block_distance(block_idx, seq_offsets, active_block)
    k_rrb = role_budget(dist, p.k_base, p.delta_role)
    k = k_rrb.copy()
    T = len(k)
    score = np.full(T, np.nan)
    group = np.zeros(T, dtype=np.int64)
    ranked = np.zeros(T, dtype=bool)
    key = ranking_key(p.signal, conf_prev1, conf_prev2, hist_len, p.theta, p.w_cf, p.v_ref, p.tau)
    b = np.asarray(block_idx)
    msk = np.asarray(masked).astype(bool)
    hist = np.asarray(hist_len)
    k_cur = p.k_base + p.delta_role
    so = np.asarray(seq_offsets)
    for s in range(len(so) - 1):
        lo, hi = int(so[s]), int(so[s + 1])
        idx = np.arange(lo, hi)
        J = idx[msk[lo:hi] & (b[lo:hi] == int(active_block[s]))]
        Jp = J[hist[J] >= 1]
        # every token of J starts at K_cur (its RRB count, since d = 0)
        k[J] = k_cur
        if len(Jp) == 0:
            continue
        g = fger_groups(key[Jp], Jp, p.q)
        k[Jp] = k_cur + p.delta_cur * g
        score[Jp] = key[Jp]
        group[Jp] = g
        ranked[Jp] = True
    k_unclamped = k.copy()
    k = np.minimum(np.maximum(k, p.k_min), p.k_max)
    return BudgetResult(k, k_unclamped, k_rrb, score, group, ranked)


# ---------------------------------------------------------------------------------------
# decoding state between denoising forwards (Section 3.1, Eq. (1))
# ---------------------------------------------------------------------------------------
@dataclass
class StateResult:
    masked: np.ndarray        # [T] uint8
    hist_len: np.ndarray      # [T] int8
    conf_prev1: np.ndarray    # [T] float32, c^{t} after the update (the new c^{t-1})
    conf_prev2: np.ndarray    # [T] float32
    active_block: np.ndarray  # [B] int32
    committed: np.ndarray     # [T] bool, positions committed by this forward
    remaining: np.ndarray     # [B] masked positions left in each sequence


def advance_state(block_idx, masked, hist_len, conf_prev1, conf_prev2, seq_offsets,
                  active_block, conf_t, theta: float, min_commit: int = 0) -> StateResult:
    """One forward's commitment and bookkeeping, per sequence.

    Confidence-threshold commitment (Eq. (1)): the committed set is the masked
    positions of the active block whose confidence reaches theta.  With
    min_commit = 1, a forward that would commit nothing commits the single most
    confident such position instead (lowest position on ties), a common guard
    for progress that the paper does not state.  Every position that was masked
    when the forward ran records its new confidence: c^{t-2} <- c^{t-1},
    c^{t-1} <- c^t, history length capped at 2.  When no masked position is left
    in the active block, the sequence moves to the next block (if any)."""
    b = np.asarray(block_idx, dtype=np.int64)
    m = np.asarray(masked).astype(np.uint8).copy()
    h = np.asarray(hist_len).astype(np.int8).copy()
    c1 = np.asarray(conf_prev1, dtype=np.float32).copy()
    c2 = np.asarray(conf_prev2, dtype=np.float32).copy()
    ct = np.asarray(conf_t, dtype=np.float32)
    a = np.asarray(active_block, dtype=np.int32).copy()
    th = np.float32(theta)
    T = len(b)
    committed = np.zeros(T, dtype=bool)
    remaining = np.zeros(len(a), dtype=np.int64)
    for s in range(len(a)):
        lo, hi = int(seq_offsets[s]), int(seq_offsets[s + 1])
        idx = np.arange(lo, hi)
        was_masked = idx[m[lo:hi] == 1]
        J = was_masked[b[was_masked] == a[s]]
        C = J[ct[J] >= th]
        if min_commit and len(C) == 0 and len(J) > 0:
            best = J[np.lexsort((J, -ct[J].astype(np.float64)))[0]]
            C = np.array([best])
        c2[was_masked] = c1[was_masked]
        c1[was_masked] = ct[was_masked]
        h[was_masked] = np.minimum(h[was_masked].astype(np.int64) + 1, 2).astype(np.int8)
        m[C] = 0
        committed[C] = True
        last_block = int(b[lo:hi].max()) if hi > lo else int(a[s])
        left_in_active = int(((m[lo:hi] == 1) & (b[lo:hi] == a[s])).sum())
        if left_in_active == 0 and a[s] < last_block:
            a[s] += 1
        remaining[s] = int(m[lo:hi].sum())
    return StateResult(m, h, c1, c2, a, committed, remaining)


# ---------------------------------------------------------------------------------------
# variable-count token-choice routing (Section 3.2, Eq. (2))
# ---------------------------------------------------------------------------------------
@dataclass
class RouteResult:
    offsets: np.ndarray   # [T+1] exclusive prefix of k
    expert: np.ndarray    # [P] selected experts, token-major, in rank order
    token: np.ndarray     # [P] owning token of each pair
    weight: np.ndarray    # [P] alpha_{i,e}, fp64


def topk_route(r: np.ndarray, k: np.ndarray, norm_topk: int = 1) -> RouteResult:
    """T_i = TopK_e(r_{i,e}, k_i) with experts ordered by (score desc, index asc),
    and the normalised router weight alpha over the selected experts.

    norm_topk = 1: alpha_e = exp(r_e - r_max) / sum_{e' in T_i} exp(r_e' - r_max);
    norm_topk = 0: the same numerator over the sum over all E experts."""
    r = np.asarray(r, dtype=np.float64)
    T, E = r.shape
    k = np.asarray(k, dtype=np.int64)
    offs = np.zeros(T + 1, dtype=np.int64)
    offs[1:] = np.cumsum(k)
    P = int(offs[-1])
    ex = np.zeros(P, dtype=np.int64)
    tok = np.zeros(P, dtype=np.int64)
    wt = np.zeros(P, dtype=np.float64)
    e_idx = np.arange(E)
    for i in range(T):
        ki = int(k[i])
        if ki == 0:
            continue
        row = r[i] + 0.0                       # -0.0 -> +0.0
        order = np.lexsort((e_idx, -row))      # score descending, index ascending
        sel = order[:ki]
        rmax = row[order[0]]
        num = np.exp(row[sel] - rmax)
        den = num.sum() if norm_topk else np.exp(row - rmax).sum()
        lo = offs[i]
        ex[lo:lo + ki] = sel
        tok[lo:lo + ki] = i
        wt[lo:lo + ki] = num / den
    return RouteResult(offs, ex, tok, wt)


# ---------------------------------------------------------------------------------------
# score-derived count rules compared in Appendix B (Top-p, Expert-Threshold Routing)
# ---------------------------------------------------------------------------------------
def router_probs(r: np.ndarray) -> np.ndarray:
    """Routing mass of every expert: the softmax of the router scores over all E
    experts, fp64.  r: [T,E]."""
    r = np.asarray(r, dtype=np.float64)
    ex = np.exp(r - r.max(axis=1, keepdims=True))
    return ex / ex.sum(axis=1, keepdims=True)


def topp_counts(r: np.ndarray, p: float, k_min: int, k_max: int):
    """Top-p (Appendix B): the smallest number of router-ranked experts (score
    descending, index ascending) whose cumulative routing mass reaches p, clamped to
    [k_min, k_max].  Returns (k, cum) where cum[i] is the cumulative mass of the
    unclamped prefix (for margin checks)."""
    r = np.asarray(r, dtype=np.float64)
    T, E = r.shape
    prob = router_probs(r)
    pp = _p64(p)
    k = np.zeros(T, dtype=np.int64)
    cum_at = np.zeros(T, dtype=np.float64)
    e_idx = np.arange(E)
    for i in range(T):
        order = np.lexsort((e_idx, -(r[i] + 0.0)))
        cum = 0.0
        n = E
        for j, e in enumerate(order):
            cum += prob[i, e]
            if cum >= pp:
                n = j + 1
                break
        k[i] = min(max(n, k_min), k_max)
        cum_at[i] = cum
    return k, cum_at


def threshold_counts(r: np.ndarray, tau: float, k_min: int, k_max: int) -> np.ndarray:
    """Expert-Threshold Routing (Appendix B): the number of experts whose routing mass
    exceeds tau, clamped to [k_min, k_max]."""
    prob = router_probs(r)
    n = (prob > _p64(tau)).sum(axis=1)
    return np.clip(n, k_min, k_max).astype(np.int64)


@dataclass
class PermResult:
    expert_offsets: np.ndarray  # [E+1]
    sorted_token: np.ndarray    # [P] token of the pair at each expert-sorted row
    pair_to_sorted: np.ndarray  # [P] row of pair j in expert-sorted order


def pair_permutation(pair_token: np.ndarray, pair_expert: np.ndarray, E: int) -> PermResult:
    """Group the P = sum_i k_i expert-token pairs by expert: rows sorted by
    (expert ascending, token ascending)."""
    pair_token = np.asarray(pair_token, dtype=np.int64)
    pair_expert = np.asarray(pair_expert, dtype=np.int64)
    order = np.lexsort((pair_token, pair_expert))
    counts = np.bincount(pair_expert, minlength=E) if len(pair_expert) else np.zeros(E, np.int64)
    eo = np.zeros(E + 1, dtype=np.int64)
    eo[1:] = np.cumsum(counts)
    p2s = np.empty(len(order), dtype=np.int64)
    p2s[order] = np.arange(len(order))
    return PermResult(eo, pair_token[order], p2s)


# ---------------------------------------------------------------------------------------
# experts and the combine (Eq. (2); SwiGLU expert of Appendix A)
# ---------------------------------------------------------------------------------------
def swiglu_expert(x: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray) -> np.ndarray:
    """E(x) = W_d (SiLU(W_g x) * (W_u x)), SiLU(g) = g * sigma(g); rows of x are tokens.
    Weights are fp64 arrays in [out, in] layout."""
    g = x @ wg.T
    u = x @ wu.T
    a = g * sigmoid(g) * u
    return a @ wd.T


def _expert_f64(weights_of, e):
    wg, wu, wd = weights_of(e)
    return bf16_to_f64(wg), bf16_to_f64(wu), bf16_to_f64(wd)


def moe_layer(h_bits: np.ndarray, route: RouteResult, weights_of, E: int,
              shared=None, tokens: Optional[Sequence[int]] = None) -> np.ndarray:
    """MoE(h_i) = sum_{e in T_i} alpha_{i,e} E_e(h_i)  (Eq. (2)), fp64.

    ``weights_of(e)`` returns the bf16 bit arrays (W_g [f,d], W_u [f,d], W_d [d,f])
    of expert e.  ``shared`` is an optional always-on expert (same triple) added
    with weight 1.  ``tokens`` restricts the output to a subset of tokens (rows of
    the result follow that subset); all experts those tokens selected are run."""
    T = len(route.offsets) - 1
    toks = np.arange(T) if tokens is None else np.asarray(tokens, dtype=np.int64)
    x_all = bf16_to_f64(h_bits[toks])
    out = np.zeros((len(toks), h_bits.shape[1]), dtype=np.float64)
    pos_of = {int(t): j for j, t in enumerate(toks)}
    # pairs of the requested tokens, grouped by expert
    sel_pairs = np.concatenate([np.arange(route.offsets[t], route.offsets[t + 1]) for t in toks]
                               ) if len(toks) else np.zeros(0, np.int64)
    sel_pairs = sel_pairs.astype(np.int64)
    experts = np.unique(route.expert[sel_pairs]) if len(sel_pairs) else []
    contrib = {}
    for e in experts:
        pe = sel_pairs[route.expert[sel_pairs] == e]
        rows = np.array([pos_of[int(t)] for t in route.token[pe]], dtype=np.int64)
        wg, wu, wd = _expert_f64(weights_of, int(e))
        y = swiglu_expert(x_all[rows], wg, wu, wd)
        for j, pj in enumerate(pe):
            contrib[int(pj)] = y[j]
    # weighted sum in slot (rank) order for each token
    for j, t in enumerate(toks):
        for pj in range(int(route.offsets[t]), int(route.offsets[t + 1])):
            out[j] += route.weight[pj] * contrib[pj]
    if shared is not None:
        sg, su, sd = (bf16_to_f64(w) for w in shared)
        out += swiglu_expert(x_all, sg, su, sd)
    return out


def dense_masked_moe(h_bits: np.ndarray, r: np.ndarray, k: np.ndarray, weights_of, E: int,
                     norm_topk: int = 1, shared=None) -> np.ndarray:
    """A second formulation of the same layer: run every expert on every token,
    build the selection mask from the score ranking, and sum mask * alpha * E_e(h)
    over all experts.  Used to pin ``moe_layer`` (small sizes only)."""
    x = bf16_to_f64(h_bits)
    r = np.asarray(r, dtype=np.float64) + 0.0
    T = x.shape[0]
    # rank of each expert for each token under (score desc, index asc): count of
    # experts that beat it
    beats = (r[:, None, :] > r[:, :, None]) | (
        (r[:, None, :] == r[:, :, None]) & (np.arange(E)[None, None, :] < np.arange(E)[None, :, None]))
    rank = beats.sum(axis=2)                                  # [T, E]
    mask = rank < np.asarray(k)[:, None]
    ex = np.exp(r - r.max(axis=1, keepdims=True))
    den = (ex * mask).sum(axis=1, keepdims=True) if norm_topk else ex.sum(axis=1, keepdims=True)
    den = np.where(den == 0, 1.0, den)
    alpha = np.where(mask, ex / den, 0.0)
    out = np.zeros((T, x.shape[1]), dtype=np.float64)
    for e in range(E):
        wg, wu, wd = _expert_f64(weights_of, e)
        out += alpha[:, e:e + 1] * swiglu_expert(x, wg, wu, wd)
    if shared is not None:
        sg, su, sd = (bf16_to_f64(w) for w in shared)
        out += swiglu_expert(x, sg, su, sd)
    return out


def fixed_topk_moe(h_bits: np.ndarray, r: np.ndarray, K: int, weights_of, E: int) -> np.ndarray:
    """Default fixed token-choice routing written on its own: every token takes the
    K best-scoring experts (stable sort, so equal scores keep index order) with
    softmax weights renormalised over those K."""
    x = bf16_to_f64(h_bits)
    r = np.asarray(r, dtype=np.float64)
    T = x.shape[0]
    top = np.argsort(-r, axis=1, kind="stable")[:, :K]
    out = np.zeros((T, x.shape[1]), dtype=np.float64)
    ys = {}
    for e in range(E):
        wg, wu, wd = _expert_f64(weights_of, e)
        ys[e] = swiglu_expert(x, wg, wu, wd)
    for i in range(T):
        s = r[i, top[i]]
        w = np.exp(s - s.max())
        w = w / w.sum()
        for j in range(K):
            out[i] += w[j] * ys[int(top[i, j])][i]
    return out


def routed_expert_flops(d: int, f: int, pairs: int) -> int:
    """Routed-expert linear FLOPs, 6 * h * d_exp * pairs (Appendix A, Eq. (10))."""
    return 6 * int(d) * int(f) * int(pairs)
