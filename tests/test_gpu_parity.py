"""GPU parity: every entry point of libreflex (through the C ABI) against the fp64
oracle on the same seeded inputs.

Bars: counts, TopK indices, pair offsets and the permutation are bit-exact;
router logits within 1e-4 of the row's largest |logit|; routing weights within
1e-5 relative; layer outputs within relative L2 1e-2 and max-abs 2e-2.
"""
from __future__ import annotations

import functools

import numpy as np
import pytest

import oracle
from gpu_common import layer_tolerance_check, note, oracle_budget, require_gpu
from synth import AllocParams, Workload, make_fuzz_workload, make_workload
from synth.device import bf16_bits, state_tensors, to_device

pytestmark = pytest.mark.gpu

SMALL = ["tiny_t128_e8", "tiny_roles_t128_e8"]
FULL = ["lladamoe_t1024_e64", "llada2mini_t4096_e256", "skewed_t16384_e256"]
FUZZ = list(range(12))


@pytest.fixture(scope="module")
def torch():
    return require_gpu()


@functools.lru_cache(maxsize=None)
def workload(name) -> Workload:
    if name.startswith("fuzz"):
        return make_fuzz_workload(int(name[4:]))
    return make_workload(name)


@functools.lru_cache(maxsize=4)
def host_weights(name, layer=0):
    w = workload(name)
    return {"w_gate": w.w_gate(layer), "w_up": w.w_up(layer), "w_down": w.w_down(layer),
            "w_router": w.w_router(layer), "shared": w.shared_weights(layer)}


@functools.lru_cache(maxsize=4)
def dev_weights(name, layer=0):
    hw = host_weights(name, layer)
    w = workload(name)
    d = {k: to_device(hw[k]) for k in ("w_gate", "w_up", "w_down", "w_router")}
    d["router_bias"] = None if w.router_bias is None else to_device(w.router_bias)
    if hw["shared"] is not None:
        d["ws_gate"], d["ws_up"], d["ws_down"] = (to_device(x) for x in hw["shared"])
    return d


def weights_of(name, layer=0):
    hw = host_weights(name, layer)
    return lambda e: (hw["w_gate"][e], hw["w_up"][e], hw["w_down"][e])


def _lib():
    from paper_2608_01784_amd import _lib as L
    return L


def gpu_logits(torch, name):
    w = workload(name)
    dw = dev_weights(name)
    logits = torch.empty((w.T, w.E), dtype=torch.float32, device="cuda")
    _lib().reflex_router_logits(to_device(w.h), dw["w_router"], dw["router_bias"], logits)
    torch.cuda.synchronize()
    return logits


# ----------------------------------------------------------------------------- router
@pytest.mark.parametrize("name", SMALL + FULL + [f"fuzz{s}" for s in FUZZ])
def test_router_logits(torch, name):
    w = workload(name)
    got = gpu_logits(torch, name).cpu().numpy().astype(np.float64)
    ref = oracle.router_scores(w.h, host_weights(name)["w_router"], w.router_bias)
    scale = np.abs(ref).max(axis=1, keepdims=True)
    err = np.abs(got - ref) / np.maximum(scale, 1e-30)
    note(f"{name}: max row-relative logit error {err.max():.3e}")
    assert err.max() <= 1e-4


@pytest.mark.parametrize("T,d,E,with_bias", [(4100, 384, 100, True), (4096, 128, 8, False),
                                             (9000, 128, 37, False), (8200, 512, 60, True),
                                             (16400, 128, 250, False), (20000, 256, 200, True)])
def test_router_logits_large_t(torch, T, d, E, with_bias):
    # T >= 4096: the LDS-staged kernel with 32 x 64 tiles (first three cases), the
    # register kernel with 32-token tiles for at most 64 experts and d a multiple of 256
    # (fourth), the LDS-staged kernel with 128 x 64 tiles where those number 512 or more
    # (last two); ragged last token tile and expert counts that are not a multiple of
    # the 64-expert tile
    w = make_fuzz_workload(300 + T % 97, T=T, d=d, E=E, f=64)
    rng = np.random.default_rng([T, d, E])
    bias = (rng.standard_normal(E) * 0.5).astype(np.float32) if with_bias else None
    wr = w.w_router()
    logits = torch.empty((T, E), dtype=torch.float32, device="cuda")
    _lib().reflex_router_logits(to_device(w.h), to_device(wr),
                                None if bias is None else to_device(bias), logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy().astype(np.float64)
    ref = oracle.router_scores(w.h, wr, bias)
    err = np.abs(got - ref) / np.maximum(np.abs(ref).max(axis=1, keepdims=True), 1e-30)
    note(f"router T={T} d={d} E={E}: max row-relative logit error {err.max():.3e}")
    assert err.max() <= 1e-4


# ----------------------------------------------------------------------------- budget
def gpu_budget(torch, w: Workload, params=None):
    p = w.params if params is None else params
    st = state_tensors(w)
    k = torch.full((w.T,), -7, dtype=torch.int32, device="cuda")
    pairs = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    fps = torch.empty((w.T,), dtype=torch.float64, device="cuda")
    _lib().reflex_assign_budget(st["block_idx"], st["masked"], st["hist_len"], st["conf_prev1"],
                                st["conf_prev2"], st["seq_offsets"], st["active_block"], p, k,
                                pairs, fps)
    torch.cuda.synchronize()
    return k.cpu().numpy(), int(pairs.item()), fps.cpu().numpy()


def check_budget(torch, w, params=None):
    p = w.params if params is None else params
    k, pairs, fps = gpu_budget(torch, w, p)
    ref = oracle_budget(w, p)
    # ranking keys: same fp64 formula; exp may differ in the last ulp
    ranked = ref.ranked
    assert np.array_equal(np.isnan(fps), ~ranked)
    if ranked.any():
        np.testing.assert_allclose(fps[ranked], ref.score[ranked], rtol=4e-16 * 8, atol=1e-300)
    if not np.array_equal(k, ref.k):
        # a disagreement is only acceptable when two keys are within rounding of
        # each other; re-rank with the GPU's keys to confirm the integer logic
        bad = np.nonzero(k != ref.k)[0]
        note(f"{w.name}: {len(bad)} counts differ; re-ranking with GPU keys")
        for s in range(w.B):
            lo, hi = w.seq_offsets[s], w.seq_offsets[s + 1]
            idx = np.arange(lo, hi)[ranked[lo:hi]]
            if len(idx):
                g = oracle.fger_groups(fps[idx], idx, p.q)
                kk = np.clip(p.k_base + p.delta_role + p.delta_cur * g, p.k_min, p.k_max)
                assert np.array_equal(k[idx], kk)
        pytest.fail(f"{w.name}: counts differ from the oracle at {bad[:10]}")
    assert pairs == int(ref.k.sum())
    return k, ref


@pytest.mark.parametrize("name", SMALL + FULL + [f"fuzz{s}" for s in range(30)])
def test_budget_counts_bit_exact(torch, name):
    check_budget(torch, workload(name))


@pytest.mark.parametrize("signal", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("name", ["llada2mini_t4096_e256", "fuzz3", "fuzz7"])
def test_budget_ranking_signals(torch, name, signal):
    w = workload(name)
    check_budget(torch, w, w.params.replace(signal=signal))


@pytest.mark.parametrize("preset", ["full", "rrb_only", "fger_only", "frontier_only",
                                    "progress_only", "confidence_only", "uncertainty_only"])
@pytest.mark.parametrize("name", ["lladamoe_t1024_e64", "llada2mini_t4096_e256", "fuzz5"])
def test_budget_paper_presets(torch, name, preset):
    # the library's presets, converted to the oracle's parameters field by field
    w = workload(name)
    c = _lib().reflex_alloc_preset(preset, w.params.k_min, w.params.k_max, w.params.w_cf)
    p = AllocParams.make(c.k_base, c.delta_role, c.delta_cur, c.k_min, c.k_max, q=c.q,
                         theta=c.theta, w_cf=c.w_cf, v_ref=c.v_ref, tau=c.tau).replace(signal=c.signal)
    k, ref = check_budget(torch, w, p)
    if preset == "rrb_only":          # no reallocation: the clamped role budget
        assert np.array_equal(k, np.clip(ref.k_rrb, p.k_min, p.k_max))
    if preset == "fger_only" and p.k_max >= 10 and p.k_min <= 6:
        assert int(k.sum()) == 8 * w.T            # FGER alone preserves the budget


@pytest.mark.parametrize("active", [1, 2, 3, 9, 15, 16])
def test_budget_every_role_position(torch, active):
    check_budget(torch, make_workload("lladamoe_t1024_e64", active=active))


def _long_sequence_workload(seed, n_masked, n_prompt=300, extra_seqs=3):
    """One sequence whose active block holds thousands of masked tokens (several LDS
    slices of the ranking), followed by short sequences, one of them empty."""
    rng = np.random.default_rng(seed)
    blk = n_masked + 17
    b = np.concatenate([np.zeros(n_prompt, np.int32), np.full(blk, 1, np.int32),
                        np.full(blk, 2, np.int32)])
    m = np.zeros(len(b), np.uint8)
    m[n_prompt + rng.choice(blk, n_masked, replace=False)] = 1
    m[n_prompt + blk:] = 1
    offs = [0, len(b)]
    acts = [1]
    bs, ms = [b], [m]
    for j in range(extra_seqs):
        L = 0 if j == 1 else 40
        bs.append(np.repeat(np.arange(0, 5, dtype=np.int32), 8)[:L])
        ms.append((rng.random(L) < 0.7).astype(np.uint8))
        acts.append(2)
        offs.append(offs[-1] + L)
    b = np.concatenate(bs)
    m = np.concatenate(ms)
    T = len(b)
    c1 = rng.random(T).astype(np.float32)
    c2 = np.clip(c1 - rng.uniform(-0.2, 0.3, T).astype(np.float32), 0, 1).astype(np.float32)
    c1[::97] = c1[5]          # exact key ties
    c2[::97] = c2[5]
    hist = rng.choice(np.array([0, 1, 2, 2], np.int8), T)
    p = AllocParams.make(8, 4, 2, 1, 16, q=0.25)
    return Workload(f"long{n_masked}", seed, T, 128, 8, 64, 0, 1, p, np.zeros((T, 128), np.uint16),
                    b, np.array(offs, np.int32), np.array(acts, np.int32), m, hist, c1, c2)


@pytest.mark.parametrize("n_masked", [63, 64, 65, 2047, 2048, 2049, 5000])
def test_budget_long_active_block(torch, n_masked):
    check_budget(torch, _long_sequence_workload(n_masked, n_masked))


# ------------------------------------------------------------------------ TopK + alpha
def gpu_topk(torch, logits, k, k_max, norm):
    T, E = logits.shape
    cap = T * k_max
    off = torch.full((T + 1,), -7, dtype=torch.int32, device="cuda")
    ex = torch.full((max(cap, 1),), -7, dtype=torch.int32, device="cuda")
    wt = torch.full((max(cap, 1),), float("nan"), dtype=torch.float32, device="cuda")
    _lib().reflex_topk_variable(logits, k, k_max, norm, off, ex[:cap] if cap else ex, wt[:cap] if cap else wt)
    torch.cuda.synchronize()
    return off.cpu().numpy(), ex.cpu().numpy(), wt.cpu().numpy()


def check_topk(torch, logits_dev, k_np, k_max, norm):
    k_dev = to_device(k_np.astype(np.int32))
    off, ex, wt = gpu_topk(torch, logits_dev, k_dev, k_max, norm)
    r = logits_dev.cpu().numpy().astype(np.float64)
    ref = oracle.topk_route(r, np.clip(k_np, 0, k_max), norm)
    P = int(ref.offsets[-1])
    assert np.array_equal(off, ref.offsets)
    assert np.array_equal(ex[:P], ref.expert)
    if P:
        rel = np.abs(wt[:P] - ref.weight) / np.abs(ref.weight)
        note(f"alpha max rel err {rel.max():.3e}")
        assert rel.max() <= 1e-5
    return off, ex, wt


@pytest.mark.parametrize("norm", [1, 0])
@pytest.mark.parametrize("name", SMALL + FULL + [f"fuzz{s}" for s in FUZZ])
def test_topk_bit_exact(torch, name, norm):
    w = workload(name)
    k = oracle_budget(w).k
    check_topk(torch, gpu_logits(torch, name), k, w.params.k_max, norm)


@pytest.mark.parametrize("E,k_max", [(8, 8), (64, 12), (256, 32), (255, 32), (1, 1), (100, 7)])
def test_topk_ties_zeros_and_extremes(torch, E, k_max):
    rng = np.random.default_rng(E)
    T = 300
    r = (rng.integers(-2, 3, (T, E)) * 0.25).astype(np.float32)   # many exact ties
    r[::7] = 0.0
    r[::14, ::2] = -0.0                                            # -0.0 ties +0.0
    r[3] = np.float32(-3.4e38)
    r[4, :] = np.float32(1e30)
    k = rng.integers(-3, k_max + 4, T).astype(np.int32)          # clamped to [0, k_max]
    k[:5] = k_max
    check_topk(torch, to_device(r), k, k_max, 1)
    check_topk(torch, to_device(r), k, k_max, 0)


# ------------------------------------------------------------------------ permutation
def gpu_permute(torch, off, ex, T, E, cap):
    L = _lib()
    off_d = to_device(off.astype(np.int32))
    ex_d = to_device(np.pad(ex[: int(off[-1])], (0, cap - int(off[-1])),
                            constant_values=-5).astype(np.int32))
    pairs = off_d[T:T + 1]
    eo = torch.full((E + 1,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((cap,), -7, dtype=torch.int32, device="cuda")
    p2s = torch.full((cap,), -7, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(L.reflex_permute_workspace_size(cap, E), 256), dtype=torch.uint8,
                     device="cuda")
    L.reflex_permute(off_d, ex_d, pairs, E, eo, st, p2s, ws)
    torch.cuda.synchronize()
    return eo.cpu().numpy(), st.cpu().numpy(), p2s.cpu().numpy()


def check_permute(torch, off, ex, T, E, cap):
    eo, st, p2s = gpu_permute(torch, off, ex, T, E, cap)
    P = int(off[-1])
    tok = np.repeat(np.arange(T), np.diff(off))
    ref = oracle.pair_permutation(tok, ex[:P], E)
    assert np.array_equal(eo, ref.expert_offsets)
    assert np.array_equal(st[:P], ref.sorted_token)
    assert np.array_equal(p2s[:P], ref.pair_to_sorted)
    assert np.all(st[P:] == -7) and np.all(p2s[P:] == -7)      # nothing written past P


@pytest.mark.parametrize("name", SMALL + FULL + [f"fuzz{s}" for s in FUZZ])
def test_permute_bit_exact(torch, name):
    w = workload(name)
    k = oracle_budget(w).k
    route = oracle.topk_route(gpu_logits(torch, name).cpu().numpy().astype(np.float64), k)
    check_permute(torch, route.offsets, route.expert, w.T, w.E, w.T * w.params.k_max)


@pytest.mark.parametrize("T,E,kind", [(1, 1, "one"), (5000, 3, "skew"), (9000, 256, "one_expert"),
                                      (4097, 17, "ragged"), (300, 256, "sparse")])
def test_permute_skewed_and_ragged(torch, T, E, kind):
    rng = np.random.default_rng(T + E)
    kmax = min(E, 4)
    k = rng.integers(0, kmax + 1, T)
    if kind == "one_expert":
        k[:] = 1
    r = rng.standard_normal((T, E))
    if kind in ("skew", "one_expert"):
        r[:, 0] += 100.0
    route = oracle.topk_route(r, k)
    check_permute(torch, route.offsets, route.expert, T, E, T * kmax)


# --------------------------------------------------------------------- SwiGLU experts
def gpu_swiglu(torch, name, eo, st, cap):
    L = _lib()
    w = workload(name)
    dw = dev_weights(name)
    y = torch.full((cap, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.reflex_swiglu_workspace_size(cap, w.E, w.f), dtype=torch.uint8, device="cuda")
    L.reflex_grouped_swiglu(to_device(w.h), to_device(st.astype(np.int32)),
                            to_device(eo.astype(np.int32)), dw["w_gate"], dw["w_up"], dw["w_down"],
                            y, ws)
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("name", SMALL + FULL + ["fuzz1", "fuzz4", "fuzz9"])
def test_grouped_swiglu(torch, name):
    w = workload(name)
    k = oracle_budget(w).k
    route = oracle.topk_route(gpu_logits(torch, name).cpu().numpy().astype(np.float64), k)
    perm = oracle.pair_permutation(route.token, route.expert, w.E)
    cap = w.T * w.params.k_max
    st = np.zeros(cap, np.int64)
    st[:len(perm.sorted_token)] = perm.sorted_token
    ybits = bf16_bits(gpu_swiglu(torch, name, perm.expert_offsets, st, cap))
    eo = perm.expert_offsets
    counts = np.diff(eo)
    # all experts at small sizes; at full size the largest, the smallest nonempty and a
    # seeded sample of the rest
    nz = np.nonzero(counts)[0]
    if len(nz) > 24:
        rng = np.random.default_rng(0)
        pick = set(rng.choice(nz, 20, replace=False).tolist())
        pick |= {int(nz[np.argmax(counts[nz])]), int(nz[np.argmin(counts[nz])])}
        nz = sorted(pick)
    wo = weights_of(name)
    got, ref = [], []
    for e in nz:
        rows = np.arange(eo[e], eo[e + 1])
        if len(rows) > 512:
            rows = rows[np.linspace(0, len(rows) - 1, 512).astype(int)]
        wg, wu, wd = (oracle.bf16_to_f64(a) for a in wo(e))
        x = oracle.bf16_to_f64(w.h[perm.sorted_token[rows]])
        ref.append(oracle.swiglu_expert(x, wg, wu, wd))
        got.append(oracle.bf16_to_f64(ybits[rows]))
    layer_tolerance_check(np.concatenate(got), np.concatenate(ref), f"{name} experts")
    P = int(eo[-1])
    assert np.isnan(oracle.bf16_to_f64(ybits[P:P + 256])).all()    # rows past P untouched


@pytest.mark.parametrize("seed", range(10))
def test_tall_swiglu_fuzz(torch, seed):
    # The 256-row tile kernels (chosen where experts average 512 pair rows or more at
    # capacity) on seeded random shapes: ragged and empty experts, expert sizes at tile
    # edges, partial last N tiles (d % 256 = 128 in the down GEMM, f % 128 = 64 in the up
    # GEMM), a single K step in the down GEMM (f = 64) and a gather with repeated tokens;
    # every row of every expert against the fp64 definition, rows past P untouched.
    from synth.workloads import bf16_bits_from_f32
    L = _lib()
    rng = np.random.default_rng([seed, 2608])
    E = int(rng.choice([1, 2, 3, 5]))
    d = int(rng.choice([128, 256, 384, 640]))
    f = int(rng.choice([64, 128, 192, 320]))
    T = int(rng.integers(64, 1200))
    counts = rng.integers(0, 1300, E)
    counts[rng.integers(0, E)] = rng.choice([0, 1, 255, 256, 257, 511, 512, 513])
    P = int(counts.sum())
    cap = max(P, 512 * E)
    eo = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    st = np.zeros(cap, np.int32)
    st[:P] = rng.integers(0, T, P)

    def bf16(shape, scale):
        return bf16_bits_from_f32((rng.standard_normal(shape) * scale).astype(np.float32))

    h = bf16((T, d), 1.0)
    wg, wu = bf16((E, f, d), d ** -0.5), bf16((E, f, d), d ** -0.5)
    wd = bf16((E, d, f), 0.3 * f ** -0.5)
    y = torch.full((cap, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.reflex_swiglu_workspace_size(cap, E, f), dtype=torch.uint8, device="cuda")
    L.reflex_grouped_swiglu(to_device(h), to_device(st), to_device(eo), to_device(wg),
                            to_device(wu), to_device(wd), y, ws)
    torch.cuda.synchronize()
    yb = bf16_bits(y)
    got, ref = [], []
    for e in range(E):
        rows = np.arange(eo[e], eo[e + 1])
        if len(rows):
            x = oracle.bf16_to_f64(h[st[rows]])
            ref.append(oracle.swiglu_expert(x, oracle.bf16_to_f64(wg[e]), oracle.bf16_to_f64(wu[e]),
                                            oracle.bf16_to_f64(wd[e])))
            got.append(oracle.bf16_to_f64(yb[rows]))
    what = f"tall fuzz {seed}: E={E} T={T} d={d} f={f} counts={counts.tolist()}"
    if got:
        layer_tolerance_check(np.concatenate(got), np.concatenate(ref), what)
    assert np.isnan(oracle.bf16_to_f64(yb[P:])).all(), what


# --------------------------------------------------------------------------- combine
@pytest.mark.parametrize("with_shared", [False, True])
@pytest.mark.parametrize("T,d,E,kmax", [(1, 128, 4, 2), (333, 256, 16, 6), (1024, 2048, 64, 12),
                                        (64, 256, 32, 32),     # up to 32 pairs: two batches of rows
                                        (40, 256, 96, 80),     # > 64 pairs: the per-pair loop
                                        (4100, 256, 32, 20)])  # T >= 4096: batches of 8 rows
def test_combine(torch, T, d, E, kmax, with_shared):
    L = _lib()
    rng = np.random.default_rng(T)
    k = rng.integers(0, kmax + 1, T)
    route = oracle.topk_route(rng.standard_normal((T, E)), k)
    perm = oracle.pair_permutation(route.token, route.expert, E)
    cap = T * kmax
    P = int(k.sum())
    from synth.workloads import bf16_bits_from_f32
    y = bf16_bits_from_f32(rng.standard_normal((cap, d)).astype(np.float32) * 0.3)
    sh = bf16_bits_from_f32(rng.standard_normal((T, d)).astype(np.float32)) if with_shared else None
    wt = route.weight.astype(np.float32)
    p2s = np.zeros(cap, np.int32)
    p2s[:P] = perm.pair_to_sorted
    wpad = np.zeros(cap, np.float32)
    wpad[:P] = wt
    out = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    L.reflex_combine(to_device(y), to_device(route.offsets.astype(np.int32)), to_device(p2s),
                     to_device(wpad), None if sh is None else to_device(sh), out)
    torch.cuda.synchronize()
    got = oracle.bf16_to_f64(bf16_bits(out))
    yv = oracle.bf16_to_f64(y)
    ref = np.zeros((T, d))
    for i in range(T):
        for j in range(route.offsets[i], route.offsets[i + 1]):
            ref[i] += float(wt[j]) * yv[perm.pair_to_sorted[j]]
    if sh is not None:
        ref += oracle.bf16_to_f64(sh)
    # only the final bf16 rounding (and fp32 accumulation) separates the two
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-6)


# ------------------------------------------------------------------------ fused layer
def fused(torch, name, layer=0, uniform_k=0, k_in=None, norm_topk=1):
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    w = workload(name)
    dw = dev_weights(name, layer)
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params, uniform_k=uniform_k, norm_topk=norm_topk)
    out = lay.forward(to_device(w.h), TokenState(**state_tensors(w)),
                      k_in=None if k_in is None else to_device(k_in.astype(np.int32)))
    torch.cuda.synchronize()
    return (oracle.bf16_to_f64(bf16_bits(out)), lay.k.cpu().numpy(), int(lay.pairs.item()),
            lay.logits.cpu().numpy().astype(np.float64))


def sample_tokens(w, n=256):
    if w.T <= 1200:
        return None
    return np.sort(np.random.default_rng(1).choice(w.T, n, replace=False))


def compare_layer(name, out, k, logits, norm_topk=1, tag=""):
    w = workload(name)
    hw = host_weights(name)
    toks = sample_tokens(w)
    rows = slice(None) if toks is None else toks
    # (i) selection pinned: the oracle routes from the GPU's fp32 logits
    route = oracle.topk_route(logits, k, norm_topk)
    ref = oracle.moe_layer(w.h, route, weights_of(name), w.E, shared=hw["shared"], tokens=toks)
    layer_tolerance_check(out[rows], ref, f"{name}{tag} (selection pinned)")
    # (ii) independent: the oracle's own fp64 logits; tokens whose selected set differs
    # must be explained by a logit margin below the router tolerance
    r_or = oracle.router_scores(w.h, hw["w_router"], w.router_bias)
    # the forward's own scores (split-K partials added by the route kernel on the fused
    # router + budget path) within the router tolerance of the fp64 scores, per row
    err = np.abs(logits - r_or).max(axis=1)
    assert np.all(err <= 1e-4 * np.abs(r_or).max(axis=1)), float((err / np.abs(r_or).max(axis=1)).max())
    route_i = oracle.topk_route(r_or, k, norm_topk)
    ref_i = oracle.moe_layer(w.h, route_i, weights_of(name), w.E, shared=hw["shared"], tokens=toks)
    tl = np.arange(w.T) if toks is None else toks
    same = np.array([set(route.expert[route.offsets[t]:route.offsets[t + 1]]) ==
                     set(route_i.expert[route_i.offsets[t]:route_i.offsets[t + 1]]) for t in tl])
    for j in np.nonzero(~same)[0]:
        t = tl[j]
        srt = np.sort(r_or[t])[::-1]
        kk = int(k[t])
        margin = srt[kk - 1] - srt[kk] if 0 < kk < w.E else np.inf
        assert margin <= 1e-4 * np.abs(r_or[t]).max(), (t, margin)
    note(f"{name}{tag}: {int((~same).sum())} of {len(tl)} tokens select differently (near ties)")
    layer_tolerance_check(out[rows][same], ref_i[same], f"{name}{tag} (independent)")


@pytest.mark.parametrize("name", SMALL + FULL + ["fuzz0", "fuzz2", "fuzz5", "fuzz8"])
def test_fused_forward(torch, name):
    w = workload(name)
    out, k, pairs, logits = fused(torch, name)
    ref_b = oracle_budget(w)
    assert np.array_equal(k, ref_b.k)
    assert pairs == ref_b.pairs
    compare_layer(name, out, k, logits)


@pytest.mark.parametrize("name", SMALL + ["lladamoe_t1024_e64"])
def test_fused_full_softmax(torch, name):
    out, k, _, logits = fused(torch, name, norm_topk=0)
    compare_layer(name, out, k, logits, norm_topk=0, tag=" norm0")


@pytest.mark.parametrize("name", SMALL + ["lladamoe_t1024_e64", "llada2mini_t4096_e256"])
def test_uniform_path_is_fixed_topk(torch, name):
    w = workload(name)
    K = w.params.k_base
    out, k, pairs, logits = fused(torch, name, uniform_k=K)
    assert np.all(k == K) and pairs == K * w.T
    compare_layer(name, out, k, logits, tag=" uniform")


def test_reused_counts_and_zero_count_tokens(torch):
    name = "tiny_t128_e8"
    w = workload(name)
    k = np.random.default_rng(5).integers(0, w.params.k_max + 1, w.T)
    k[:10] = 0
    out, _, pairs, logits = fused(torch, name, k_in=k)
    assert pairs == int(k.sum())
    assert np.all(out[:10] == 0.0)
    compare_layer(name, out, k, logits, tag=" k_in")


def test_reused_counts_clamped_to_uniform_capacity(torch):
    # uniform_k > 0 sets the pair capacity (T * uniform_k) even when counts are passed in;
    # the caller's counts are then clamped to uniform_k
    name = "tiny_t128_e8"
    w = workload(name)
    k = np.random.default_rng(6).integers(0, w.params.k_max + 1, w.T)
    out, _, pairs, logits = fused(torch, name, uniform_k=2, k_in=k)
    kc = np.minimum(k, 2)
    assert pairs == int(kc.sum())
    compare_layer(name, out, kc, logits, tag=" k_in clamped")


def test_deterministic(torch):
    name = "llada2mini_t4096_e256"
    a = fused(torch, name)
    b = fused(torch, name)
    for x, y in zip(a, b):
        assert np.array_equal(np.asarray(x), np.asarray(y))


@pytest.mark.parametrize("seed,E,kmax,T", [(101, 1, 1, 77), (102, 256, 32, 500), (103, 2, 2, 1),
                                           (104, 64, 12, 1537)])
def test_fused_edge_shapes(torch, seed, E, kmax, T):
    w = make_fuzz_workload(seed, T=T, d=128, E=E, f=64, k_max=kmax)
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()),
          "router_bias": None if w.router_bias is None else to_device(w.router_bias)}
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params)
    out = lay.forward(to_device(w.h), TokenState(**state_tensors(w)))
    torch.cuda.synchronize()
    out = oracle.bf16_to_f64(bf16_bits(out))
    k = lay.k.cpu().numpy()
    assert np.array_equal(k, oracle_budget(w).k)
    route = oracle.topk_route(lay.logits.cpu().numpy().astype(np.float64), k)
    wg, wu, wd = w.w_gate(), w.w_up(), w.w_down()
    ref = oracle.moe_layer(w.h, route, lambda e: (wg[e], wu[e], wd[e]), w.E)
    layer_tolerance_check(out, ref, f"edge E={E} k_max={kmax} T={T}")


@pytest.mark.parametrize("seed,T,d,E,f,kmax", [(110, 1100, 256, 4, 192, 3), (111, 3000, 128, 8, 64, 4),
                                                (112, 700, 384, 1, 128, 1)])
def test_fused_many_rows_per_expert(torch, seed, T, d, E, f, kmax):
    # few experts with many pairs each: every expert spans several 128-row M tiles
    # with a ragged last one; f = 192 also leaves a partial last N tile in the up GEMM
    w = make_fuzz_workload(seed, T=T, d=d, E=E, f=f, k_max=kmax)
    assert w.T * w.params.k_max // w.E >= 512
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()),
          "router_bias": None if w.router_bias is None else to_device(w.router_bias)}
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params)
    out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), TokenState(**state_tensors(w)))))
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    assert np.array_equal(k, oracle_budget(w).k)
    route = oracle.topk_route(lay.logits.cpu().numpy().astype(np.float64), k)
    wg, wu, wd = w.w_gate(), w.w_up(), w.w_down()
    ref = oracle.moe_layer(w.h, route, lambda e: (wg[e], wu[e], wd[e]), w.E)
    layer_tolerance_check(out, ref, f"many rows per expert T={T} d={d} E={E} f={f}")


@pytest.mark.parametrize("E", [16, 2])
def test_one_expert_takes_every_token(torch, E):
    # a huge router bias sends every token to expert 1: one expert with T rows spans many
    # M tiles, every other expert is empty.
    w = make_fuzz_workload(200, T=2000, d=256, E=E, f=128, k_max=1)
    w.router_bias = np.zeros(E, np.float32)
    w.router_bias[1] = 1e4
    w.params = w.params.replace(k_min=1, k_max=1)
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()), "router_bias": to_device(w.router_bias)}
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params)
    out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), TokenState(**state_tensors(w)))))
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    assert np.all(k == 1)
    route = oracle.topk_route(lay.logits.cpu().numpy().astype(np.float64), k)
    assert np.all(route.expert == 1)
    wg, wu, wd = w.w_gate(), w.w_up(), w.w_down()
    ref = oracle.moe_layer(w.h, route, lambda e: (wg[e], wu[e], wd[e]), w.E)
    layer_tolerance_check(out, ref, "one expert")


def _fuzz_layer(torch, w, k_in=None):
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    dw = {"w_gate": to_device(w.w_gate()), "w_up": to_device(w.w_up()), "w_down": to_device(w.w_down()),
          "w_router": to_device(w.w_router()),
          "router_bias": None if w.router_bias is None else to_device(w.router_bias)}
    lay = MoELayer(w.T, w.d, ExpertWeights(**dw), w.params)
    return lay, TokenState(**state_tensors(w))


def _fuzz_ref(w, logits, k):
    route = oracle.topk_route(logits, k)
    wg, wu, wd = w.w_gate(), w.w_up(), w.w_down()
    return oracle.moe_layer(w.h, route, lambda e: (wg[e], wu[e], wd[e]), w.E)


@pytest.mark.parametrize("T", [4096, 4112])
def test_fused_route_sort_limit(torch, T):
    # the fused forward sorts the pairs inside its route launch while (16-token blocks) x
    # experts <= 16384 (T = 4096, E = 64: exactly the limit, 256 workgroups) and with the
    # block-sort launches above it (T = 4112)
    w = make_fuzz_workload(120, T=T, d=128, E=64, f=64, k_max=12)
    lay, st = _fuzz_layer(torch, w)
    out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), st)))
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    assert np.array_equal(k, oracle_budget(w).k)
    assert int(lay.pairs.item()) == int(k.sum())
    ref = _fuzz_ref(w, lay.logits.cpu().numpy().astype(np.float64), k)
    layer_tolerance_check(out, ref, f"route sort limit T={T}")


def _fused_routing(torch, lay, w):
    """The fused forward's own pair list and permutation, read from its workspace."""
    from paper_2608_01784_amd import _lib as L
    cap = w.T * lay.kcap
    args = (w.T, w.E, w.d, w.f, w.f_shared, lay.kcap)

    def arr(field, n, dtype):
        off = L.reflex_workspace_offset(*args, field)
        return lay.ws[off:off + 4 * n].cpu().numpy().view(dtype)

    return {"pair_offsets": arr("pair_offsets", w.T + 1, np.int32),
            "pair_expert": arr("pair_expert", cap, np.int32),
            "pair_weight": arr("pair_weight", cap, np.float32),
            "expert_offsets": arr("expert_offsets", w.E + 1, np.int32),
            "sorted_token": arr("sorted_token", cap, np.int32),
            "pair_to_sorted": arr("pair_to_sorted", cap, np.int32)}


@pytest.mark.parametrize("case", ["tiny_t128_e8", "tiny_roles_t128_e8", "lladamoe_t1024_e64",
                                  "T4096", "T4112", "T8192", "T5003E96", "T16384E256",
                                  "T65536E16", "T4096E256D2048", "T2000E256D2048"])
def test_fused_route_and_permutation_bit_exact(torch, case):
    # the fused forward's TopK pair list and permutation against the oracle's TopK and
    # permutation on the forward's own fp32 scores: sorted inside the route launch for
    # layers up to 16384 (16-token block, expert) counts (the tiny and LLaDA-MoE layers,
    # T = 4096 at E = 64), by the block-sort launches above (T = 4112, the 16-layer
    # stack's T = 8192 at E = 64, a ragged T = 5003 at E = 96, the skewed layer's
    # T = 16384 at E = 256 with up to 16 experts a token, and T = 65536 at E = 16: four
    # 1024-block chunks per expert column).  At d = 2048 the route kernel adds split-K
    # partial scores as it loads them, here with four slots of experts a lane: the
    # router's 4 K slices at T = 4096, the front kernel's 8 at T = 2000.
    import re
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    if case.startswith("T"):
        m = re.fullmatch(r"T(\d+)(?:E(\d+))?(?:D(\d+))?", case)
        T, E, d = int(m[1]), int(m[2] or 64), int(m[3] or 128)
        w = make_fuzz_workload(120, T=T, d=d, E=E, f=64, k_max=16 if E >= 16 else E)
        lay, st = _fuzz_layer(torch, w)
    else:
        w = workload(case)
        lay = MoELayer(w.T, w.d, ExpertWeights(**dev_weights(case)), w.params)
        st = TokenState(**state_tensors(w))
    lay.forward(to_device(w.h), st)
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    got = _fused_routing(torch, lay, w)
    route = oracle.topk_route(lay.logits.cpu().numpy().astype(np.float64), k)
    P = int(route.offsets[-1])
    assert int(lay.pairs.item()) == P
    assert np.array_equal(got["pair_offsets"], route.offsets)
    assert np.array_equal(got["pair_expert"][:P], route.expert)
    np.testing.assert_allclose(got["pair_weight"][:P], route.weight, rtol=1e-5, atol=0)
    ref = oracle.pair_permutation(route.token, route.expert, w.E)
    assert np.array_equal(got["expert_offsets"], ref.expert_offsets)
    assert np.array_equal(got["sorted_token"][:P], ref.sorted_token)
    assert np.array_equal(got["pair_to_sorted"][:P], ref.pair_to_sorted)
    note(f"{case}: P={P} pairs, TopK and permutation bit-exact")


@pytest.mark.parametrize("T", [700, 4400])
def test_fused_consecutive_calls_and_no_pairs(torch, T):
    # the sort's completion counter (the route launch's at T = 700, the block sort's at
    # T = 4400) is re-armed by every forward: three forwards in a row on one workspace,
    # with caller counts that differ (the last one all zero, P = 0: an all-zero output),
    # each checked against the oracle
    w = make_fuzz_workload(121, T=T, d=256, E=16 if T < 1000 else 64, f=128, k_max=6)
    lay, st = _fuzz_layer(torch, w)
    rng = np.random.default_rng(7)
    for n, k in enumerate([rng.integers(0, 7, w.T), rng.integers(0, 3, w.T), np.zeros(w.T, np.int64)]):
        out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), st,
                                                       k_in=to_device(k.astype(np.int32)))))
        torch.cuda.synchronize()
        assert int(lay.pairs.item()) == int(k.sum()), n
        if k.sum() == 0:
            assert np.all(out == 0.0)
            continue
        ref = _fuzz_ref(w, lay.logits.cpu().numpy().astype(np.float64), k)
        layer_tolerance_check(out, ref, f"consecutive call {n}")


@pytest.mark.parametrize("seed,T,d,E", [(130, 333, 1024, 100), (134, 95, 512, 256), (132, 1000, 768, 64)])
def test_fused_split_router_partials(torch, seed, T, d, E):
    # on the fused router + budget path the scores come out as d/256 partial sums that
    # the route kernel adds in slice order, with the bias: several slices (3 of them
    # for d = 768), expert blocks past 64 with E off a multiple of 64, token counts off
    # the 32-token tile, several sequences, a router bias
    import dataclasses
    w = make_fuzz_workload(seed, T=T, d=d, E=E, f=128, k_max=min(E, 8))
    if w.router_bias is None:
        bias = (np.random.default_rng(seed).standard_normal(E) * 0.5).astype(np.float32)
        w = dataclasses.replace(w, router_bias=bias)
    assert len(w.seq_offsets) > 2
    lay, st = _fuzz_layer(torch, w)
    out = oracle.bf16_to_f64(bf16_bits(lay.forward(to_device(w.h), st)))
    torch.cuda.synchronize()
    k = lay.k.cpu().numpy()
    assert np.array_equal(k, oracle_budget(w).k)
    logits = lay.logits.cpu().numpy().astype(np.float64)
    r_or = oracle.router_scores(w.h, w.w_router(), w.router_bias)
    err = np.abs(logits - r_or).max(axis=1)
    assert np.all(err <= 1e-4 * np.abs(r_or).max(axis=1)), float((err / np.abs(r_or).max(axis=1)).max())
    layer_tolerance_check(out, _fuzz_ref(w, logits, k), f"split router T={T} d={d} E={E}")
