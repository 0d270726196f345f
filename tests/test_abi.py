"""The C-ABI library loads, exports every entry point include/reflex.h declares,
agrees with the binding on struct layouts, and rejects invalid arguments on the
host before launching anything (so these run without a GPU)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from conftest import ROOT

_lib = pytest.importorskip("paper_2608_01784_amd._lib")

HEADER = os.path.join(ROOT, "include", "reflex.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libreflex.so is not built (python -m paper_2608_01784_amd.build)")
    return _lib.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(reflex_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 14
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (reflex_[a-z0-9_]+)$", out, flags=re.M))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        assert hasattr(L, n)


def test_binding_covers_every_entry_point():
    assert set(declared_functions()) == set(_lib._SIGS)


def test_struct_layouts_and_version(L):
    assert L.reflex_sizeof_moe_args() == ctypes.sizeof(_lib.MoeArgsC)
    assert L.reflex_sizeof_alloc_params() == ctypes.sizeof(_lib.AllocParamsC) == 44
    assert L.reflex_version() >= 100
    for rc in (0, -1, -2, -3, -4, -5, -6, 7):
        assert isinstance(_lib.status_string(rc), str)


def test_workspace_sizes(L):
    T, E, d, f, k = 1024, 64, 2048, 1024, 12
    ws = L.reflex_workspace_size(T, E, d, f, 0, k)
    cap = T * k
    # dominant terms: expert outputs [cap, d] and activations [cap, f] in bf16
    assert ws >= cap * d * 2 + cap * f * 2 + T * E * 4
    assert ws < (cap * d * 2 + cap * f * 2 + T * E * 4) * 1.05 + (1 << 20)
    assert L.reflex_workspace_size(T, E, d, f, 512, k) >= ws + T * d * 2 + T * 512 * 2
    assert L.reflex_workspace_size(T, E, d, f, 0, k) >= L.reflex_permute_workspace_size(cap, E)
    assert L.reflex_workspace_size(T, E, d, f, 0, k) >= L.reflex_swiglu_workspace_size(cap, E, f)
    # invalid shapes -> 0
    assert L.reflex_workspace_size(T, 300, d, f, 0, k) == 0      # E > 256
    assert L.reflex_workspace_size(T, E, 200, f, 0, k) == 0      # d % 128
    assert L.reflex_workspace_size(T, E, d, 100, 0, k) == 0      # f % 64
    assert L.reflex_workspace_size(T, 8, d, f, 0, 9) == 0        # k_max > E
    assert L.reflex_workspace_size(T, E, d, f, 0, 33) == 0       # k_max > 32
    assert L.reflex_permute_workspace_size(-1, E) == 0


def test_workspace_offsets_lie_inside_the_workspace(L):
    T, E, d, f, k = 1000, 64, 2048, 1024, 12
    ws = L.reflex_workspace_size(T, E, d, f, 0, k)
    cap = T * k
    sizes = {0: 4 * (T + 1), 1: 4 * cap, 2: 4 * cap, 3: 4 * (E + 1), 4: 4 * cap, 5: 4 * cap}
    spans = []
    for field, n in sizes.items():
        off = L.reflex_workspace_offset(T, E, d, f, 0, k, field)
        assert off % 256 == 0 and off + n <= ws, field
        spans.append((off, off + n))
    spans.sort()
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))     # no two arrays overlap
    bad = ctypes.c_size_t(-1).value
    assert L.reflex_workspace_offset(T, E, d, f, 0, k, 6) == bad
    assert L.reflex_workspace_offset(T, 300, d, f, 0, k, 0) == bad


FAKE = 1 << 20           # 16-byte aligned stand-in address, never dereferenced
MIS = FAKE + 4           # 4-byte aligned only: invalid for vector-accessed data
ODD = FAKE + 2           # invalid for any 4-byte element type


def good_params(**kw):
    p = dict(k_base=8, delta_role=4, delta_cur=2, k_min=2, k_max=12, q=0.25, theta=0.9,
             w_cf=0.3, v_ref=0.01, tau=0.05, signal=0)
    p.update(kw)
    return _lib.AllocParamsC(*[p[n] for n, _ in _lib.AllocParamsC._fields_])


def test_router_validation(L):
    f = L.reflex_router_logits
    assert f(None, FAKE, None, FAKE, 16, 256, 8, None) == -1
    assert f(FAKE, FAKE, None, None, 16, 256, 8, None) == -1
    assert f(FAKE, FAKE, None, FAKE, 16, 200, 8, None) == -2
    assert f(FAKE, FAKE, None, FAKE, 16, 256, 0, None) == -2
    assert f(FAKE, FAKE, None, FAKE, 16, 256, 257, None) == -2
    assert f(MIS, FAKE, None, FAKE, 16, 256, 8, None) == -2
    assert f(FAKE, FAKE, ODD, FAKE, 16, 256, 8, None) == -2
    assert f(FAKE, FAKE, None, ODD, 16, 256, 8, None) == -2
    assert f(FAKE, MIS, None, FAKE, 16, 256, 8, None) == -2     # fp32 weight read as float4
    assert f(FAKE, FAKE, None, FAKE, 0, 256, 8, None) == 0      # empty: nothing launched


@pytest.mark.parametrize("field,value", [
    ("q", 0.0), ("q", 0.51), ("tau", 0.0), ("tau", -1.0), ("w_cf", 0.0), ("theta", float("nan")),
    ("v_ref", float("inf")), ("k_min", 13), ("k_max", 33), ("k_min", -1), ("delta_cur", -1),
    ("delta_role", -2), ("k_base", -1), ("signal", 5), ("signal", -1)])
def test_budget_rejects_bad_parameters(L, field, value):
    p = good_params(**{field: value})
    rc = L.reflex_assign_budget(*([FAKE] * 7), 1, 16, ctypes.byref(p), FAKE, FAKE, None, None)
    assert rc == -3


def test_budget_validation(L):
    p = good_params()
    f = L.reflex_assign_budget
    assert f(*([FAKE] * 7), 1, 16, None, FAKE, FAKE, None, None) == -1
    assert f(*([FAKE] * 6), None, 1, 16, ctypes.byref(p), FAKE, FAKE, None, None) == -1
    assert f(*([FAKE] * 7), 1, 16, ctypes.byref(p), FAKE, None, None, None) == -1
    assert f(*([FAKE] * 7), 0, 16, ctypes.byref(p), FAKE, FAKE, None, None) == -2   # T > 0, B = 0
    assert f(*([FAKE] * 7), 1, -1, ctypes.byref(p), FAKE, FAKE, None, None) == -2
    assert f(*([FAKE] * 7), 1, 16, ctypes.byref(p), FAKE, FAKE, MIS, None) == -2
    assert f(*([FAKE] * 7), 0, 0, ctypes.byref(p), FAKE, FAKE, None, None) == 0


def test_topk_validation(L):
    f = L.reflex_topk_variable
    assert f(FAKE, FAKE, 16, 8, 4, 1, FAKE, FAKE, None, 64, None) == -1
    assert f(FAKE, FAKE, 16, 8, 9, 1, FAKE, FAKE, FAKE, 200, None) == -2     # k_max > E
    assert f(FAKE, FAKE, 16, 64, 33, 1, FAKE, FAKE, FAKE, 9999, None) == -2  # k_max > 32
    assert f(FAKE, FAKE, 16, 8, 4, 2, FAKE, FAKE, FAKE, 64, None) == -3      # norm_topk
    assert f(FAKE, FAKE, 16, 8, 4, 1, FAKE, FAKE, FAKE, 63, None) == -4      # capacity < T k_max
    assert f(FAKE, FAKE, 0, 8, 4, 1, FAKE, FAKE, FAKE, 0, None) == 0


@pytest.mark.parametrize("preset,field,value", [
    ("full", None, None), ("rrb_only", "delta_cur", 0), ("fger_only", "delta_role", 0),
    ("frontier_only", "signal", 1), ("progress_only", "signal", 2), ("confidence_only", "signal", 3),
    ("uncertainty_only", "signal", 4)])
def test_alloc_presets_hold_the_paper_settings(L, preset, field, value):
    # Section 5.1: K_base 8, delta_role 4, delta_cur 2, q 0.25, theta 0.9, v_ref 0.01, tau 0.05
    from paper_2608_01784_amd import _lib
    p = _lib.reflex_alloc_preset(preset, 2, 12, 0.30)
    expect = {"k_base": 8, "delta_role": 4, "delta_cur": 2, "k_min": 2, "k_max": 12, "signal": 0}
    if field is not None:
        expect[field] = value
    for k, v in expect.items():
        assert getattr(p, k) == v, k
    f32 = lambda x: float(np.float32(x))  # noqa: E731
    assert (p.q, p.theta, p.w_cf, p.v_ref, p.tau) == (0.25, f32(0.9), f32(0.30), f32(0.01), f32(0.05))


def test_alloc_preset_validation(L):
    from paper_2608_01784_amd import _lib
    out = _lib.AllocParamsC()
    assert L.reflex_alloc_preset(7, 2, 12, 0.3, ctypes.byref(out)) == -3
    assert L.reflex_alloc_preset(0, 2, 12, 0.3, None) == -1
    assert L.reflex_alloc_preset(0, 13, 12, 0.3, ctypes.byref(out)) == -3
    assert L.reflex_alloc_preset(0, 2, 12, 0.0, ctypes.byref(out)) == -3     # w_cf > 0


def test_advance_state_validation(L):
    f = L.reflex_advance_state
    assert f(None, FAKE, FAKE, 1, 16, 0.9, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -1
    assert f(FAKE, FAKE, FAKE, 1, 16, 0.9, 0, FAKE, FAKE, ODD, FAKE, FAKE, None, None) == -2
    assert f(FAKE, FAKE, FAKE, 0, 16, 0.9, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -2  # B < 1
    assert f(FAKE, FAKE, FAKE, 1, 16, 0.0, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -3  # theta
    assert f(FAKE, FAKE, FAKE, 1, 16, 1.5, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -3
    assert f(FAKE, FAKE, FAKE, 1, 16, 0.9, 2, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -3  # min_commit
    assert f(FAKE, FAKE, FAKE, 0, 0, 0.9, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == 0


def test_count_rule_validation(L):
    f = L.reflex_count_rule
    assert f(None, 16, 8, 1, 0.2, 1, 4, FAKE, None, None) == -1
    assert f(FAKE, 16, 8, 1, 0.2, 1, 4, ODD, None, None) == -2          # misaligned k_out
    assert f(FAKE, 16, 8, 3, 0.2, 1, 4, FAKE, None, None) == -3         # unknown rule
    assert f(FAKE, 16, 8, 0, 0.2, 1, 4, FAKE, None, None) == -3         # the budget is not a rule
    assert f(FAKE, 16, 8, 1, 0.0, 1, 4, FAKE, None, None) == -3         # p must be > 0
    assert f(FAKE, 16, 8, 1, 1.5, 1, 4, FAKE, None, None) == -3
    assert f(FAKE, 16, 8, 2, 1.0, 1, 4, FAKE, None, None) == -3         # tau must be < 1
    assert f(FAKE, 16, 8, 2, float("nan"), 1, 4, FAKE, None, None) == -3
    assert f(FAKE, 16, 8, 1, 0.2, 5, 4, FAKE, None, None) == -2         # k_min > k_max
    assert f(FAKE, 16, 8, 1, 0.2, 1, 9, FAKE, None, None) == -2         # k_max > E
    assert f(FAKE, 0, 8, 2, 0.02, 1, 4, FAKE, None, None) == 0


def test_permute_swiglu_combine_validation(L):
    cap, E, f_ = 64, 8, 128
    need = L.reflex_permute_workspace_size(cap, E)
    assert L.reflex_permute(FAKE, FAKE, FAKE, 16, E, cap, FAKE, FAKE, FAKE, FAKE, need - 1, None) == -4
    assert L.reflex_permute(FAKE, FAKE, None, 16, E, cap, FAKE, FAKE, FAKE, FAKE, need, None) == -1
    # a 4-byte-aligned scalar (e.g. pair_offsets + T) is a valid pair-count pointer
    assert L.reflex_permute(FAKE, FAKE, MIS, 16, E, cap, FAKE, FAKE, FAKE, FAKE, need - 1, None) == -4
    assert L.reflex_permute(FAKE, FAKE, ODD, 16, E, cap, FAKE, FAKE, FAKE, FAKE, need, None) == -2
    assert L.reflex_permute(FAKE, FAKE, FAKE, 16, E, cap, FAKE, FAKE, FAKE, MIS, need, None) == -2
    assert L.reflex_permute(FAKE, FAKE, FAKE, 16, 0, cap, FAKE, FAKE, FAKE, FAKE, need, None) == -2
    need = L.reflex_swiglu_workspace_size(cap, E, f_)
    g = L.reflex_grouped_swiglu
    assert g(*([FAKE] * 6), 16, E, 256, f_, cap, FAKE, FAKE, need - 1, None) == -4
    assert g(*([FAKE] * 6), 16, E, 256, 100, cap, FAKE, FAKE, need, None) == -2
    assert g(*([FAKE] * 6), 16, E, 250, f_, cap, FAKE, FAKE, need, None) == -2
    assert g(*([FAKE] * 5), None, 16, E, 256, f_, cap, FAKE, FAKE, need, None) == -1
    c = L.reflex_combine
    assert c(FAKE, FAKE, FAKE, None, None, 16, 256, cap, FAKE, None) == -1
    assert c(FAKE, FAKE, FAKE, FAKE, MIS, 16, 256, cap, FAKE, None) == -2
    assert c(FAKE, FAKE, FAKE, FAKE, None, 16, 96, cap, FAKE, None) == -2
    assert c(FAKE, FAKE, FAKE, FAKE, None, 0, 256, cap, FAKE, None) == 0


def _args(**kw):
    a = _lib.MoeArgsC()
    a.T, a.d, a.E, a.f, a.f_shared, a.norm_topk, a.uniform_k, a.B = 16, 256, 8, 128, 0, 1, 0, 1
    for n in _lib._ARG_PTRS:
        setattr(a, n, FAKE)
    a.router_bias = None
    a.k_in = None
    a.residual_a = a.residual_b = None
    a.ws_gate = a.ws_up = a.ws_down = None
    a.params = good_params(k_max=4, k_min=1, k_base=2, delta_role=1, delta_cur=1)
    a.out = FAKE
    a.k_out = a.pairs_out = a.logits_out = None
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def test_moe_forward_validation(L):
    f = L.reflex_moe_forward
    ws_need = L.reflex_workspace_size(16, 8, 256, 128, 0, 4)
    assert f(ctypes.byref(_args()), FAKE, ws_need - 1, None) == -4
    assert f(ctypes.byref(_args(h=None)), FAKE, ws_need, None) == -1
    assert f(ctypes.byref(_args(masked=None)), FAKE, ws_need, None) == -1      # budget path needs state
    assert f(ctypes.byref(_args(f_shared=128)), FAKE, 1 << 30, None) == -1     # shared weights missing
    assert f(ctypes.byref(_args(d=200)), FAKE, ws_need, None) == -2
    assert f(ctypes.byref(_args(norm_topk=3)), FAKE, ws_need, None) == -3
    assert f(ctypes.byref(_args(uniform_k=9)), FAKE, 1 << 30, None) == -2      # uniform_k > E
    assert f(ctypes.byref(_args(B=0)), FAKE, ws_need, None) == -2
    bad = _args()
    bad.params.q = 0.7
    assert f(ctypes.byref(bad), FAKE, ws_need, None) == -3
    assert f(ctypes.byref(_args(T=0)), FAKE, ws_need, None) == 0
    assert f(None, FAKE, ws_need, None) == -1


def test_product_path_has_no_cpu_fallback():
    # the package must not import the oracle anywhere
    pkg = os.path.join(ROOT, "paper_2608_01784_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith(".py"):
                src = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in src, fn
