"""ctypes binding of libreflex.so: argument marshalling only.

Every function below has the name of the C entry point it calls, takes torch
tensors (device memory) and the current HIP stream, and raises ReflexError on a
negative status.  No step of the layer is computed here.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import c_double, c_float, c_int, c_int32, c_size_t, c_void_p

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libreflex.so")

_lib = None


class ReflexError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: status {status} ({status_string(status)})")


class AllocParamsC(ctypes.Structure):
    _fields_ = [("k_base", c_int32), ("delta_role", c_int32), ("delta_cur", c_int32),
                ("k_min", c_int32), ("k_max", c_int32), ("q", c_float), ("theta", c_float),
                ("w_cf", c_float), ("v_ref", c_float), ("tau", c_float), ("signal", c_int32)]


_ARG_PTRS = ["h", "w_gate", "w_up", "w_down", "ws_gate", "ws_up", "ws_down", "w_router",
             "router_bias", "block_idx", "seq_offsets", "active_block", "masked", "hist_len",
             "conf_prev1", "conf_prev2", "k_in", "residual_a", "residual_b"]
_OUT_PTRS = ["out", "k_out", "pairs_out", "logits_out"]


class MoeArgsC(ctypes.Structure):
    _fields_ = ([(n, c_int32) for n in ("T", "d", "E", "f", "f_shared", "norm_topk", "uniform_k", "B",
                                        "k_rule")]
                + [("k_threshold", ctypes.c_float)]
                + [(n, c_void_p) for n in _ARG_PTRS]
                + [("params", AllocParamsC)]
                + [(n, c_void_p) for n in _OUT_PTRS])


_SIGS = {
    "reflex_version": (c_int, []),
    "reflex_status_string": (ctypes.c_char_p, [c_int]),
    "reflex_sizeof_alloc_params": (c_size_t, []),
    "reflex_sizeof_moe_args": (c_size_t, []),
    "reflex_workspace_size": (c_size_t, [c_int] * 6),
    "reflex_permute_workspace_size": (c_size_t, [c_int, c_int]),
    "reflex_workspace_offset": (c_size_t, [c_int] * 7),
    "reflex_swiglu_workspace_size": (c_size_t, [c_int, c_int, c_int]),
    "reflex_router_logits": (c_int, [c_void_p] * 4 + [c_int] * 3 + [c_void_p]),
    "reflex_assign_budget": (c_int, [c_void_p] * 7 + [c_int, c_int, ctypes.POINTER(AllocParamsC)]
                             + [c_void_p] * 4),
    "reflex_alloc_preset": (c_int, [c_int, c_int, c_int, ctypes.c_float, ctypes.POINTER(AllocParamsC)]),
    "reflex_advance_state": (c_int, [c_void_p] * 3 + [c_int, c_int, ctypes.c_float, c_int]
                             + [c_void_p] * 7),
    "reflex_count_rule": (c_int, [c_void_p, c_int, c_int, c_int, ctypes.c_float, c_int, c_int,
                                  c_void_p, c_void_p, c_void_p]),
    "reflex_topk_variable": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_int, c_void_p,
                                     c_void_p, c_void_p, c_int32, c_void_p]),
    "reflex_permute": (c_int, [c_void_p] * 3 + [c_int, c_int, c_int32] + [c_void_p] * 4
                       + [c_size_t, c_void_p]),
    "reflex_grouped_swiglu": (c_int, [c_void_p] * 6 + [c_int] * 4 + [c_int32, c_void_p, c_void_p,
                                                                     c_size_t, c_void_p]),
    "reflex_combine": (c_int, [c_void_p] * 5 + [c_int, c_int, c_int32, c_void_p, c_void_p]),
    "reflex_moe_forward": (c_int, [ctypes.POINTER(MoeArgsC), c_void_p, c_size_t, c_void_p]),
    "reflex_moe_forward_timed": (c_int, [ctypes.POINTER(MoeArgsC), c_void_p, c_size_t, c_void_p,
                                         ctypes.POINTER(c_void_p), c_int]),
    "reflex_moe_forward_noalloc": (c_int, [ctypes.POINTER(MoeArgsC), c_void_p]),
}

N_STAGE_EVENTS = 9
STAGES = ("router", "counts", "topk", "permute", "gemm_up", "gemm_down", "shared", "combine")


def lib():
    """The loaded library; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_01784_amd.build`")
        # torch first: its HIP runtime (same soname) is then the one libreflex binds
        # to, so streams and events are shared by one runtime in the process
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        if L.reflex_sizeof_moe_args() != ctypes.sizeof(MoeArgsC) or \
                L.reflex_sizeof_alloc_params() != ctypes.sizeof(AllocParamsC):
            raise RuntimeError("libreflex ABI struct layout does not match the binding")
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().reflex_status_string(status).decode()


def _check(rc: int, where: str):
    if rc != 0:
        raise ReflexError(rc, where)


def ptr(t):
    """Device address of a tensor (or None / a raw integer address)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def stream_handle(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def alloc_params(p) -> AllocParamsC:
    """AllocParamsC from any object with the hyper-parameter attributes."""
    return AllocParamsC(int(p.k_base), int(p.delta_role), int(p.delta_cur), int(p.k_min),
                        int(p.k_max), float(p.q), float(p.theta), float(p.w_cf), float(p.v_ref),
                        float(p.tau), int(getattr(p, "signal", 0)))


# --------------------------------------------------------------------------------------
# entry points
# --------------------------------------------------------------------------------------
def reflex_workspace_size(T, E, d, f, f_shared, k_max) -> int:
    return lib().reflex_workspace_size(T, E, d, f, f_shared, k_max)


def reflex_permute_workspace_size(pair_capacity, E) -> int:
    return lib().reflex_permute_workspace_size(pair_capacity, E)


def reflex_swiglu_workspace_size(pair_capacity, E, f) -> int:
    return lib().reflex_swiglu_workspace_size(pair_capacity, E, f)


def reflex_router_logits(h, w_router, bias, logits, stream=None):
    T, d = h.shape
    E = w_router.shape[0]
    _check(lib().reflex_router_logits(ptr(h), ptr(w_router), ptr(bias), ptr(logits), T, d, E,
                                      stream_handle(stream)), "reflex_router_logits")


def reflex_assign_budget(block_idx, masked, hist_len, conf_prev1, conf_prev2, seq_offsets,
                         active_block, params, k_out, pairs_out, fps_out=None, stream=None):
    T = block_idx.shape[0]
    B = active_block.shape[0]
    prm = alloc_params(params)
    _check(lib().reflex_assign_budget(ptr(block_idx), ptr(masked), ptr(hist_len), ptr(conf_prev1),
                                      ptr(conf_prev2), ptr(seq_offsets), ptr(active_block), B, T,
                                      ctypes.byref(prm), ptr(k_out), ptr(pairs_out), ptr(fps_out),
                                      stream_handle(stream)), "reflex_assign_budget")


def reflex_advance_state(conf_t, block_idx, seq_offsets, theta, min_commit, masked, hist_len,
                         conf_prev1, conf_prev2, active_block, remaining=None, stream=None):
    T = block_idx.shape[0]
    B = active_block.shape[0]
    _check(lib().reflex_advance_state(ptr(conf_t), ptr(block_idx), ptr(seq_offsets), B, T, theta,
                                      min_commit, ptr(masked), ptr(hist_len), ptr(conf_prev1),
                                      ptr(conf_prev2), ptr(active_block), ptr(remaining),
                                      stream_handle(stream)), "reflex_advance_state")


RULE_BUDGET, RULE_TOP_P, RULE_THRESHOLD = 0, 1, 2
PRESETS = ("full", "rrb_only", "fger_only", "frontier_only", "progress_only", "confidence_only",
           "uncertainty_only")


def reflex_alloc_preset(preset, k_min, k_max, w_cf) -> AllocParamsC:
    """The paper's hyper-parameters for a named or numbered preset (host only)."""
    idx = PRESETS.index(preset) if isinstance(preset, str) else int(preset)
    out = AllocParamsC()
    _check(lib().reflex_alloc_preset(idx, k_min, k_max, w_cf, ctypes.byref(out)),
           "reflex_alloc_preset")
    return out


def reflex_count_rule(logits, rule, threshold, k_min, k_max, k_out, pairs_out=None, stream=None):
    T, E = logits.shape
    _check(lib().reflex_count_rule(ptr(logits), T, E, rule, threshold, k_min, k_max, ptr(k_out),
                                   ptr(pairs_out), stream_handle(stream)), "reflex_count_rule")


def reflex_topk_variable(logits, k, k_max, norm_topk, pair_offsets, pair_expert, pair_weight,
                         stream=None):
    T, E = logits.shape
    cap = pair_expert.shape[0]
    _check(lib().reflex_topk_variable(ptr(logits), ptr(k), T, E, k_max, norm_topk,
                                      ptr(pair_offsets), ptr(pair_expert), ptr(pair_weight), cap,
                                      stream_handle(stream)), "reflex_topk_variable")


def reflex_permute(pair_offsets, pair_expert, pairs, E, expert_offsets, sorted_token,
                   pair_to_sorted, ws, stream=None):
    T = pair_offsets.shape[0] - 1
    cap = pair_expert.shape[0]
    _check(lib().reflex_permute(ptr(pair_offsets), ptr(pair_expert), ptr(pairs), T, E, cap,
                                ptr(expert_offsets), ptr(sorted_token), ptr(pair_to_sorted),
                                ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)),
           "reflex_permute")


def reflex_grouped_swiglu(h, sorted_token, expert_offsets, w_gate, w_up, w_down, y_sorted, ws,
                          stream=None):
    T, d = h.shape
    E, f, _ = w_gate.shape
    cap = y_sorted.shape[0]
    _check(lib().reflex_grouped_swiglu(ptr(h), ptr(sorted_token), ptr(expert_offsets), ptr(w_gate),
                                       ptr(w_up), ptr(w_down), T, E, d, f, cap, ptr(y_sorted),
                                       ptr(ws), ws.numel() * ws.element_size(),
                                       stream_handle(stream)), "reflex_grouped_swiglu")


def reflex_combine(y_sorted, pair_offsets, pair_to_sorted, pair_weight, shared_y, out, stream=None):
    T, d = out.shape
    cap = pair_to_sorted.shape[0]
    _check(lib().reflex_combine(ptr(y_sorted), ptr(pair_offsets), ptr(pair_to_sorted),
                                ptr(pair_weight), ptr(shared_y), T, d, cap, ptr(out),
                                stream_handle(stream)), "reflex_combine")


WS_FIELDS = {"pair_offsets": 0, "pair_expert": 1, "pair_weight": 2, "expert_offsets": 3,
             "sorted_token": 4, "pair_to_sorted": 5}


def reflex_workspace_offset(T, E, d, f, f_shared, k_max, field: str) -> int:
    off = lib().reflex_workspace_offset(T, E, d, f, f_shared, k_max, WS_FIELDS[field])
    if off == ctypes.c_size_t(-1).value:
        raise ReflexError(-2, "reflex_workspace_offset")
    return off


def reflex_moe_forward(args: MoeArgsC, ws, stream=None):
    _check(lib().reflex_moe_forward(ctypes.byref(args), ptr(ws), ws.numel() * ws.element_size(),
                                    stream_handle(stream)), "reflex_moe_forward")


NOALLOC_SCRATCH_BYTES = 96 << 20     # REFLEX_NOALLOC_SCRATCH_BYTES


def reflex_moe_forward_noalloc(args: MoeArgsC, stream=None):
    _check(lib().reflex_moe_forward_noalloc(ctypes.byref(args), stream_handle(stream)),
           "reflex_moe_forward_noalloc")


def reflex_moe_forward_timed(args: MoeArgsC, ws, events, stream=None):
    """``events``: sequence of N_STAGE_EVENTS hipEvent_t handles (ints)."""
    arr = (c_void_p * N_STAGE_EVENTS)(*events)
    _check(lib().reflex_moe_forward_timed(ctypes.byref(args), ptr(ws), ws.numel() * ws.element_size(),
                                          stream_handle(stream), arr, N_STAGE_EVENTS),
           "reflex_moe_forward_timed")


