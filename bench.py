#!/usr/bin/env python3
"""Throughput of the REFLEX variable-K MoE layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one full pass of the layer (router -> counts -> TopK -> permutation ->
SwiGLU experts -> combine) over the workload's tokens, through
``reflex_moe_forward_timed``; for the 16-layer stack it is all 16 layers, with
counts computed once and shared by every layer.  Inputs and weights are resident
in device memory before timing starts.  HIP events recorded by the library at
every stage boundary give per-stage times; the stage that dominates gets a
roofline figure from its algorithmic bytes (or FLOPs) per launch.  The
fixed-count path (k_i = K_base, default token-choice routing) is timed alongside.
The CPU oracle is timed on a bounded sample of the same workload as a reported
baseline.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import csv
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + TFLOP/s (alloc. expert FLOPs) as % bf16 MFMA peak, var-K"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
DEFAULT_WORKLOAD = "lladamoe_stack16_t8192"   # the largest single-GPU workload
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
COPY_CAL_BYTES = 1 << 28       # the plain device copy that calibrates the byte counters
# rocprofv3 kernel names of the stages with a counter-derived traffic figure
# the grouped GEMM's kernels per stage: 128-row tiles, or 256-row tiles for launches
# whose experts average many rows (the library picks one per launch)
MALL_FLUSH_BYTES = 512 << 20   # read before each cold step: twice the Infinity Cache
STAGE_KERNELS = {"gemm_up": ("swiglu_gemm_kernel<true>", "swiglu_gemm_tall_kernel<true>"),
                 "gemm_down": ("swiglu_gemm_kernel<false>", "swiglu_gemm_tall_kernel<false>")}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded (same soname)."""

    def __init__(self):
        import torch  # noqa: F401  (loads the runtime first)
        h = ctypes.CDLL("libamdhip64.so.7")
        vp = ctypes.c_void_p
        h.hipEventCreate.argtypes = [ctypes.POINTER(vp)]
        h.hipEventDestroy.argtypes = [vp]
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        h.hipEventRecord.argtypes = [vp, vp]
        self.h = h
        self.events = []

    def create(self):
        e = ctypes.c_void_p()
        rc = self.h.hipEventCreate(ctypes.byref(e))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")
        self.events.append(e.value)
        return e.value

    def record(self, e, stream=None):
        rc = self.h.hipEventRecord(e, stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def ms(self, a, b) -> float:
        out = ctypes.c_float()
        rc = self.h.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)

    def close(self):
        for e in self.events:
            self.h.hipEventDestroy(e)
        self.events = []


def expert_counts(lay, h, state, torch):
    """Per-expert pair counts of the counts the layer just used, through the library's
    own TopK and permutation entry points (outside the timed region)."""
    from paper_2608_01784_amd import _lib
    T, E = lay.T, lay.w.E
    cap = T * lay.kcap
    off = torch.empty(T + 1, dtype=torch.int32, device="cuda")
    ex = torch.empty(max(cap, 1), dtype=torch.int32, device="cuda")
    wt = torch.empty(max(cap, 1), dtype=torch.float32, device="cuda")
    _lib.reflex_topk_variable(lay.logits, lay.k, lay.kcap, lay.norm_topk, off, ex, wt)
    eo = torch.empty(E + 1, dtype=torch.int32, device="cuda")
    st = torch.empty(max(cap, 1), dtype=torch.int32, device="cuda")
    p2s = torch.empty(max(cap, 1), dtype=torch.int32, device="cuda")
    ws = torch.empty(max(_lib.reflex_permute_workspace_size(cap, E), 256), dtype=torch.uint8,
                     device="cuda")
    _lib.reflex_permute(off, ex, off[T:T + 1], E, eo, st, p2s, ws)
    torch.cuda.synchronize()
    import numpy as np
    return np.diff(eo.cpu().numpy())


def stage_roofline(stage, ms, d, f, P, touched, T, E):
    """Algorithmic work of one launch of a stage: the bytes the operation itself must
    move once and the FLOPs of its contraction; bound = the larger of the two times at
    peak.  For the expert GEMMs the algorithmic bytes are the touched experts' weights
    plus the layer's input h read once (up) or its output written once (down); the
    pipeline's own traffic between the stages (the P gathered input rows beyond h, the
    P activation rows written and read back, the P expert-output rows) is reported as
    `overhead_bytes` and not credited."""
    overhead = 0
    if stage == "gemm_up":
        flops = 4 * d * f * P
        nbytes = touched * 2 * f * d * 2 + T * d * 2
        overhead = max(P - T, 0) * d * 2 + P * f * 2
    elif stage == "gemm_down":
        flops = 2 * d * f * P
        nbytes = touched * d * f * 2 + T * d * 2
        overhead = P * f * 2 + max(P - T, 0) * d * 2
    elif stage == "router":
        flops = 2 * T * E * d
        nbytes = T * d * 2 + E * d * 4 + T * E * 4
    elif stage == "combine":
        flops = 0
        nbytes = P * d * 2 + P * 8 + (T + 1) * 4 + T * d * 2
    elif stage == "topk":
        flops = 0
        nbytes = T * E * 4 + T * 4 + (T + 1) * 4 + P * 8
    elif stage == "permute":
        flops = 0
        nbytes = P * 4 * 4 + (T + 1) * 4
    else:
        return None
    t_mem = nbytes / (PEAK_HBM_GBS * 1e9)
    t_mfma = flops / (PEAK_BF16_TFLOPS * 1e12)
    if flops and t_mfma > t_mem:
        ach = flops / (ms * 1e-3) / 1e12
        return {"kernel": stage, "bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": None,
                "algorithmic_flops": int(flops), "algorithmic_bytes": int(nbytes),
                "overhead_bytes": int(overhead), "ms": round(ms, 5)}
    ach = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": stage, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None,
            "algorithmic_bytes": int(nbytes), "algorithmic_flops": int(flops),
            "overhead_bytes": int(overhead), "ms": round(ms, 5)}


def kernel_source_digest() -> str:
    """sha256 over the sources of the grouped GEMM (its kernel and shared header): a
    stored counter reading is valid only for the kernel it was taken on."""
    hsh = hashlib.sha256()
    for rel in ("gemm.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2608_01784_amd", "csrc", rel), "rb") as fh:
            hsh.update(fh.read())
    return hsh.hexdigest()


def _counter_rows(path):
    """(kernel name, counter, value) of every dispatch in a rocprofv3 counter CSV, in
    dispatch order."""
    rows = []
    with open(path, newline="") as fh:
        for r in csv.DictReader(fh):
            name = r["Kernel_Name"].replace("void ", "").replace("rfx::(anonymous namespace)::", "")
            name = re.sub(r"\(.*", "", name)
            rows.append((int(r.get("Dispatch_Id") or len(rows)), name, r["Counter_Name"],
                         float(r["Counter_Value"])))
    rows.sort(key=lambda t: t[0])
    return [t[1:] for t in rows]


def _per_dispatch_kib(path, counter, kernel=None, per_forward=1):
    """Mean counter value (KiB) per dispatch of `kernel`; without a kernel name, of the
    dispatches with the largest reading (the calibration copy).  With `per_forward` = 2
    each forward launches the kernel twice (routed experts and the shared expert, on two
    streams, so either may come first): the dispatches are taken in consecutive pairs and
    the larger reading of each pair is the routed launch (it reads and writes P > T rows
    against the shared expert's T, and all the routed weights)."""
    vals = [(n, v) for n, c, v in _counter_rows(path) if c == counter]
    if kernel is None:
        top = max(v for _, v in vals)
        sel = [v for _, v in vals if v >= 0.5 * top]
    else:
        mine = [v for n, v in vals if n == kernel]
        if len(mine) % per_forward:
            raise SystemExit(f"{len(mine)} {counter} dispatches of {kernel} in {path}: "
                             f"not {per_forward} per forward")
        sel = [max(mine[i:i + per_forward]) for i in range(0, len(mine), per_forward)]
    if not sel:
        raise SystemExit(f"no {counter} dispatches of {kernel or 'the copy'} in {path}")
    return sum(sel) / len(sel), len(sel)


def ingest_pmc(workload, layout, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv,
               shared=False):
    """Turn two rocprofv3 --pmc runs of the bench (FETCH_SIZE, WRITE_SIZE) and the same two
    counters on a plain copy of COPY_CAL_BYTES into HBM bytes per GEMM launch, stored in
    the traffic file under the current GEMM source digest.  With a shared expert
    (`shared`), every forward launches each GEMM kernel twice, for the routed experts and
    for the shared expert's dense GEMM; only the routed launches are counted."""
    cf, _ = _per_dispatch_kib(copy_fetch_csv, "FETCH_SIZE")
    cw, _ = _per_dispatch_kib(copy_write_csv, "WRITE_SIZE")
    k_fetch = COPY_CAL_BYTES / (cf * 1024.0)      # true read bytes per counted byte
    k_write = COPY_CAL_BYTES / (cw * 1024.0)
    data = {"calibration": {}, "entries": []}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            data = json.load(fh)
    data["calibration"] = {"copy_bytes": COPY_CAL_BYTES, "fetch_kib": round(cf, 1),
                           "write_kib": round(cw, 1), "fetch_factor": round(k_fetch, 4),
                           "write_factor": round(k_write, 4)}
    digest = kernel_source_digest()
    for stage, knames in STAGE_KERNELS.items():
        present = {n for n, c, _ in _counter_rows(fetch_csv) if c == "FETCH_SIZE"}
        kname = next((k for k in knames if k in present), knames[0])
        per_fwd = 2 if shared and kname in STAGE_KERNELS[stage][:1] else 1
        fk, nf = _per_dispatch_kib(fetch_csv, "FETCH_SIZE", kname, per_fwd)
        wk, nw = _per_dispatch_kib(write_csv, "WRITE_SIZE", kname, per_fwd)
        ent = {"workload": workload, "expert_weights": layout, "kernel": stage,
               "kernel_name": kname, "source_sha256": digest,
               "fetch_kib_per_dispatch": round(fk, 1), "write_kib_per_dispatch": round(wk, 1),
               "dispatches": [nf, nw],
               "read_bytes": int(fk * 1024 * k_fetch), "write_bytes": int(wk * 1024 * k_write)}
        ent["traffic_bytes"] = ent["read_bytes"] + ent["write_bytes"]
        data["entries"] = [e for e in data["entries"]
                           if (e["workload"], e["expert_weights"], e["kernel"]) != (workload, layout, stage)]
        data["entries"].append(ent)
        print(json.dumps(ent))
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(data, fh, indent=1)
        fh.write("\n")


def measured_traffic(workload, layout, stage):
    """HBM bytes per launch from stored counter readings, or None when there are none for
    this workload and kernel or the kernel source has changed since they were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as fh:
        data = json.load(fh)
    digest = kernel_source_digest()
    for e in data.get("entries", []):
        if (e["workload"], e["expert_weights"], e["kernel"]) == (workload, layout, stage):
            return e["traffic_bytes"] if e["source_sha256"] == digest else None
    return None


def copy_calibration():
    """The plain device copy of COPY_CAL_BYTES whose counter readings scale FETCH_SIZE and
    WRITE_SIZE to bytes (run under rocprofv3 --pmc)."""
    import torch
    src = torch.ones(COPY_CAL_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_CAL_BYTES, "copies": 3}))


def _dist(xs):
    """Median and 10th / 90th percentiles of per-step times (ms)."""
    import numpy as np
    v = np.asarray(xs, dtype=np.float64)
    return {"median": round(float(np.median(v)), 4), "p10": round(float(np.percentile(v, 10)), 4),
            "p90": round(float(np.percentile(v, 90)), 4)}


def run_path(torch, w, dws, residuals, h0, state, uniform_k, steps, warmup, ev: HipEvents,
             cold=False):
    """Time `steps` steps of the layer (or layer stack) through the plain fused entry
    point (wall clock and one event pair around all of them), then `steps` more with an
    event pair around each (the per-step distribution), then `steps` more through the
    timed entry point for the per-stage split (its events add a little time of their
    own, so those passes are kept out of the step time).  With `cold`, a last pass of
    `steps` timed-entry steps reads a MALL_FLUSH_BYTES buffer before each step, so the
    256 MB Infinity Cache holds none of the weights when a step starts.  Returns timings
    and the layer objects used."""
    from paper_2608_01784_amd import _lib
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer
    L = w.n_layers
    lays = [MoELayer(w.T, w.d, dws[l], w.params, uniform_k=uniform_k) for l in range(L)]
    res = residuals
    hbuf = [h0, torch.empty_like(h0), torch.empty_like(h0)]
    evs = [[[ev.create() for _ in range(_lib.N_STAGE_EVENTS)] for _ in range(L)]
           for _ in range(steps)]

    def step(events=None):
        h = hbuf[0]
        k_in = None
        for l in range(L):
            lay = lays[l]
            out = hbuf[1 + (l & 1)] if L > 1 else None
            args = lay.args(h, state if k_in is None else None, k_in=k_in,
                            residual_a=h if L > 1 else None,
                            residual_b=res[l] if (L > 1 and res is not None) else None, out=out)
            if events is None:
                _lib.reflex_moe_forward(args, lay.ws)
            else:
                _lib.reflex_moe_forward_timed(args, lay.ws, events[l])
            if L > 1:
                k_in = lays[0].k
                h = out

    for _ in range(warmup):
        step()
    e_begin, e_end = ev.create(), ev.create()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev.record(e_begin)
    for s in range(steps):
        step()
    ev.record(e_end)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    gpu_step_ms = ev.ms(e_begin, e_end) / steps
    marks = [ev.create() for _ in range(steps + 1)]
    ev.record(marks[0])
    for s in range(steps):
        step()
        ev.record(marks[s + 1])
    torch.cuda.synchronize()
    per_step = [ev.ms(marks[s], marks[s + 1]) for s in range(steps)]

    def stage_pass(flush):
        for s in range(steps):
            if flush is not None:
                # read (not write) the buffer: the cache ends up holding only clean lines
                # of it, so no write-back of dirty lines competes with the step
                flush.max()
            step(evs[s])
        torch.cuda.synchronize()
        n_ev = _lib.N_STAGE_EVENTS
        stage = {}
        for i, name in enumerate(_lib.STAGES):
            stage[name] = sum(ev.ms(evs[s][l][i], evs[s][l][i + 1]) for s in range(steps)
                              for l in range(L)) / (steps * L)
        totals = [sum(ev.ms(evs[s][l][0], evs[s][l][n_ev - 1]) for l in range(L))
                  for s in range(steps)]
        return stage, totals

    stage_ms, _ = stage_pass(None)
    out = {"wall_ms": (t1 - t0) * 1e3 / steps, "gpu_ms": gpu_step_ms, "stage_ms": stage_ms,
           "step_dist": _dist(per_step), "layers": lays}
    if cold:
        flush = torch.ones(MALL_FLUSH_BYTES // 4, dtype=torch.int32, device=h0.device)
        c_stage, c_tot = stage_pass(flush)
        del flush
        out["cold"] = {"stage_ms": c_stage, "step_dist": _dist(c_tot),
                       "flush_bytes": MALL_FLUSH_BYTES}
    return out


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, host, seconds):
    """Time the oracle (as it is) on a bounded sample of the workload: the whole layer
    (router, budget, TopK, permutation, experts, combine) and, separately, its routing
    half (budget, router, TopK, permutation)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):  # pragma: no cover
        affinity = os.cpu_count() or 1
    wg, wu, wd = host["w_gate"], host["w_up"], host["w_down"]
    wof = lambda e: (wg[e], wu[e], wd[e])  # noqa: E731
    n_sample = w.T if w.T <= 4096 else 1024
    toks = None if n_sample == w.T else np.sort(np.random.default_rng(0).choice(w.T, n_sample, replace=False))
    t_route = t_exp = 0.0
    reps = 0
    t_start = time.perf_counter()
    while True:
        a = time.perf_counter()
        bud = oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1, w.conf_prev2,
                                   w.seq_offsets, w.active_block, w.params)
        r = oracle.router_scores(w.h, host["w_router"], w.router_bias)
        route = oracle.topk_route(r, bud.k, w.norm_topk)
        oracle.pair_permutation(route.token, route.expert, w.E)
        b = time.perf_counter()
        oracle.moe_layer(w.h, route, wof, w.E, shared=host["shared"], tokens=toks)
        c = time.perf_counter()
        t_route += b - a
        t_exp += c - b
        reps += 1
        if c - t_start >= seconds:
            break
    route_s = t_route / reps
    per_layer = route_s + (t_exp / reps) * (w.T / n_sample)
    sample = (f"{reps} full oracle layer(s) of {w.name}" if toks is None else
              f"{reps} rep(s) of layer 0 of {w.name}: routing on all {w.T} tokens, experts+combine "
              f"on {n_sample} sampled tokens, scaled to {w.T}")
    return {"value": round(w.T / per_layer, 2), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle", "sample": sample + f"; {w.n_layers} layer(s) per step counted",
            "seconds": round(t_route + t_exp, 2), "affinity_cores": int(affinity),
            "blas_threads": int(threads), "cpu_model": _cpu_model(),
            "layer_ms": round(per_layer * 1e3, 2), "routing_ms": round(route_s * 1e3, 2),
            "routing_tokens_per_s": round(w.T / route_s, 1)}


def trajectory_stats(a, torch):
    """Decode a whole synthetic generation (every block, from all-masked) with the fused
    layer and the state kernel; report forwards (NFE), pairs and AvgK next to fixed
    top-K_base routing over the same forwards."""
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    from paper_2608_01784_amd.trajectory import run_trajectory
    from synth import forward_confidence, generation_start, make_workload
    from synth.device import to_device
    w = make_workload(a.workload, seed=a.seed)
    if w.n_layers != 1:
        raise SystemExit("--trajectory runs single-layer workloads")
    dv = {k: to_device(getattr(w, k)(0)) for k in ("w_gate", "w_up", "w_down", "w_router")}
    dv["router_bias"] = None if w.router_bias is None else to_device(w.router_bias)
    sh = w.shared_weights(0)
    if sh is not None:
        dv["ws_gate"], dv["ws_up"], dv["ws_down"] = (to_device(x) for x in sh)
    lay = MoELayer(w.T, w.d, ExpertWeights(**dv), w.params)
    st = TokenState(**{k: to_device(v) for k, v in generation_start(w).items()})
    h = to_device(w.h)
    confs = [to_device(forward_confidence(a.seed, t, w.T)) for t in range(64)]
    t0 = time.perf_counter()
    stats = run_trajectory(lay, h, st, lambda t: confs[t] if t < len(confs) else
                           to_device(forward_confidence(a.seed, t, w.T)), theta=w.params.theta)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    P = stats.total_pairs
    print(json.dumps({"trajectory": {
        "workload": w.name, "data": "synthetic confidences (seeded, rising per forward)",
        "forwards": stats.forwards, "total_pairs": P,
        "avg_k": round(P / (stats.forwards * w.T), 4),
        "uniform_pairs": stats.forwards * w.T * w.params.k_base,
        "pair_ratio_vs_uniform": round(P / (stats.forwards * w.T * w.params.k_base), 4),
        "alloc_tflop": round(6 * w.d * w.f * P / 1e12, 3),
        "wall_s": round(wall, 3), "pairs_per_forward": stats.pairs}}), flush=True)


def dense_reference(a, torch):
    """The vendor library's dense bf16 GEMM (hipBLASLt through torch.bmm) on batched shapes
    with the FLOPs of the workload's routed up and down GEMMs: E experts of P/E rows each (P
    from one variable-K forward), [E, P/E, d] x [E, d, 2f] and [E, P/E, f] x [E, f, d], and
    one large [P, d] x [d, 2f] product.  A reference point for what a tuned dense GEMM reaches
    on this chip at these sizes, not a drop-in: no row gather, no SwiGLU, equal rows per
    expert.  Operands are contiguous (no transposed views)."""
    from paper_2608_01784_amd.layer import ExpertWeights, MoELayer, TokenState
    from synth import make_workload
    from synth.device import state_tensors, to_device
    w = make_workload(a.workload, seed=a.seed)
    E, d, f, T = w.E, w.d, w.f, w.T
    lay = MoELayer(T, d, ExpertWeights(w_gate=to_device(w.w_gate(0)), w_up=to_device(w.w_up(0)),
                                       w_down=to_device(w.w_down(0)),
                                       w_router=to_device(w.w_router(0))), w.params)
    lay.forward(to_device(w.h), TokenState(**state_tensors(w)))
    torch.cuda.synchronize()
    P = int(lay.pairs.item())
    w.release(0)
    del lay
    m = max(1, round(P / E))
    g = torch.Generator(device="cuda")
    g.manual_seed(a.seed)

    def rnd(*shape):
        return (torch.randn(*shape, device="cuda", generator=g) * 0.02).bfloat16()

    def timed(fn, flops, iters=20):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(iters):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / iters
        tf = flops / (ms * 1e-3) / 1e12
        return {"ms": round(ms, 5), "tflops": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4)}

    out = {"mode": "dense_reference", "workload": w.name, "library": "hipBLASLt (torch.bmm / mm)",
           "pairs": P, "experts": E, "rows_per_expert": m}
    xa, wa = rnd(E, m, d), rnd(E, d, 2 * f)
    out["up_batched"] = timed(lambda: torch.bmm(xa, wa), 2.0 * E * m * d * 2 * f)
    del xa, wa
    xb, wb = rnd(E, m, f), rnd(E, f, d)
    out["down_batched"] = timed(lambda: torch.bmm(xb, wb), 2.0 * E * m * f * d)
    del xb, wb
    xc, wc = rnd(P, d), rnd(d, 2 * f)
    out["up_one_gemm"] = timed(lambda: torch.mm(xc, wc), 2.0 * P * d * 2 * f)
    print(json.dumps(out), flush=True)


def device_figures(torch):
    """The chip as the runtime reports it, the dense bf16 peak re-derived from that (4096
    FLOP per clock per CU from the 32x32x16 bf16 MFMA rate of 4 SIMDs), and two measured
    device-memory rates (plain torch copy and fill of 1 GiB, outside any timed region).
    The roofline keeps the published peaks; these figures are reported beside them."""
    p = torch.cuda.get_device_properties(0)
    cus = int(p.multi_processor_count)

    def attr(code):
        # hipDeviceGetAttribute of the HIP runtime torch has loaded (ROCm 7 attribute codes:
        # 5 peak clock kHz, 59 memory bus bits, 60 peak memory clock kHz); 0 if unavailable
        import ctypes
        try:
            hip = ctypes.CDLL("libamdhip64.so")
            v = ctypes.c_int(0)
            return v.value if hip.hipDeviceGetAttribute(ctypes.byref(v), code, 0) == 0 else 0
        except OSError:
            return 0

    clk_mhz = attr(5) / 1e3
    out = {"name": p.name, "arch": p.gcnArchName, "cus": cus, "clock_mhz": round(clk_mhz, 1),
           "l2_bytes": int(p.L2_cache_size), "hbm_bytes": int(p.total_memory),
           "memory_clock_mhz": round(attr(60) / 1e3, 1), "memory_bus_bits": attr(59),
           "derived_bf16_tflops": round(4096 * cus * clk_mhz * 1e6 / 1e12, 1)}
    n = 1 << 29                                      # bf16 elements: 1 GiB
    x = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    x.fill_(1.0)
    y = torch.empty_like(x)

    def rate(fn, nbytes, reps=10):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return round(nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)

    out["measured_copy_gbs"] = rate(lambda: y.copy_(x), 2 * 2 * n)     # 1 GiB read + 1 GiB written
    out["measured_fill_gbs"] = rate(lambda: y.fill_(0.5), 2 * n)
    del x, y
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-uniform", action="store_true")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the pass that evicts the Infinity Cache (a 512 MiB read) before "
                         "each step")
    ap.add_argument("--trajectory", action="store_true",
                    help="run a synthetic multi-forward decoding trajectory (all blocks, from an "
                         "all-masked start) and print its forward and pair statistics instead")
    ap.add_argument("--dense-reference", action="store_true",
                    help="time the vendor library's dense bf16 GEMM at the workload's routed GEMM "
                         "sizes (FLOPs) and print that instead")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only the plain 256 MiB device copy that calibrates the byte counters")
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                      "COPY_WRITE_CSV"),
                    help="store HBM traffic per GEMM launch from rocprofv3 counter CSVs (no GPU)")
    a = ap.parse_args()
    layout = "row-major"
    if a.ingest_pmc:
        from synth import make_workload
        ingest_pmc(a.workload, layout, *a.ingest_pmc,
                   shared=make_workload(a.workload, seed=a.seed).f_shared > 0)
        return
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(no collectives, no sharding); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_01784_amd import _lib
    from paper_2608_01784_amd.layer import ExpertWeights, TokenState
    from synth import make_workload
    from synth.device import state_tensors, to_device

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if a.copy_calibration:
        copy_calibration()
        return
    _lib.lib()
    if a.dense_reference:
        dense_reference(a, torch)
        return
    if a.trajectory:
        trajectory_stats(a, torch)
        return
    log(f"generating {a.workload} (seed {a.seed})")
    w = make_workload(a.workload, seed=a.seed)
    hosts, dws = [], []
    for l in range(w.n_layers):
        host = {"w_gate": w.w_gate(l), "w_up": w.w_up(l), "w_down": w.w_down(l),
                "w_router": w.w_router(l), "shared": w.shared_weights(l)}
        dv = {k: to_device(host[k]) for k in ("w_gate", "w_up", "w_down", "w_router")}
        dv["router_bias"] = None if w.router_bias is None else to_device(w.router_bias)
        if host["shared"] is not None:
            dv["ws_gate"], dv["ws_up"], dv["ws_down"] = (to_device(x) for x in host["shared"])
        dws.append(ExpertWeights(**dv))
        hosts.append(host if l == 0 else None)
        if l > 0:
            w.release(l)
        if w.n_layers > 1:
            log(f"layer {l} weights resident")
    residuals = [to_device(w.residual(l)) for l in range(w.n_layers)] if w.n_layers > 1 else None
    h0 = to_device(w.h)
    state = TokenState(**state_tensors(w))
    torch.cuda.synchronize()

    ev = HipEvents()
    log(f"timing variable-K path: {a.warmup} warmup + {a.steps} steps")
    var = run_path(torch, w, dws, residuals, h0, state, 0, a.steps, a.warmup, ev,
                   cold=not a.no_cold)
    lay0 = var["layers"][0]
    P = int(lay0.pairs.item())
    counts = expert_counts(lay0, h0, state, torch)
    touched = int((counts > 0).sum())
    uni = None
    if not a.no_uniform:
        log("timing fixed-count path (k = K_base)")
        uni = run_path(torch, w, dws, residuals, h0, state, w.params.k_base, a.steps, a.warmup, ev)
    ev.close()
    log("device figures (runtime properties, 1 GiB copy and fill)")
    dev = device_figures(torch)

    T, d, f, E, L = w.T, w.d, w.f, w.E, w.n_layers
    step_ms = var["wall_ms"]
    tokens_per_s = T / (step_ms * 1e-3)
    alloc_flops = 6 * d * f * P * L                # Eq. (10) per step
    alloc_tflops = alloc_flops / (step_ms * 1e-3) / 1e12
    stages = var["stage_ms"]
    dom = max(("gemm_up", "gemm_down", "router", "combine", "topk", "permute"), key=lambda s: stages[s])
    roof = stage_roofline(dom, stages[dom], d, f, P, touched, T, E)
    roof_all = {s: stage_roofline(s, stages[s], d, f, P, touched, T, E)
                for s in ("gemm_up", "gemm_down", "router", "topk", "permute", "combine")}
    for s in STAGE_KERNELS:
        roof_all[s]["traffic"] = measured_traffic(w.name, layout, s)
    roof["traffic"] = roof_all[dom]["traffic"]
    out = {
        "metric": METRIC, "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "tokens": T, "hidden": d, "experts": E, "expert_ffn": f,
                   "shared_ffn": w.f_shared, "layers": L, "k_base": w.params.k_base,
                   "k_range": [w.params.k_min, w.params.k_max], "path": "variable-K (REFLEX)",
                   "expert_weights": layout},
        "alloc_tflops": round(alloc_tflops, 2),
        "pct_bf16_peak": round(100 * alloc_tflops / PEAK_BF16_TFLOPS, 2),
        "pairs_per_layer": P, "avg_k": round(P / T, 4), "experts_touched": touched,
        "max_expert_rows": int(counts.max()), "gpu_ms_per_step": round(var["gpu_ms"], 4),
        "stage_ms": {k: round(v, 5) for k, v in stages.items()},
        "step_ms_dist": var["step_dist"],
        "roofline": roof,
        "roofline_all": roof_all,
        "device": dev,
    }
    if "cold" in var:
        cs = var["cold"]["stage_ms"]
        out["cold"] = {"flush_bytes": var["cold"]["flush_bytes"],
                       "step_ms_dist": var["cold"]["step_dist"],
                       "stage_ms": {k: round(v, 5) for k, v in cs.items()},
                       "roofline": {s: stage_roofline(s, cs[s], d, f, P, touched, T, E)
                                    for s in ("gemm_up", "gemm_down")}}
    if uni is not None:
        lu = uni["layers"][0]
        Pu = int(lu.pairs.item())
        u_ms = uni["wall_ms"]
        out["uniform"] = {"k": w.params.k_base, "ms_per_step": round(u_ms, 4),
                          "tokens_per_s": round(T / (u_ms * 1e-3), 1), "pairs_per_layer": Pu,
                          "alloc_tflops": round(6 * d * f * Pu * L / (u_ms * 1e-3) / 1e12, 2),
                          "stage_ms": {k: round(v, 5) for k, v in uni["stage_ms"].items()}}
        out["var_over_uniform"] = {"pairs": round(P / Pu, 4), "time": round(step_ms / u_ms, 4)}
    if not a.no_cpu_baseline:
        log(f"timing the CPU oracle (~{a.cpu_seconds:.0f} s)")
        out["cpu_baseline"] = cpu_baseline(w, hosts[0], a.cpu_seconds)
        if L > 1:
            out["cpu_baseline"]["value"] = round(out["cpu_baseline"]["value"] / L, 2)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
