"""Seeded synthetic workloads shaped like LLaDA-MoE and LLaDA2.0-mini MoE layers.

Every array is drawn from ``numpy.random.default_rng`` with a seed key made of
(workload seed, tensor tag, layer, expert), so any single expert's weights can
be regenerated alone (the CPU oracle uses that to check sampled tokens at full
size without materialising every weight in fp64).

Layout of the decoding state follows block-wise DLM inference (Section 3.1):
prompt positions carry block index 0, target positions are split into blocks
1..Q of ``n_blk`` tokens, one block per sequence is active, blocks before it
are fully committed, blocks after it are fully masked.  The hyper-parameter
defaults are the ones the paper states in its experimental setting
(Section 5.1): n_blk = 32, theta = 0.9, K_base = 8, delta_role = 4,
delta_cur = 2, q = 0.25, v_ref = 0.01, tau = 0.05, w_cf = 0.30 (LLaDA-MoE) or
0.25 (LLaDA2.0-mini).

bf16 tensors are carried as ``uint16`` bit patterns, rounded to nearest-even
from float32 draws.  Nothing here computes any step of the method.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import numpy as np

# Tags that separate the random streams of the different tensors.
_TAG_H, _TAG_WG, _TAG_WU, _TAG_WD, _TAG_WR = 1, 2, 3, 4, 5
_TAG_SG, _TAG_SU, _TAG_SD, _TAG_LAYOUT, _TAG_CONF, _TAG_RES, _TAG_BIAS = 6, 7, 8, 9, 10, 11, 12

_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the bits.

    Input generation only: the drawn values are stored in the precision the
    kernels consume.  (Inputs are finite normals, so NaN handling is not needed.)
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = u + np.uint32(0x7FFF)
    r += (u >> np.uint32(16)) & np.uint32(1)
    return (r >> np.uint32(16)).astype(np.uint16)


def _f32(x: float) -> float:
    """The float32 value nearest to x, as a Python float (exact)."""
    return float(np.float32(x))


@dataclass(frozen=True)
class AllocParams:
    """REFLEX allocation hyper-parameters (Eqs. (3), (5)-(9)).

    Real-valued ones are float32 values (the library takes them as float), so
    both the oracle and the kernels start from the same binary numbers.
    ``signal`` selects the active-block ranking key: 0 = Frontier-Progress
    Score (Eq. (8)); 1..4 are the single-signal variants of Appendix C
    (frontier only, progress only, confidence only, uncertainty only).
    """
    k_base: int
    delta_role: int
    delta_cur: int
    k_min: int
    k_max: int
    q: float
    theta: float
    w_cf: float
    v_ref: float
    tau: float
    signal: int = 0

    @staticmethod
    def make(k_base, delta_role, delta_cur, k_min, k_max, q=0.25, theta=0.9,
             w_cf=0.30, v_ref=0.01, tau=0.05, signal=0) -> "AllocParams":
        return AllocParams(int(k_base), int(delta_role), int(delta_cur), int(k_min),
                           int(k_max), _f32(q), _f32(theta), _f32(w_cf), _f32(v_ref),
                           _f32(tau), int(signal))

    def replace(self, **kw) -> "AllocParams":
        d = dict(self.__dict__)
        d.update(kw)
        return AllocParams.make(**d)


@dataclass
class Workload:
    """One synthetic MoE-layer (or layer-stack) workload.

    Token state arrays (length T): ``block_idx`` (b(i), prompt = 0),
    ``masked`` (1 if the position is still [MASK]), ``hist_len`` (how many of
    the two latest confidence observations exist: 0, 1 or 2), ``conf_prev1``
    and ``conf_prev2`` (c^{t-1}, c^{t-2}).  Sequences are contiguous token
    ranges ``seq_offsets[s]:seq_offsets[s+1]`` with active block
    ``active_block[s]``.
    """
    name: str
    seed: int
    T: int
    d: int
    E: int
    f: int
    f_shared: int
    n_layers: int
    params: AllocParams
    h: np.ndarray
    block_idx: np.ndarray
    seq_offsets: np.ndarray
    active_block: np.ndarray
    masked: np.ndarray
    hist_len: np.ndarray
    conf_prev1: np.ndarray
    conf_prev2: np.ndarray
    router_bias: Optional[np.ndarray] = None
    w_scale: float = 0.02
    wr_scale: float = 0.02
    residual_scale: float = 0.1
    norm_topk: int = 1
    _cache: Dict = field(default_factory=dict, repr=False)

    @property
    def B(self) -> int:
        return int(self.active_block.shape[0])

    @property
    def uniform_k(self) -> int:
        return self.params.k_base

    # ---- weights, drawn per (layer, tensor, expert) --------------------------------
    def _normal_bf16(self, key, shape, scale) -> np.ndarray:
        rng = np.random.default_rng([self.seed] + list(key))
        a = np.empty(int(np.prod(shape)), dtype=np.float32)
        rng.standard_normal(out=a, dtype=np.float32)
        a *= np.float32(scale)
        return bf16_bits_from_f32(a).reshape(shape)

    def expert_weights(self, layer: int, e: int):
        """(W_gate [f,d], W_up [f,d], W_down [d,f]) of one routed expert, bf16 bits."""
        f, d, s = self.f, self.d, self.w_scale
        return (self._normal_bf16((_TAG_WG, layer, e), (f, d), s),
                self._normal_bf16((_TAG_WU, layer, e), (f, d), s),
                self._normal_bf16((_TAG_WD, layer, e), (d, f), s))

    def _stacked(self, layer: int, which: int) -> np.ndarray:
        key = ("stack", layer, which)
        if key in self._cache:
            return self._cache[key]
        f, d, E, s = self.f, self.d, self.E, self.w_scale
        shape = (f, d) if which != _TAG_WD else (d, f)
        out = np.empty((E,) + shape, dtype=np.uint16)

        def job(e):
            out[e] = self._normal_bf16((which, layer, e), shape, s)
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(job, range(E)))
        return out

    def release(self, layer: int) -> None:
        """Drop the cached stacked weights of one layer (after they were uploaded)."""
        for which in (_TAG_WG, _TAG_WU, _TAG_WD):
            self._cache.pop(("stack", layer, which), None)

    def w_gate(self, layer: int = 0) -> np.ndarray:
        """[E, f, d] bf16 bits (nn.Linear layout, d contiguous)."""
        return self._stacked(layer, _TAG_WG)

    def w_up(self, layer: int = 0) -> np.ndarray:
        return self._stacked(layer, _TAG_WU)

    def w_down(self, layer: int = 0) -> np.ndarray:
        """[E, d, f] bf16 bits (f contiguous)."""
        return self._stacked(layer, _TAG_WD)

    def shared_weights(self, layer: int = 0):
        """Always-on shared expert (W_gate [fs,d], W_up [fs,d], W_down [d,fs]) or None."""
        if self.f_shared <= 0:
            return None
        fs, d, s = self.f_shared, self.d, self.w_scale
        return (self._normal_bf16((_TAG_SG, layer, 0), (fs, d), s),
                self._normal_bf16((_TAG_SU, layer, 0), (fs, d), s),
                self._normal_bf16((_TAG_SD, layer, 0), (d, fs), s))

    def w_router(self, layer: int = 0) -> np.ndarray:
        """[E, d] float32 router weight."""
        rng = np.random.default_rng([self.seed, _TAG_WR, layer])
        a = rng.standard_normal((self.E, self.d), dtype=np.float32)
        a *= np.float32(self.wr_scale)
        return a

    def residual(self, layer: int) -> np.ndarray:
        """Fixed bf16 [T,d] perturbation added after layer ``layer`` of a stack
        (stands in for the attention block between MoE layers)."""
        return self._normal_bf16((_TAG_RES, layer, 0), (self.T, self.d), self.residual_scale)


# ---------------------------------------------------------------------------------------
# layouts
# ---------------------------------------------------------------------------------------
def _dlm_sequence(rng, n_prompt, n_blocks, n_blk, active, masked_frac):
    """One sequence: prompt (b = 0) then blocks 1..n_blocks of n_blk tokens."""
    b = np.concatenate([np.zeros(n_prompt, np.int32),
                        np.repeat(np.arange(1, n_blocks + 1, dtype=np.int32), n_blk)])
    m = (b > active).astype(np.uint8)
    start = n_prompt + (active - 1) * n_blk
    n_m = int(round(masked_frac * n_blk))
    n_m = min(max(n_m, 1), n_blk)
    pos = rng.choice(n_blk, size=n_m, replace=False)
    m[start + pos] = 1
    return b, m


def _confidence(rng, T, beta: bool):
    c1 = (rng.beta(2.0, 2.0, T) if beta else rng.random(T)).astype(np.float32)
    delta = rng.uniform(-0.2, 0.3, T).astype(np.float32)
    c2 = np.clip(c1 - delta, np.float32(0), np.float32(1)).astype(np.float32)
    return c1, c2


def _hidden(seed, T, d):
    rng = np.random.default_rng([seed, _TAG_H])
    a = np.empty(T * d, dtype=np.float32)
    rng.standard_normal(out=a, dtype=np.float32)
    return bf16_bits_from_f32(a).reshape(T, d)


def _tiny(seed, roles: bool) -> Workload:
    rng = np.random.default_rng([seed, _TAG_LAYOUT])
    T, d, E, f = 128, 256, 8, 512
    if roles:
        act, fut = 3, 5
    else:
        act, fut = 1, 2
    b = np.concatenate([np.zeros(64, np.int32), np.full(32, act, np.int32),
                        np.full(32, fut, np.int32)])
    m = np.zeros(T, np.uint8)
    m[64 + rng.choice(32, 16, replace=False)] = 1
    m[96:] = 1
    c1, c2 = _confidence(np.random.default_rng([seed, _TAG_CONF]), T, beta=False)
    hist = np.where(m == 1, 2, 0).astype(np.int8)
    p = AllocParams.make(2, 1, 1, 1, 4, q=0.25, theta=0.9, w_cf=0.30, v_ref=0.01, tau=0.05)
    return Workload("tiny_roles_t128_e8" if roles else "tiny_t128_e8", seed, T, d, E, f, 0, 1, p,
                    _hidden(seed, T, d), b, np.array([0, T], np.int32),
                    np.array([act], np.int32), m, hist, c1, c2)


def _dlm_batch(seed, B, n_prompt, n_blocks, n_blk, active: Optional[List[int]] = None):
    rng = np.random.default_rng([seed, _TAG_LAYOUT])
    bs, ms, acts = [], [], []
    for s in range(B):
        a = int(rng.integers(1, n_blocks + 1)) if active is None else int(active[s])
        frac = float(rng.uniform(0.2, 0.9))
        b, m = _dlm_sequence(rng, n_prompt, n_blocks, n_blk, a, frac)
        bs.append(b)
        ms.append(m)
        acts.append(a)
    L = n_prompt + n_blocks * n_blk
    return (np.concatenate(bs), np.concatenate(ms), np.arange(0, (B + 1) * L, L, dtype=np.int32),
            np.array(acts, np.int32))


def _llada(seed, name, B, E, f, f_shared, n_layers, w_cf, active=None) -> Workload:
    d = 2048
    b, m, so, act = _dlm_batch(seed, B, 512, 16, 32, active)
    T = int(so[-1])
    c1, c2 = _confidence(np.random.default_rng([seed, _TAG_CONF]), T, beta=True)
    hist = np.where(m == 1, 2, 0).astype(np.int8)
    p = AllocParams.make(8, 4, 2, 2, 12, q=0.25, theta=0.9, w_cf=w_cf, v_ref=0.01, tau=0.05)
    return Workload(name, seed, T, d, E, f, f_shared, n_layers, p, _hidden(seed, T, d),
                    b, so, act, m, hist, c1, c2)


def _skewed(seed) -> Workload:
    rng = np.random.default_rng([seed, _TAG_LAYOUT])
    S, E, f, d = 256, 256, 512, 2048
    bs = []
    acts = rng.integers(1, 9, S).astype(np.int32)
    for s in range(S):
        bs.append(np.concatenate([np.zeros(32, np.int32), np.full(32, acts[s], np.int32)]))
    b = np.concatenate(bs)
    m = np.tile(np.concatenate([np.zeros(32, np.uint8), np.ones(32, np.uint8)]), S)
    T = S * 64
    c1, c2 = _confidence(np.random.default_rng([seed, _TAG_CONF]), T, beta=True)
    hist = np.where(m == 1, 2, 0).astype(np.int8)
    # Zipf(1.2) skew of the routing mass: expert e gets logit offset -1.2 ln(pi_e),
    # pi a seeded permutation of the ranks 1..E.
    perm = np.random.default_rng([seed, _TAG_BIAS]).permutation(E) + 1
    bias = (-1.2 * np.log(perm.astype(np.float64))).astype(np.float32)
    p = AllocParams.make(8, 4, 2, 1, 16, q=0.25, theta=0.9, w_cf=0.30, v_ref=0.01, tau=0.05)
    return Workload("skewed_t16384_e256", seed, T, d, E, f, 0, 1, p, _hidden(seed, T, d), b,
                    np.arange(0, T + 1, 64, dtype=np.int32), acts, m, hist, c1, c2,
                    router_bias=bias)


_MAKERS: Dict[str, Callable[..., Workload]] = {
    # 128 tokens, d=256, E=8, f=512; prompt + active block 1 (half masked) + future block 2
    "tiny_t128_e8": lambda seed, active=None: _tiny(seed, roles=False),
    # same, blocks relabelled 3 (active) and 5 (future) so all three role levels occur
    "tiny_roles_t128_e8": lambda seed, active=None: _tiny(seed, roles=True),
    # LLaDA-MoE-shaped layer: 1 x 1024 tokens, d=2048, E=64, f=1024
    "lladamoe_t1024_e64": lambda seed, active=None: _llada(
        seed, "lladamoe_t1024_e64", 1, 64, 1024, 0, 1, 0.30,
        None if active is None else [active]),
    # LLaDA2.0-mini-shaped layer: 4 x 1024 tokens, E=256, f=512, one shared expert f=512
    "llada2mini_t4096_e256": lambda seed, active=None: _llada(
        seed, "llada2mini_t4096_e256", 4, 256, 512, 512, 1, 0.25,
        None if active is None else [active] * 4),
    # 16 stacked LLaDA-MoE-shaped layers over 8 x 1024 tokens
    "lladamoe_stack16_t8192": lambda seed, active=None: _llada(
        seed, "lladamoe_stack16_t8192", 8, 64, 1024, 0, 16, 0.30,
        None if active is None else [active] * 8),
    # skewed load: 256 sequences x (32 prompt + 32 masked active), E=256, Zipf router bias
    "skewed_t16384_e256": lambda seed, active=None: _skewed(seed),
}
WORKLOAD_NAMES = tuple(_MAKERS)


def make_workload(name: str, seed: int = 0, active: Optional[int] = None) -> Workload:
    return _MAKERS[name](seed, active=active)


def make_fuzz_workload(seed: int, T: Optional[int] = None, d: Optional[int] = None,
                       E: Optional[int] = None, f: Optional[int] = None,
                       f_shared: int = 0, k_max: Optional[int] = None,
                       hist_mix: bool = True) -> Workload:
    """Random small workload: several sequences of random length, random block
    sizes and active blocks, mixed history lengths, random count bounds."""
    rng = np.random.default_rng([seed, 777])
    d = d if d is not None else int(rng.choice([128, 256]))
    f = f if f is not None else int(rng.choice([128, 256]))
    E = E if E is not None else int(rng.choice([1, 2, 5, 8, 16, 60, 64, 128, 255, 256]))
    T_target = T if T is not None else int(rng.integers(1, 700))
    bs, ms, acts, offs = [], [], [], [0]
    while offs[-1] < T_target:
        n_blk = int(rng.choice([4, 8, 16, 32, 64]))
        n_prompt = int(rng.integers(0, 80))
        n_blocks = int(rng.integers(1, 8))
        a = int(rng.integers(1, n_blocks + 1))
        b, m = _dlm_sequence(rng, n_prompt, n_blocks, n_blk, a, float(rng.uniform(0.05, 1.0)))
        room = T_target - offs[-1]
        b, m = b[:room], m[:room]
        bs.append(b)
        ms.append(m)
        acts.append(a)
        offs.append(offs[-1] + len(b))
    b = np.concatenate(bs).astype(np.int32)
    m = np.concatenate(ms).astype(np.uint8)
    T = int(offs[-1])
    c1, c2 = _confidence(rng, T, beta=bool(rng.integers(0, 2)))
    if hist_mix:
        hist = rng.choice(np.array([0, 1, 2, 2, 2], np.int8), T).astype(np.int8)
    else:
        hist = np.full(T, 2, np.int8)
    km = k_max if k_max is not None else int(rng.integers(1, min(E, 32) + 1))
    kmin = int(rng.integers(1, km + 1))
    kb = int(rng.integers(kmin, km + 1))
    p = AllocParams.make(kb, int(rng.integers(0, 4)), int(rng.integers(0, 3)), kmin, km,
                         q=float(rng.choice([0.125, 0.25, 0.3, 0.5])), theta=0.9,
                         w_cf=float(rng.choice([0.25, 0.30])), v_ref=0.01, tau=0.05)
    bias = None
    if rng.integers(0, 2):
        bias = (rng.standard_normal(E) * 0.5).astype(np.float32)
    return Workload(f"fuzz_{seed}", seed, T, d, E, f, f_shared, 1, p, _hidden(seed + 10_000, T, d),
                    b, np.array(offs, np.int32), np.array(acts, np.int32), m, hist, c1, c2,
                    router_bias=bias)
