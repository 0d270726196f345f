"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI and
the oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle


def require_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_01784_amd import _lib
    _lib.lib()          # fail loudly if the HIP library is missing
    return torch


def note(msg):
    print(msg, flush=True, file=sys.stderr)


def layer_tolerance_check(got: np.ndarray, ref: np.ndarray, what: str,
                          rel_l2_tol=1e-2, max_abs_tol=2e-2):
    """The layer-output bar: relative L2 error <= 1e-2 and max-abs error <= 2e-2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = got - ref
    rel = np.linalg.norm(err) / max(np.linalg.norm(ref), 1e-30)
    mx = float(np.abs(err).max()) if err.size else 0.0
    note(f"{what}: rel_l2={rel:.3e} max_abs={mx:.3e}")
    assert rel <= rel_l2_tol, f"{what}: rel-L2 {rel:.3e}"
    assert mx <= max_abs_tol, f"{what}: max-abs {mx:.3e}"
    return rel, mx


def oracle_budget(w, params=None):
    p = w.params if params is None else params
    return oracle.assign_budget(w.block_idx, w.masked, w.hist_len, w.conf_prev1, w.conf_prev2,
                                w.seq_offsets, w.active_block, p)
