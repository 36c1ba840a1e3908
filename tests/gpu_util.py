"""Helpers for the GPU parity tests: the comparison rules against the oracle.

Codes: bit-exact, except an element whose oracle pre-rounding position lies
within NEAR of a rounding boundary (k + 1/2) may differ by exactly 1; such
elements are counted and reported. Metadata: bit-exact. Parameters: relative
tolerance per step count.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

NEAR = 1e-4


def require_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    import paper_2608_22322_amd as al

    al.lib()  # fails loudly if the HIP library is missing


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def near_boundary(y: np.ndarray) -> np.ndarray:
    y = np.asarray(y, dtype=np.float64)
    frac = y - np.floor(y)
    return np.abs(frac - 0.5) < NEAR


def compare_codes(gpu, orc, y, what: str) -> int:
    """Assert the code rule; returns the number of allowed near-boundary differences."""
    g = np.asarray(gpu).astype(np.int64)
    o = np.asarray(orc).astype(np.int64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    diff = np.nonzero(g != o)[0]
    if diff.size == 0:
        return 0
    n = y.shape[0]
    assert np.all(diff < n), f"{what}: padded codes differ at {diff[diff >= n][:8]}"
    yy = y[diff]
    ok = near_boundary(yy) & (np.abs(g[diff] - o[diff]) == 1)
    bad = diff[~ok]
    assert bad.size == 0, (f"{what}: {bad.size} codes differ away from a rounding boundary, e.g. idx {bad[:6]} "
                           f"gpu {g[bad[:6]]} oracle {o[bad[:6]]} y {y[bad[:6]]}")
    return int(diff.size)


def compare_bits(gpu, orc, what: str) -> None:
    g = np.ascontiguousarray(gpu, dtype=np.float32).view(np.uint32)
    o = np.ascontiguousarray(orc, dtype=np.float32).view(np.uint32)
    bad = np.nonzero(g != o)[0]
    assert bad.size == 0, (f"{what}: {bad.size} values differ, e.g. idx {bad[:6]} gpu "
                           f"{g.view(np.float32)[bad[:6]]} oracle {o.view(np.float32)[bad[:6]]}")


def compare_params(gpu, orc, rtol: float, what: str) -> float:
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(orc, dtype=np.float64)
    scale = np.sqrt(np.mean(o * o)) if o.size else 0.0
    err = np.abs(g - o)
    lim = rtol * (np.abs(o) + scale)
    worst = int(np.argmax(err - lim)) if o.size else 0
    assert np.all(err <= lim), (f"{what}: param error {err[worst]:.3e} > {lim[worst]:.3e} at {worst} "
                                f"(gpu {g[worst]!r} oracle {o[worst]!r})")
    nrm = np.linalg.norm(o)
    rel = float(np.linalg.norm(g - o) / nrm) if nrm > 0 else 0.0
    assert rel <= rtol, (what, rel)
    return rel


def to_np(t, n=None):
    import torch

    a = t.detach()
    if a.dtype == torch.int16:
        out = a.cpu().numpy().view(np.uint16)
    elif a.dtype == torch.bfloat16:
        out = a.view(torch.int16).cpu().numpy().view(np.uint16)
    else:
        out = a.cpu().numpy()
    return out if n is None else out[:n]
