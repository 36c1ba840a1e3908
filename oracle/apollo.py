"""TEST INFRASTRUCTURE -- the CPU oracle of the APOLLO projected-state step. Not part of the product path.

Plain binary64 numpy, written from the paper's description of APOLLO as a projected-state optimizer
(section 3.1: first and second moments kept in a low-rank projection of the gradient, from which a
channel-wise scale of the original gradient is derived; section 6 setup: rank 256, channel-wise
scaling, projection refreshed every 200 steps; Table 4: UF8 momentum with AL8 second moments, block
2048). The paper gives no formulas for APOLLO; the steps below are the published APOLLO method as
this repository reads it (each reading is listed with the design notes):

  A   = G (rows >= cols: the columns are projected, channels are the rows)
        or G^T (rows < cols: the rows are projected, channels are the columns)   -- C x L
  R   = fl32(A Pi)                Pi: L x r, entries N(0, 1/r), an input        -- C x r
  M, V, Rt: one AdamW step on R with zero parameters, lr 1, no weight decay:
        M = fl32(b1 M^ + (1 - b1) R), V = fl32(b2 V^ + (1 - b2) R^2),
        Rt = fl32((M / bc1) / (sqrt(V / bc2) + eps)); M and V re-encoded with their codes
  s_c = ||Rt_c|| / (||R_c|| + 1e-8)                                              -- channel scale
  Gs  = A s  (each channel of G times its scale), n = ||Gs||
  limiter (steps >= 2): lam = max(n / (prev + 1e-8), gamma) / gamma, prev <- fl32(n / lam);
        step 1: lam = 1, prev <- fl32(n)
  p   = fl32(p (1 - lr wd) - lr (g s_c / lam))      (s_c / lam formed first, in binary64)

The moments reuse the AdamW oracle (``oracle.adamw_step``), so the codes follow the same
definitions (section 4). APOLLO's own implementation is not available: against it this step is
parity unpinned; the CPU tests pin it by brute-force projection, an identity projection (then the
projected direction is torch.optim.AdamW's), the step-1 channel scale and the limiter in closed
form, and the two projection sides under transposition. Sums are exact (``oracle.exact_sum``). Only tests, the smoke check and the
benchmark's CPU baseline may import this module; it shares no code with the HIP library.
"""
from __future__ import annotations

import math

import numpy as np

from . import State, adamw_step, exact_sum

LIMIT_EPS = 1e-8   # APOLLO's guard in the channel ratio and the limiter ratio


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def layout(rows: int, cols: int):
    """(right, C, L): right projection (channels = rows) when rows >= cols; C channels of L inputs each."""
    right = rows >= cols
    return right, (rows if right else cols), (cols if right else rows)


def project(g64: np.ndarray, rows: int, cols: int, proj: np.ndarray) -> np.ndarray:
    """R = fl32(A Pi) as a C x r float32 array (channel-major)."""
    right, C, L = layout(rows, cols)
    G = g64.reshape(rows, cols)
    A = G if right else G.T
    assert proj.shape[0] == L
    return (A @ proj.astype(np.float64)).astype(np.float32)


def apollo_step(p: np.ndarray, g, rows: int, cols: int, proj: np.ndarray, m: State, v: State, t: int,
                prev: np.ndarray, lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0, gamma=1.01):
    """One APOLLO step on one 2-D tensor, in place (p, m, v, prev). g: float32 array or uint16 bf16 bits.
    prev: float32 array of one element (the limiter's previous update norm). gamma <= 0 disables the
    limiter. Returns the intermediate quantities for tests."""
    assert p.dtype == np.float32 and p.shape[0] == rows * cols
    g = np.asarray(g)
    g64 = bf16_to_f64(g) if g.dtype == np.uint16 else g.astype(np.float32).astype(np.float64)
    right, C, L = layout(rows, cols)
    r = proj.shape[1]
    R = project(g64, rows, cols, proj)                       # C x r
    z = np.zeros(C * r, dtype=np.float32)
    adamw_step(z, R.ravel(), m, v, t, lr=1.0, beta1=beta1, beta2=beta2, eps=eps, wd=0.0)
    Rt = -z.reshape(C, r)                                    # the AdamW direction on R
    s = np.empty(C)
    for c in range(C):
        num = math.sqrt(exact_sum(Rt[c].astype(np.float64) ** 2))
        den = math.sqrt(exact_sum(R[c].astype(np.float64) ** 2)) + LIMIT_EPS
        s[c] = num / den
    G = g64.reshape(rows, cols)
    A = G if right else G.T
    Gs = A * s[:, None]
    n = math.sqrt(exact_sum((Gs * Gs).ravel()))
    lam = 1.0
    if gamma > 0:
        if t >= 2:
            lam = max(n / (float(prev[0]) + LIMIT_EPS), gamma) / gamma
            prev[0] = np.float32(n / lam)
        else:
            prev[0] = np.float32(n)
    sl = s / lam                                             # per channel, binary64
    scale = sl[:, None] if right else sl[None, :]            # broadcast over W's layout
    upd = G * scale
    pd = p.astype(np.float64).reshape(rows, cols) * (1.0 - lr * wd) - lr * upd
    p[:] = pd.astype(np.float32).ravel()
    return {"R": R, "Rt": Rt, "s": s, "norm": n, "lam": lam}
