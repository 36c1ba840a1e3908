"""Controlled probes of section 5 on the oracle, and their seeded synthetic inputs.

The paper's probes draw states from distributions it describes only in words: three
log-normal regimes in base-2 space (narrow, medium, wide), a sparse regime with exact
zeros, and, for the temporal probe, a K-step second-moment EMA (new-observation weight
0.001) fed with fresh gradients each step. The stand-ins here:

* regimes: log2 v ~ N(mu, sigma^2) per element, narrow (-16, 0.15), medium (-12, 2.5),
  wide (-60, 3.0); a 2048-element block spans about 1, 18 and 21 binary orders;
* sparse: the narrow regime with a seeded 90% of entries set to exact zero;
* operator gradient: g = sqrt(v) * z with z ~ N(0, 1) and g = 0 where v = 0, so every live
  element carries the same expected update magnitude;
* temporal probe: i.i.d. N(0, sigma^2) gradients, a fresh draw per step.

The operator of the single-step probes is the inverse square root that consumes V: an
AdamW step with beta1 = 0 (the update is g / (sqrt(v_new) + eps)) at a step count where
both bias corrections are exactly 1, from zero parameters with lr 1 and no decay, so the
parameter after the step is minus the update. The temporal probe runs AdamW with FP32
momentum, as the paper's does.

Oracle-side versions of the protocols live here; the library's own are in
paper_2608_22322_amd.diagnostics.
"""
from __future__ import annotations

import math

import numpy as np

import oracle
from paper_2608_22322_amd import synth

REGIMES = {"narrow": (-16.0, 0.15), "medium": (-12.0, 2.5), "wide": (-60.0, 3.0)}
PROBE_FLOOR = -126.0   # no floor inside the probes' range: the block interval is the data's own
OPERATOR_T = 1_000_000  # 1 - 0.999^t rounds to 1 in binary64


def lognormal(key: int, n: int, mu: float, sigma: float) -> np.ndarray:
    z = synth.normal_f32(key, n, 1.0).astype(np.float64)
    return (2.0 ** (mu + sigma * z)).astype(np.float32)


def regime_state(name: str, seed: int, n: int = 2048) -> np.ndarray:
    mu, sigma = REGIMES[name]
    return lognormal(synth.state_key(seed, 1), n, mu, sigma)


def sparse_state(seed: int, n: int = 2048, zero_frac: float = 0.9) -> np.ndarray:
    v = regime_state("narrow", seed, n)
    keep = synth.normal_f32(synth.state_key(seed, 3), n, 1.0, mask_key=synth.state_key(seed, 4),
                            mask_frac=zero_frac)
    v[keep == 0] = 0.0
    return v


def operator_grad(v: np.ndarray, seed: int) -> np.ndarray:
    z = synth.normal_f32(synth.state_key(seed, 2), v.shape[0], 1.0).astype(np.float64)
    g = (np.sqrt(v.astype(np.float64)) * z).astype(np.float32)
    g[v == 0] = 0.0
    return g


def drift_grad(seed: int, t: int, n: int, sigma: float) -> np.ndarray:
    return synth.normal_f32(synth.grad_key(seed, t), n, sigma)


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    d = a.astype(np.float64) - b.astype(np.float64)
    return math.sqrt(math.fsum((d * d).tolist())) / math.sqrt(math.fsum((b.astype(np.float64) ** 2).tolist()))


def oracle_state_error(v: np.ndarray, bits: int, block: int, floor: float = PROBE_FLOOR) -> float:
    codes, meta, _ = oracle.al_quantize(bits, v, block, floor)
    return rel_l2(oracle.al_dequantize(bits, codes, meta, v.shape[0], block), v)


def oracle_operator_error(v: np.ndarray, g: np.ndarray, bits: int, block: int,
                          floor: float = PROBE_FLOOR) -> float:
    """E_upd of the inverse-square-root operator with v coded by AL<bits> against exact v."""
    n = v.shape[0]
    codec = oracle.AL8 if bits == 8 else oracle.AL16
    pr, pq = np.zeros(n, np.float32), np.zeros(n, np.float32)
    mr, vr = oracle.State(oracle.FP32, n), oracle.State(oracle.FP32, n)
    vr.codes[:] = v
    oracle.adamw_step(pr, g, mr, vr, OPERATOR_T, lr=1.0, beta1=0.0, wd=0.0)
    mq, vq = oracle.State(oracle.FP32, n), oracle.State(codec, n, block, floor)
    vq.codes[:], vq.meta[:], _ = oracle.al_quantize(bits, v, block, floor)
    oracle.adamw_step(pq, g, mq, vq, OPERATOR_T, lr=1.0, beta1=0.0, wd=0.0)
    return rel_l2(pq, pr)


def oracle_adamw_drift(n: int, steps: int, block: int, bits: int = 8, seed: int = 5, sigma: float = 1e-3,
                       floor: float | None = None, beta2: float = 0.999, eps: float = 1e-8):
    """Temporal probe on the oracle: AdamW with FP32 momentum and an FP32 or AL<bits> second moment
    over the same gradients; steps 1..K-1 at lr 0, step K from zero parameters at lr 1e-3.
    Returns (V drift, E_upd of step K)."""
    floor = float(np.float32(2 * math.log2(eps))) if floor is None else floor
    codec = oracle.AL8 if bits == 8 else oracle.AL16
    pr, pq = np.zeros(n, np.float32), np.zeros(n, np.float32)
    mr, vr = oracle.State(oracle.FP32, n), oracle.State(oracle.FP32, n)
    mq, vq = oracle.State(oracle.FP32, n), oracle.State(codec, n, block, floor)
    for t in range(1, steps + 1):
        g = drift_grad(seed, t, n, sigma)
        lr = 1e-3 if t == steps else 0.0
        oracle.adamw_step(pr, g, mr, vr, t, lr=lr, beta2=beta2, eps=eps, wd=0.0)
        oracle.adamw_step(pq, g, mq, vq, t, lr=lr, beta2=beta2, eps=eps, wd=0.0)
    return rel_l2(vq.decode(), vr.codes), rel_l2(pq, pr)


def oracle_adafactor_drift(rows: int, cols: int, steps: int, bits: int, block: int, seed: int = 6,
                           sigma: float = 1e-3, eps1: float = 1e-30):
    """Temporal probe for a factored second moment (Adafactor, one rows x cols tensor).
    Returns ({"vr": drift, "vc": drift}, E_upd of step K)."""
    n = rows * cols
    floor = float(np.float32(math.log2(eps1)))
    codec = oracle.AL8 if bits == 8 else oracle.AL16
    pr, pq = np.zeros(n, np.float32), np.zeros(n, np.float32)
    rr, rc = oracle.State(oracle.FP32, rows), oracle.State(oracle.FP32, cols)
    qr, qc = oracle.State(codec, rows, block, floor), oracle.State(codec, cols, block, floor)
    for t in range(1, steps + 1):
        g = drift_grad(seed, t, n, sigma)
        lr = 1e-3 if t == steps else 0.0
        oracle.adafactor_step(pr, g, rows, cols, rr, rc, None, t, lr=lr, eps1=eps1)
        oracle.adafactor_step(pq, g, rows, cols, qr, qc, None, t, lr=lr, eps1=eps1)
    return {"vr": rel_l2(qr.decode(), rr.codes), "vc": rel_l2(qc.decode(), rc.codes)}, rel_l2(pq, pr)
