"""Seeded, counter-based synthetic inputs (host side).

This module is the only code shared by the CPU oracle's tests and the HIP
path. It holds none of the optimizer's or the codec's arithmetic: it only
turns (seed, stream, tensor, step, element index) into parameter and gradient
values. The device kernel ``al_synth_fill`` in the HIP library implements the
same definition, element for element, so that full-size inputs can be made in
HBM while any sampled element can be regenerated here for the oracle.

Definition (every operation is exact integer arithmetic or one IEEE binary32
multiply, so host and device agree bit for bit):

* ``mix64`` is the SplitMix64 output function (Steele, Lea & Flood, 2014).
* A stream key is a 64-bit value derived on the host from the base seed and
  a path of small integers (see :func:`stream_key`); the device gets the key.
* Element ``e`` of a stream draws three words
  ``w_k = mix64(key + (3e + k + 1) * GAMMA)``, ``k = 0, 1, 2`` (mod 2^64),
  and sums their twelve 16-bit fields: ``S`` in ``[0, 12 * 65535]``.
  ``S - 393210`` is a centred Irwin-Hall(12) variate with standard deviation
  ``sqrt(65536^2 - 1)``; it is exact in binary32.
* The value is ``fl32(fl32(S - 393210) * c)`` with ``c = fl32(sigma /
  sqrt(65536^2 - 1))``: an approximately normal draw with standard deviation
  ``sigma``, bounded at about 6 sigma.
* A zero mask draws ``z = mix64(mask_key + (e + 1) * GAMMA)``; the element is
  exactly zero when ``z < floor(frac * 2^64)``.
* bfloat16 output rounds the binary32 value to nearest-even on its bit
  pattern.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
M64 = (1 << 64) - 1
IH_CENTER = 393210  # 12 * 65535 / 2
IH_SD = math.sqrt(65536.0 * 65536.0 - 1.0)

BASE_SEED = 921  # the paper's training seed (experimental setup, first subsection of section 6)

# stream tags
TAG_PARAM = 1
TAG_GRAD = 2
TAG_MASK = 3
TAG_STATE = 4
TAG_PROJ = 5


def mix64_int(z: int) -> int:
    """SplitMix64 output function on a Python int (mod 2^64)."""
    z &= M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function on a uint64 array (wrapping arithmetic)."""
    z = z.astype(np.uint64, copy=True)
    z ^= z >> np.uint64(30)
    z *= np.uint64(0xBF58476D1CE4E5B9)
    z ^= z >> np.uint64(27)
    z *= np.uint64(0x94D049BB133111EB)
    z ^= z >> np.uint64(31)
    return z


def stream_key(seed: int, tag: int, *path: int) -> int:
    """64-bit key of the stream (seed, tag, path...)."""
    k = mix64_int((seed + GAMMA) & M64)
    k = mix64_int(k ^ tag)
    for p in path:
        k = mix64_int((k + (p + 1) * GAMMA) & M64)
    return k


def normal_scale(sigma: float) -> np.float32:
    """binary32 multiplier that maps a centred Irwin-Hall(12) integer to N(0, sigma)."""
    return np.float32(sigma / IH_SD)


def mask_threshold(frac: float) -> int:
    """Elements whose mask word is below this value are exactly zero."""
    if frac <= 0.0:
        return 0
    return min(int(math.floor(frac * 2.0**64)), M64)


def _indices(n_or_idx) -> np.ndarray:
    if isinstance(n_or_idx, (int, np.integer)):
        return np.arange(int(n_or_idx), dtype=np.uint64)
    return np.asarray(n_or_idx, dtype=np.uint64)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_f32(key: int, n_or_idx, sigma: float, mask_key: int = 0, mask_frac: float = 0.0,
               chunk: int = 1 << 20) -> np.ndarray:
    """binary32 draws for element indices ``range(n)`` (or an index array). Chunks of the index range are
    drawn on a few threads (numpy's integer kernels release the interpreter lock); every element depends
    only on its own index, so the result does not depend on the split."""
    idx = _indices(n_or_idx)
    out = np.empty(idx.shape[0], dtype=np.float32)
    c = normal_scale(sigma)
    thr = mask_threshold(mask_frac)
    g = np.uint64(GAMMA)
    kk = np.uint64(key)

    def fill(s: int) -> None:
        e = idx[s:s + chunk]
        base = e * np.uint64(3)
        total = np.zeros(e.shape[0], dtype=np.int64)
        for k in range(3):
            w = mix64(kk + (base + np.uint64(k + 1)) * g)
            for sh in (0, 16, 32, 48):
                total += ((w >> np.uint64(sh)) & np.uint64(0xFFFF)).astype(np.int64)
        zi = (total - IH_CENTER).astype(np.float32)
        v = zi * c  # one binary32 multiply, round to nearest even
        if thr > 0:
            z = mix64(np.uint64(mask_key) + (e + np.uint64(1)) * g)
            v[z < np.uint64(thr)] = np.float32(0.0)
        out[s:s + chunk] = v

    starts = range(0, idx.shape[0], chunk)
    if len(starts) <= 1:
        for s in starts:
            fill(s)
    else:
        with ThreadPoolExecutor(min(_threads(), len(starts))) as ex:
            list(ex.map(fill, starts))
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary32 to bfloat16 (nearest even); returns the uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------
# Keys for the workloads: parameter init, per-step gradient, fixed zero mask.
# ----------------------------------------------------------------------------

def param_key(tensor: int, seed: int = BASE_SEED) -> int:
    return stream_key(seed, TAG_PARAM, tensor)


def grad_key(tensor: int, step: int, seed: int = BASE_SEED) -> int:
    return stream_key(seed, TAG_GRAD, tensor, step)


def mask_key(tensor: int, seed: int = BASE_SEED) -> int:
    return stream_key(seed, TAG_MASK, tensor)


def state_key(tensor: int, which: int, seed: int = BASE_SEED) -> int:
    return stream_key(seed, TAG_STATE, tensor, which)


def proj_key(tensor: int, epoch: int, seed: int = BASE_SEED) -> int:
    """Stream of the APOLLO projection matrix of a tensor for one refresh period (epoch = (t - 1) // gap)."""
    return stream_key(seed, TAG_PROJ, tensor, epoch)


def proj_matrix(tensor: int, epoch: int, L: int, rank: int, seed: int = BASE_SEED) -> np.ndarray:
    """L x rank projection with entries N(0, 1/rank) (float32, row-major)."""
    return normal_f32(proj_key(tensor, epoch, seed), L * rank, 1.0 / math.sqrt(rank)).reshape(L, rank)
