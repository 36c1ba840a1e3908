"""Seeded workload inputs in device memory, and the same values on the host.

Parameters of 2-D tensors start N(0, 0.02); 1-D (normalization) tensors start
at 1.0. Gradients of tensor i at step t use the stream (seed, grad, i, t);
a fixed per-tensor zero mask (seed, mask, i) makes a given fraction of
entries exactly zero. Device tensors are filled by the library's
``al_synth_normal``; :func:`host_param` / :func:`host_grad` regenerate any
index range on the host with identical bits (synth.py).
"""
from __future__ import annotations

import numpy as np

from . import synth
from .workloads import Shape, Workload


def host_param(i: int, shape: Shape, idx, sigma: float = 0.02, seed: int = synth.BASE_SEED) -> np.ndarray:
    idx = np.asarray(idx)
    if not shape.is_2d:
        return np.ones(idx.shape[0], np.float32)
    return synth.normal_f32(synth.param_key(i, seed), idx, sigma)


def grad_mask_frac(w: Workload, step: int) -> float:
    """Fraction of exact-zero gradient entries at a step. The 1024x1024 workload holds its 5% dormant
    entries at zero for the first five steps only."""
    if w.name.startswith("adamw-1024x1024") and step > 5:
        return 0.0
    return w.zero_frac


def host_grad(i: int, w: Workload, step: int, idx, seed: int = synth.BASE_SEED) -> np.ndarray:
    """Gradient values (fp32, or bf16 bit patterns as uint16 when the workload uses bf16)."""
    g = synth.normal_f32(synth.grad_key(i, step, seed), np.asarray(idx), w.grad_sigma,
                         synth.mask_key(i, seed), grad_mask_frac(w, step))
    return synth.to_bf16_bits(g) if w.grad_bf16 else g


def device_param(i: int, shape: Shape, device="cuda", sigma: float = 0.02, seed: int = synth.BASE_SEED):
    import torch

    from . import synth_normal

    p = torch.empty(max(shape.n, 4), dtype=torch.float32, device=device)
    if not shape.is_2d:
        p.fill_(1.0)
    else:
        synth_normal(p[: shape.n], synth.param_key(i, seed), sigma)
    return p


def device_grad_buffer(shape: Shape, w: Workload, device="cuda"):
    import torch

    return torch.empty(max(shape.n, 8), dtype=torch.bfloat16 if w.grad_bf16 else torch.float32, device=device)


def fill_grad(buf, i: int, shape: Shape, w: Workload, step: int, seed: int = synth.BASE_SEED) -> None:
    from . import synth_normal

    synth_normal(buf[: shape.n], synth.grad_key(i, step, seed), w.grad_sigma, synth.mask_key(i, seed),
                 grad_mask_frac(w, step))
