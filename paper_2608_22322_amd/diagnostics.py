"""Relative update error (section 3.2, Eq. update_error).

E_upd = ||U(S_hat, G) - U(S, G)||_2 / (||U(S, G)||_2 + eps): the update an optimizer
step produces from a state reconstructed from its codes, S_hat, against the update from
the exact state S, for the same gradient G. Both updates come from the library's step
kernels (the reference run uses FP32 states, the other the state codes produced by
al_quantize from the same values), starting from zero parameters so the parameters
after the step are the updates themselves; al_diff_norms forms the two sums of squares.
"""
from __future__ import annotations

import math

from . import (FP32, ParamState, StateSpec, adafactor_step, adafactor_workspace_bytes, adamw_step, alloc_state,
               came_step, came_workspace_bytes, diff_norms, DIFF_NORMS_OUT, quantize, tensor_array)

ROLES = ("m", "v", "vr", "vc", "cr", "cc")


def _role_spec(kind: str, cfg, role: str) -> StateSpec:
    if role == "m":
        return cfg.m
    if role in ("cr", "cc"):
        return cfg.conf
    return cfg.v


def _fp32_cfg(kind: str, cfg):
    out = type(cfg).from_buffer_copy(cfg)
    for n in {"adamw": ("m", "v"), "adafactor": ("v",), "came": ("m", "v", "conf")}[kind]:
        ss = getattr(cfg, n)
        setattr(out, n, StateSpec(FP32, ss.block, ss.log_floor))
    return out


def _run(kind: str, states, cfg, t: int, device, stream) -> None:
    import torch

    arr = tensor_array(states)
    if kind == "adamw":
        adamw_step(states, cfg, t, stream=stream, arr=arr)
        return
    nbytes = (adafactor_workspace_bytes if kind == "adafactor" else came_workspace_bytes)(states, cfg, arr=arr)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    if kind == "adafactor":
        adafactor_step(states, cfg, t, ws, stream=stream, arr=arr)
    else:
        came_step(states, cfg, t, ws, stream=stream, arr=arr)


def update_error(kind: str, ref_states, cfg, t: int, eps: float = 1e-30, stream=None) -> float:
    """E_upd of one step (kind: 'adamw', 'adafactor', 'came') over a tensor list.

    ref_states: ParamState list whose state buffers (m, v, vr, vc, cr, cc as the optimizer
    uses them) hold the exact states in FP32; grad holds G; param is ignored. cfg: the
    optimizer config with the state codes under test (its FP32 counterpart is derived). The
    reference states are not modified."""
    import torch

    if kind not in ("adamw", "adafactor", "came"):
        raise ValueError(kind)
    device = ref_states[0].grad.device
    ref, quant = [], []
    for st in ref_states:
        n = st.rows * st.cols
        r = ParamState(torch.zeros(max(n, 4), dtype=torch.float32, device=device), st.grad, st.rows, st.cols)
        q = ParamState(torch.zeros(max(n, 4), dtype=torch.float32, device=device), st.grad, st.rows, st.cols)
        for role in ROLES:
            buf = getattr(st, role)
            if buf is None:
                continue
            length = n if role in ("m", "v") else (st.rows if role in ("vr", "cr") else st.cols)
            setattr(r, role, buf.clone())
            ss = _role_spec(kind, cfg, role)
            if ss.codec == FP32:
                setattr(q, role, buf.clone())
                continue
            from . import Spec

            codes, meta = alloc_state(length, Spec(ss.codec, ss.block, ss.log_floor), device)
            quantize(ss.codec, buf[:length], ss.block, ss.log_floor, codes, meta, stream=stream)
            setattr(q, role, codes)
            setattr(q, role + "_meta", meta)
        ref.append(r)
        quant.append(q)
    _run(kind, ref, _fp32_cfg(kind, cfg), t, device, stream)
    _run(kind, quant, cfg, t, device, stream)
    out = torch.empty(DIFF_NORMS_OUT, dtype=torch.float64, device=device)
    num = den = 0.0
    for r, q, st in zip(ref, quant, ref_states):
        n = st.rows * st.cols
        diff_norms(q.param[:n], r.param[:n], out, stream=stream)
        s = out[:2].cpu()
        num += float(s[0])
        den += float(s[1])
    return math.sqrt(num) / (math.sqrt(den) + eps)


__all__ = ["update_error"]
