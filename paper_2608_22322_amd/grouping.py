"""Parameter-grouping policies (section 6, experimental setup).

G0 applies the selected state codes to every tensor. G1 sets apart one-dimensional
tensors, biases, normalisation parameters, the token embedding and the language-model
head, keeps their optimizer states unquantized (FP32) and quantizes the rest. A grouped
step is one library call per group, each with that group's state specs: the kernels
are the same, only the codes differ.
"""
from __future__ import annotations

from dataclasses import dataclass

from . import (AL8, AL16, FP32, UF8, Spec, StateSpec, adafactor_step, adafactor_workspace_bytes, adamw_step,
               adamw_workspace_bytes, alloc_state, came_step, came_workspace_bytes, state_bytes, tensor_array)

POLICIES = ("G0", "G1")


def g1_protected(name: str, rows: int, cols: int) -> bool:
    """Membership of the G1 protected group: 1-D tensors, biases, norms, embedding, LM head."""
    if rows <= 1:
        return True
    leaf = name.rsplit(".", 1)[-1]
    return leaf in ("embed", "lm_head") or "norm" in leaf or leaf.endswith("bias")


def protected_flags(shapes, policy: str) -> list[bool]:
    if policy not in POLICIES:
        raise ValueError(f"unknown grouping policy {policy!r}")
    if policy == "G0":
        return [False] * len(shapes)
    return [g1_protected(s.name, s.rows, s.cols) for s in shapes]


def fp32_spec(spec) -> "Spec":
    """The unquantized counterpart of a state spec (block and floor kept; FP32 ignores them)."""
    return Spec(FP32, spec.block, spec.log_floor)


def _with_fp32_states(kind: str, cfg):
    """A copy of an optimizer config whose state specs are all FP32."""
    out = type(cfg).from_buffer_copy(cfg)
    names = {"adamw": ("m", "v"), "adafactor": ("v",), "came": ("m", "v", "conf")}[kind]
    for n in names:
        ss = getattr(cfg, n)
        setattr(out, n, StateSpec(FP32, ss.block, ss.log_floor))
    return out


@dataclass
class _Group:
    idx: list
    arr: object
    cfg: object
    ws: object


class GroupedStep:
    """One optimizer step (kind: 'adamw', 'adafactor' or 'came') over a list of ParamState under a
    protection mask: unprotected tensors take cfg's codes, protected ones FP32 states (their
    ParamState buffers must be allocated accordingly, e.g. with attach_states)."""

    def __init__(self, kind: str, states, cfg, protected, device=None):
        import torch

        if kind not in ("adamw", "adafactor", "came"):
            raise ValueError(kind)
        self.kind = kind
        self.groups = []
        for prot in (False, True):
            idx = [i for i, p in enumerate(protected) if p == prot]
            if not idx:
                continue
            sts = [states[i] for i in idx]
            gcfg = _with_fp32_states(kind, cfg) if prot else cfg
            arr = tensor_array(sts)
            fn = {"adamw": adamw_workspace_bytes, "adafactor": adafactor_workspace_bytes,
                  "came": came_workspace_bytes}[kind]
            ws = torch.empty(max(fn(sts, gcfg, arr=arr), 256), dtype=torch.uint8, device=device or "cuda")
            self.groups.append(_Group(idx, arr, gcfg, ws))
        self.states = states

    def step(self, t: int, stream=None) -> None:
        for g in self.groups:
            sts = [self.states[i] for i in g.idx]
            if self.kind == "adamw":
                adamw_step(sts, g.cfg, t, g.ws, stream=stream, arr=g.arr)
            elif self.kind == "adafactor":
                adafactor_step(sts, g.cfg, t, g.ws, stream=stream, arr=g.arr)
            else:
                came_step(sts, g.cfg, t, g.ws, stream=stream, arr=g.arr)


def attach_states(states, kind: str, specs: dict, protected, device="cuda") -> None:
    """Allocate fresh (all-zero) state buffers on each ParamState (param, grad, rows, cols set) for
    an optimizer kind: specs maps roles ('m', 'v', 'conf') to Spec; protected tensors get FP32."""
    for st, prot in zip(states, protected):
        sp = {r: (fp32_spec(v) if prot else v) for r, v in specs.items()}
        n = st.rows * st.cols
        if kind in ("adamw", "came"):
            st.m, st.m_meta = alloc_state(n, sp["m"], device)
        if kind == "adamw":
            st.v, st.v_meta = alloc_state(n, sp["v"], device)
        elif st.rows > 1:
            st.vr, st.vr_meta = alloc_state(st.rows, sp["v"], device)
            st.vc, st.vc_meta = alloc_state(st.cols, sp["v"], device)
            if kind == "came":
                st.cr, st.cr_meta = alloc_state(st.rows, sp["conf"], device)
                st.cc, st.cc_meta = alloc_state(st.cols, sp["conf"], device)
        else:
            st.v, st.v_meta = alloc_state(n, sp["v"], device)


def grouped_state_bytes(shapes, kind: str, specs: dict, policy: str, fp32_1d: bool = True) -> int:
    """Optimizer-state bytes of a tensor list under a policy (codes padded per tensor / vector).
    specs: state role -> Spec ('m', 'v' for AdamW and CAME momentum / second moment; 'conf' for CAME).
    Factored roles apply to 2-D tensors (rows x cols vectors); fp32_1d keeps 1-D states FP32 under G0
    as well (the grouping the paper's G0 storage figures imply)."""
    prot = protected_flags(shapes, policy)
    total = 0
    for s, p in zip(shapes, prot):
        fp = p or (fp32_1d and not s.is_2d)
        if kind == "adamw":
            total += 8 * s.n if fp else sum(state_bytes(specs[r].codec, s.n, specs[r].block) for r in ("m", "v"))
            continue
        roles = ("v",) if kind == "adafactor" else ("v", "conf")
        if kind == "came":
            total += 4 * s.n if fp else state_bytes(specs["m"].codec, s.n, specs["m"].block)
        for r in roles:
            if not s.is_2d:
                if r == "v":
                    total += 4 * s.n if fp else state_bytes(specs[r].codec, s.n, specs[r].block)
                continue
            for L in (s.rows, s.cols):
                total += 4 * L if fp else state_bytes(specs[r].codec, L, specs[r].block)
    return total


__all__ = ["POLICIES", "g1_protected", "protected_flags", "fp32_spec", "GroupedStep", "attach_states",
           "grouped_state_bytes"]
