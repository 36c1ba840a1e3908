"""APOLLO, the projected-state path (section 3.1; section 6 setup: rank 256, channel-wise scaling,
projection refreshed every 200 steps; Table 4: UF8 momentum with AL8 second moments).

Which tensors are projected: the 2-D weights of the transformer blocks. The token embedding, the
LM head and 1-D tensors keep full AdamW states (with the same codes). Under this layout the storage
accounting reproduces Table 4's APOLLO FP32 optimizer state on the TinyLlama list (2078.7 MiB).

A projected tensor of shape rows x cols keeps its moments over C x r elements, C = max(rows, cols)
channels of rank r: rows >= cols projects the columns (channels are rows), otherwise the rows
(channels are columns). The projection matrix is L x r (L = min(rows, cols)) with entries
N(0, 1/r); it is an input of the step (seeded, refreshed every `gap` steps by the caller).
"""
from __future__ import annotations

import math

from . import FP32, Spec, state_bytes as _codec_bytes

RANK = 256
GAP = 200
GAMMA = 1.01


def projected(name: str, rows: int, cols: int) -> bool:
    """APOLLO projects the 2-D weights of the transformer blocks, not the embedding or the LM head."""
    if rows <= 1:
        return False
    return name.rsplit(".", 1)[-1] not in ("embed", "lm_head")


def layout(rows: int, cols: int):
    """(right, C, L): channels = rows when rows >= cols (the columns are projected), else the columns."""
    right = rows >= cols
    return right, (rows if right else cols), (cols if right else rows)


def state_elems(rows: int, cols: int, rank: int = RANK) -> int:
    """Elements of each projected moment of a rows x cols tensor."""
    return rank * layout(rows, cols)[1]


def state_bytes(shapes, rank: int = RANK, m: Spec = Spec(FP32, 256), v: Spec = Spec(FP32, 2048),
                full_m: Spec | None = None, full_v: Spec | None = None) -> int:
    """Optimizer-state bytes of APOLLO over a tensor list: projected moments (specs m, v) of the
    projected tensors plus full AdamW moments (full_m, full_v; default: the same specs) of the rest."""
    full_m = full_m or m
    full_v = full_v or v
    total = 0
    for s in shapes:
        if projected(s.name, s.rows, s.cols):
            n = state_elems(s.rows, s.cols, rank)
            total += _codec_bytes(m.codec, n, m.block) + _codec_bytes(v.codec, n, v.block)
        else:
            total += _codec_bytes(full_m.codec, s.n, full_m.block) + _codec_bytes(full_v.codec, s.n, full_v.block)
    return total


class ApolloStep:
    """One APOLLO step per call over a list of ParamState (param, grad, rows, cols) with names: projected
    tensors take al_apollo_step (projected moments, projection matrix and limiter state allocated here),
    the others al_adamw_step with the same codes (their ParamState m, v are allocated here too). The
    projection of tensor i for steps (e - 1) * gap + 1 .. e * gap is drawn from the seeded stream
    (seed, projection, i, e - 1) with entries N(0, 1/rank)."""

    def __init__(self, states, names, cfg=None, gap: int = GAP, seed: int | None = None, device="cuda"):
        import torch

        from . import (Spec, adamw_cfg, adamw_workspace_bytes, alloc_state, apollo_cfg, apollo_tensor_array,
                       apollo_workspace_bytes, synth, tensor_array, workspace)

        self.cfg = cfg or apollo_cfg()
        self.gap = gap
        self.seed = synth.BASE_SEED if seed is None else seed
        r = self.cfg.rank
        mspec = Spec(self.cfg.m.codec, self.cfg.m.block, self.cfg.m.log_floor)
        vspec = Spec(self.cfg.v.codec, self.cfg.v.block, self.cfg.v.log_floor)
        self.proj_idx, self.full_idx = [], []
        self.items, self.proj = [], []
        for i, (st, name) in enumerate(zip(states, names)):
            if projected(name, st.rows, st.cols):
                right, C, L = layout(st.rows, st.cols)
                m, mm = alloc_state(C * r, mspec, device)
                v, vm = alloc_state(C * r, vspec, device)
                pj = torch.empty(L * r, dtype=torch.float32, device=device)
                ns = torch.zeros(4, dtype=torch.float32, device=device)
                self.items.append((st.param, st.grad, st.rows, st.cols, pj, m, mm, v, vm, ns))
                self.proj.append((i, L, pj))
                self.proj_idx.append(i)
            else:
                st.m, st.m_meta = alloc_state(st.rows * st.cols, mspec, device)
                st.v, st.v_meta = alloc_state(st.rows * st.cols, vspec, device)
                self.full_idx.append(i)
        self.arr = apollo_tensor_array(self.items)
        nbytes = apollo_workspace_bytes(self.arr, len(self.items), self.cfg)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.full_states = [states[i] for i in self.full_idx]
        self.full_arr = tensor_array(self.full_states)
        self.full_cfg = adamw_cfg(lr=self.cfg.lr, beta1=self.cfg.beta1, beta2=self.cfg.beta2, eps=self.cfg.eps,
                                  weight_decay=self.cfg.weight_decay, grad_bf16=self.cfg.grad_dtype == 1,
                                  m=mspec, v=vspec)
        self.full_ws = workspace(adamw_workspace_bytes(self.full_states, self.full_cfg, arr=self.full_arr), device)
        self._epoch = None

    def refresh(self, step: int, stream=None) -> None:
        """Draw the projections of the refresh period holding `step` (no-op within a period)."""
        from . import synth, synth_normal

        e = (step - 1) // self.gap
        if e == self._epoch:
            return
        for i, L, pj in self.proj:
            synth_normal(pj, synth.proj_key(i, e, self.seed), 1.0 / math.sqrt(self.cfg.rank), stream=stream)
        self._epoch = e

    def step(self, t: int, stream=None) -> None:
        from . import adamw_step, apollo_step

        self.refresh(t, stream)
        apollo_step(self.arr, len(self.items), self.cfg, t, self.ws, stream)
        if self.full_states:
            adamw_step(self.full_states, self.full_cfg, t, self.full_ws, stream=stream, arr=self.full_arr)
