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
