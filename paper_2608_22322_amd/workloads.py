"""Parameter-list shapes and optimizer settings of the measured workloads.

Shapes follow the models the paper trains (TinyLlama-1.1B; a Llama-7B list
extends it). Tensors are listed as (rows, cols); a 1-D tensor has rows == 1.
Flattening is row-major, so a [out, in] weight is rows=out, cols=in.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Shape:
    name: str
    rows: int
    cols: int

    @property
    def n(self) -> int:
        return self.rows * self.cols

    @property
    def is_2d(self) -> bool:
        return self.rows > 1


def llama_shapes(layers: int, hidden: int, ffn: int, kv_dim: int, vocab: int) -> list[Shape]:
    out = [Shape("embed", vocab, hidden)]
    for l in range(layers):
        p = f"layer{l}."
        out += [
            Shape(p + "q", hidden, hidden),
            Shape(p + "k", kv_dim, hidden),
            Shape(p + "v", kv_dim, hidden),
            Shape(p + "o", hidden, hidden),
            Shape(p + "gate", ffn, hidden),
            Shape(p + "up", ffn, hidden),
            Shape(p + "down", hidden, ffn),
            Shape(p + "attn_norm", 1, hidden),
            Shape(p + "mlp_norm", 1, hidden),
        ]
    out += [Shape("norm", 1, hidden), Shape("lm_head", vocab, hidden)]
    return out


def tinyllama_shapes() -> list[Shape]:
    """TinyLlama-1.1B: 22 layers, hidden 2048, FFN 5632, 4 KV heads of 64, vocab 32000."""
    return llama_shapes(22, 2048, 5632, 256, 32000)


def llama7b_shapes() -> list[Shape]:
    """Llama-7B: 32 layers, hidden 4096, FFN 11008, 32 heads of 128, vocab 32000."""
    return llama_shapes(32, 4096, 11008, 4096, 32000)


def single_1024_shapes() -> list[Shape]:
    return [Shape("w", 1024, 1024)]


def total_params(shapes) -> int:
    return sum(s.n for s in shapes)


@dataclass(frozen=True)
class AdamWSettings:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01


@dataclass(frozen=True)
class AdafactorSettings:
    lr: float = 1e-3
    eps1: float = 1e-30
    clip_threshold: float = 1.0
    decay_rate: float = -0.8
    weight_decay: float = 0.0


@dataclass(frozen=True)
class CAMESettings:
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.999
    beta3: float = 0.9999
    eps1: float = 1e-30
    eps2: float = 1e-16
    clip_threshold: float = 1.0
    weight_decay: float = 0.0


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, gradient statistics and step count."""
    name: str
    shapes: list = field(default_factory=list)
    param_sigma: float = 0.02
    grad_sigma: float = 1e-3
    grad_bf16: bool = True
    zero_frac: float = 0.0
    steps: int = 1


def workload_1024() -> Workload:
    return Workload("adamw-1024x1024-fp32grad", single_1024_shapes(), grad_bf16=False,
                    zero_frac=0.05, steps=10)


def workload_tinyllama(zero_frac: float = 0.02) -> Workload:
    return Workload("tinyllama-1.1b", tinyllama_shapes(), zero_frac=zero_frac, steps=100)


def workload_llama7b() -> Workload:
    return Workload("llama-7b", llama7b_shapes(), zero_frac=0.01, steps=20)
