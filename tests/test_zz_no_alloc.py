"""The allocation-free AdamW entry point (al_adamw_step_noalloc) against al_adamw_step.

Both run the same kernels, so on identical inputs their parameters, codes and
metadata must agree bit for bit. Calls in a row on one stream share the
library's fixed table: a smaller list after a larger one, and a list at the
table's limit of 4096 tensors, must not see stale entries.
"""
import numpy as np
import pytest

from paper_2608_22322_amd import data
from paper_2608_22322_amd.workloads import Shape, Workload

from .gpu_util import log, require_gpu, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _states(al, dev, shapes, w, mspec, vspec):
    out = []
    for i, s in enumerate(shapes):
        m, mm = al.alloc_state(s.n, mspec, dev)
        v, vm = al.alloc_state(s.n, vspec, dev)
        out.append(al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols,
                                 m=m, m_meta=mm, v=v, v_meta=vm))
    return out


def _same(a_states, b_states, tag):
    for k, (a, b) in enumerate(zip(a_states, b_states)):
        for name in ("param", "m", "m_meta", "v", "v_meta"):
            x, y = to_np(getattr(a, name)), to_np(getattr(b, name))
            xb = np.ascontiguousarray(x).view(np.uint8)
            yb = np.ascontiguousarray(y).view(np.uint8)
            assert np.array_equal(xb, yb), f"{tag}: tensor {k} {name} differs at {np.nonzero(xb != yb)[0][:8]}"


class Lists:
    """A tensor list twice (one copy per entry point), with the same seeded inputs."""

    def __init__(self, al, dev, shapes, w, mspec, vspec):
        self.al, self.shapes, self.w = al, shapes, w
        self.ref = _states(al, dev, shapes, w, mspec, vspec)
        self.new = _states(al, dev, shapes, w, mspec, vspec)
        self.cfg = al.adamw_cfg(grad_bf16=w.grad_bf16, m=mspec, v=vspec)
        self.ws = al.workspace(al.adamw_workspace_bytes(self.ref, self.cfg), dev)

    def step(self, t):
        for sts in (self.ref, self.new):
            for i, (s, st) in enumerate(zip(self.shapes, sts)):
                data.fill_grad(st.grad, i, s, self.w, t)
        self.al.adamw_step(self.ref, self.cfg, t, self.ws)
        self.al.adamw_step_noalloc(self.new, self.cfg, t)


@pytest.mark.parametrize("vc,block", [("AL8", 256), ("AL8", 2048), ("AL16", 128)])
def test_noalloc_matches_workspace_path(dev, vc, block):
    import torch

    import paper_2608_22322_amd as al

    floor = al.log2_floor_of(1e-16)
    mspec = al.Spec(al.UF8, 256)
    vspec = al.Spec(al.AL8 if vc == "AL8" else al.AL16, block, floor)
    big = [Shape("a", 3, 1000), Shape("b", 1, 257), Shape("c", 64, 2048), Shape("d", 1, 1), Shape("e", 17, 256),
           Shape("f", 2048 * 3 + 5, 1), Shape("g", 300, 513)]
    small = [Shape("h", 1, 300), Shape("i", 5, 64)]
    A = Lists(al, dev, big, Workload("big", big, zero_frac=0.05, steps=3), mspec, vspec)
    B = Lists(al, dev, small, Workload("small", small, zero_frac=0.05, steps=3), mspec, vspec)
    log(f"no-alloc AdamW, {vc} B{block}: {len(big)}-tensor list, then {len(small)}-tensor list, then the first again")
    A.step(1)
    B.step(1)  # a smaller list right after a larger one: the fixed table still holds the larger one's tail
    A.step(2)
    B.step(2)
    torch.cuda.synchronize()
    _same(A.ref, A.new, "large list")
    _same(B.ref, B.new, "small list")


def test_noalloc_at_table_limit(dev):
    """4096 small ragged tensors (the fixed table's capacity), then 7 of them."""
    import torch

    import paper_2608_22322_amd as al

    rng = np.random.default_rng(5)
    shapes = [Shape(f"t{i}", 1, int(n)) for i, n in enumerate(rng.integers(1, 700, 4096))]
    mspec, vspec = al.Spec(al.UF8, 256), al.Spec(al.AL8, 256, al.log2_floor_of(1e-16))
    full = Lists(al, dev, shapes, Workload("many", shapes, zero_frac=0.05, steps=2), mspec, vspec)
    few = Lists(al, dev, shapes[:7], Workload("few", shapes[:7], zero_frac=0.05, steps=2), mspec, vspec)
    log(f"no-alloc AdamW at the table limit: {len(shapes)} tensors, {sum(s.n for s in shapes)} elements")
    full.step(1)
    few.step(1)
    full.step(2)
    torch.cuda.synchronize()
    _same(full.ref, full.new, "4096-tensor list")
    _same(few.ref, few.new, "7-tensor list")
