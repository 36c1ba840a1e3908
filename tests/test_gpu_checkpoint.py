"""Resumption through a checkpoint and state-precision migration on the GPU (section 7.1):
a run saved after step 2 and resumed from the file equals the uninterrupted run bit for bit;
migrating AL8 -> AL16 (and back) gives exactly the oracle's re-encoding of the decoded values."""
import math
import os

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import data, synth
from paper_2608_22322_amd.workloads import Shape, Workload

from .gpu_util import compare_bits, compare_codes, require_gpu, to_np

pytestmark = pytest.mark.gpu

SHAPES = [Shape("a", 64, 256), Shape("b", 1, 700), Shape("c", 37, 130)]


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _make(dev, kind, w):
    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import grouping

    if kind == "adamw":
        specs = {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL8, 256, float(np.float32(2 * math.log2(1e-8))))}
        cfg = al.adamw_cfg(m=specs["m"], v=specs["v"])
    else:
        specs = {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL16, 128, float(np.float32(math.log2(1e-30)))),
                 "conf": al.Spec(al.AL16, 128, float(np.float32(math.log2(1e-16))))}
        cfg = al.came_cfg(m=specs["m"], v=specs["v"], conf=specs["conf"])
    states = [al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
              for i, s in enumerate(SHAPES)]
    grouping.attach_states(states, kind, specs, [False] * len(SHAPES), dev)
    step = grouping.GroupedStep(kind, states, cfg, [False] * len(SHAPES), dev)
    return states, step, specs


def _role_specs(st, specs):
    out = {}
    for role in ("m", "v", "vr", "vc", "cr", "cc"):
        if getattr(st, role) is not None:
            out[role] = specs["conf"] if role in ("cr", "cc") else specs["m" if role == "m" else "v"]
    return out


@pytest.mark.parametrize("kind", ["adamw", "came"])
def test_resume_from_checkpoint_is_exact(dev, kind, tmp_path):
    import torch

    from paper_2608_22322_amd import checkpoint, grouping

    w = Workload("ckpt", SHAPES, zero_frac=0.02, steps=4)
    full, step_full, specs = _make(dev, kind, w)
    part, step_part, _ = _make(dev, kind, w)
    for t in (1, 2, 3, 4):
        for i, (s, st) in enumerate(zip(SHAPES, full)):
            data.fill_grad(st.grad, i, s, w, t)
        step_full.step(t)
    for t in (1, 2):
        for i, (s, st) in enumerate(zip(SHAPES, part)):
            data.fill_grad(st.grad, i, s, w, t)
        step_part.step(t)
    torch.cuda.synchronize()
    path = os.path.join(tmp_path, "opt.safetensors")
    checkpoint.save(path, part, [_role_specs(st, specs) for st in part], [s.name for s in SHAPES], kind, 2)
    params = [st.param.clone() for st in part]
    # fresh buffers and a stepper built over them before the load: the load overwrites them in place
    resumed, step_res, _ = _make(dev, kind, w)
    for st, p in zip(resumed, params):
        st.param.copy_(p)
    assert checkpoint.load(path, resumed, [_role_specs(st, specs) for st in resumed], kind=kind) == (kind, 2)
    for t in (3, 4):
        for i, (s, st) in enumerate(zip(SHAPES, resumed)):
            data.fill_grad(st.grad, i, s, w, t)
        step_res.step(t)
    torch.cuda.synchronize()
    for s, a, b in zip(SHAPES, full, resumed):
        assert torch.equal(a.param[:s.n], b.param[:s.n]), s.name
        for role in ("m", "v", "vr", "vc", "cr", "cc"):
            x, y = getattr(a, role), getattr(b, role)
            assert (x is None) == (y is None)
            if x is not None:
                assert torch.equal(x, y), (s.name, role)
                assert torch.equal(getattr(a, role + "_meta"), getattr(b, role + "_meta")), (s.name, role)


@pytest.mark.parametrize("src,dst", [("AL8", "AL16"), ("AL16", "AL8")])
def test_migration_matches_oracle(dev, src, dst):
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import checkpoint

    bits = {"AL8": 8, "AL16": 16}
    n, B = 5 * 256 + 77, 256
    x = np.abs(synth.normal_f32(synth.grad_key(5, 1), n, 1e-6)).astype(np.float32)
    x[::13] = 0.0
    lf = float(np.float32(-53.15))
    old, new = al.Spec(getattr(al, src), B, lf), al.Spec(getattr(al, dst), B, lf)
    codes, meta = al.alloc_state(n, old, dev)
    xd = torch.from_numpy(np.concatenate([x, np.zeros(4, np.float32)])).to(dev)
    al.quantize(old.codec, xd[:n], B, lf, codes, meta)
    st = al.ParamState(None, None, 1, n, v=codes, v_meta=meta)
    checkpoint.migrate(st, "v", old, new)
    torch.cuda.synchronize()
    o_codes, o_meta, _ = oracle.al_quantize(bits[src], x, B, lf)
    dec = oracle.al_dequantize(bits[src], o_codes, o_meta, n, B)
    w_codes, w_meta, y = oracle.al_quantize(bits[dst], dec, B, lf)
    compare_codes(to_np(st.v, w_codes.shape[0]), w_codes, y, f"{src}->{dst}")
    compare_bits(to_np(st.v_meta, w_meta.shape[0]), w_meta, f"{src}->{dst} meta")
    assert np.array_equal(to_np(st.v, n) == 0, x == 0)  # exact zeros survive the migration


def test_apollo_resume_from_checkpoint_is_exact(dev, tmp_path):
    """APOLLO: a run saved after step 2 and resumed (fresh ApolloStep, saved params) equals the
    uninterrupted run bit for bit at step 5, across a projection refresh (gap 2)."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import apollo, checkpoint

    shapes = [Shape("embed", 64, 40), Shape("layer0.q", 48, 48), Shape("layer0.down", 40, 96),
              Shape("layer0.attn_norm", 1, 48)]
    names = [s.name for s in shapes]
    w = Workload("ckpt-apollo", shapes, zero_frac=0.02, steps=5)

    def make():
        sts = [al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
               for i, s in enumerate(shapes)]
        return sts, apollo.ApolloStep(sts, names, al.apollo_cfg(rank=64), gap=2, device=dev)

    def run(sts, drv, steps):
        for t in steps:
            for i, (s, st) in enumerate(zip(shapes, sts)):
                data.fill_grad(st.grad, i, s, w, t)
            drv.step(t)

    full, dfull = make()
    run(full, dfull, range(1, 6))
    part, dpart = make()
    run(part, dpart, (1, 2))
    torch.cuda.synchronize()
    path = os.path.join(tmp_path, "apollo.safetensors")
    checkpoint.save_apollo(path, dpart, names, 2)
    params = [st.param.clone() for st in part]
    res, dres = make()
    for st, p in zip(res, params):
        st.param.copy_(p)
    assert checkpoint.load_apollo(path, dres, names) == 2
    run(res, dres, (3, 4, 5))
    torch.cuda.synchronize()
    for s, a, b in zip(shapes, full, res):
        assert torch.equal(a.param[:s.n], b.param[:s.n]), s.name
    for x, y in zip(dfull.items, dres.items):
        for k in (5, 6, 7, 8, 9):
            assert torch.equal(x[k], y[k])
    for x, y in zip(dfull.full_states, dres.full_states):
        assert torch.equal(x.m, y.m) and torch.equal(x.v, y.v) and torch.equal(x.v_meta, y.v_meta)
    with pytest.raises(ValueError):
        checkpoint.load_apollo(path, dres, ["x"] + names[1:])
