"""GPU parity of grouped steps (G0 / G1 policies, section 6): one library call per group,
protected tensors (1-D, norms, embedding, LM head) with FP32 states, checked tensor by tensor
against the oracle with each group's codes."""
import math

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import data
from paper_2608_22322_amd.workloads import Shape, Workload

from .gpu_util import compare_bits, compare_codes, compare_params, require_gpu, to_np

pytestmark = pytest.mark.gpu

SHAPES = [Shape("embed", 96, 256), Shape("layer0.q", 128, 256), Shape("layer0.attn_norm", 1, 256),
          Shape("layer0.down", 64, 384), Shape("norm", 1, 256), Shape("lm_head", 80, 256)]
F_EPS1 = float(np.float32(math.log2(1e-30)))
F_EPS2 = float(np.float32(math.log2(1e-16)))
F_V = float(np.float32(2 * math.log2(1e-8)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _cmp(codes, meta, hs, tag):
    if hs.codec == oracle.FP32:
        compare_bits(to_np(codes, hs.n), hs.codes, tag)
        return
    g = to_np(codes, hs.codes.shape[0])
    if hs.codec == oracle.UF8:
        g = g.astype(np.int8)
    compare_codes(g, hs.codes, hs.y, tag)
    compare_bits(to_np(meta, hs.meta.shape[0]), hs.meta, tag + " meta")


@pytest.mark.parametrize("kind", ["adamw", "adafactor", "came"])
@pytest.mark.parametrize("policy", ["G0", "G1"])
def test_grouped_step(dev, kind, policy):
    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import grouping

    w = Workload("grouped", SHAPES, grad_bf16=True, zero_frac=0.02, steps=3)
    prot = grouping.protected_flags(SHAPES, policy)
    if kind == "adamw":
        specs = {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL8, 256, F_V)}
        cfg = al.adamw_cfg(m=specs["m"], v=specs["v"])
    elif kind == "adafactor":
        specs = {"v": al.Spec(al.AL8, 256, F_EPS1)}
        cfg = al.adafactor_cfg(v=specs["v"])
    else:
        specs = {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL16, 128, F_EPS1), "conf": al.Spec(al.AL16, 128, F_EPS2)}
        cfg = al.came_cfg(m=specs["m"], v=specs["v"], conf=specs["conf"])
    states = [al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
              for i, s in enumerate(SHAPES)]
    grouping.attach_states(states, kind, specs, prot, dev)
    step = grouping.GroupedStep(kind, states, cfg, prot, dev)
    host = []
    for i, (s, p) in enumerate(zip(SHAPES, prot)):
        sp = {r: (grouping.fp32_spec(v) if p else v) for r, v in specs.items()}
        st = lambda r, n: oracle.State(sp[r].codec, n, sp[r].block, sp[r].log_floor)
        h = dict(p=data.host_param(i, s, np.arange(s.n)))
        if kind == "adamw":
            h.update(m=st("m", s.n), v=st("v", s.n))
        elif s.rows > 1:
            h.update(vr=st("v", s.rows), vc=st("v", s.cols), v=None)
            if kind == "came":
                h.update(cr=st("conf", s.rows), cc=st("conf", s.cols))
        else:
            h.update(vr=None, vc=None, v=st("v", s.n), cr=None, cc=None)
        if kind == "came":
            h["m"] = st("m", s.n)
        host.append(h)
    import torch

    for t in (1, 2, 3):
        for i, (s, st) in enumerate(zip(SHAPES, states)):
            data.fill_grad(st.grad, i, s, w, t)
        step.step(t)
        for i, (s, h) in enumerate(zip(SHAPES, host)):
            g = data.host_grad(i, w, t, np.arange(s.n))
            if kind == "adamw":
                oracle.adamw_step(h["p"], g, h["m"], h["v"], t)
            elif kind == "adafactor":
                oracle.adafactor_step(h["p"], g, s.rows, s.cols, h["vr"], h["vc"], h["v"], t)
            else:
                oracle.came_step(h["p"], g, s.rows, s.cols, h["m"], h["vr"], h["vc"], h["v"], h["cr"], h["cc"], t)
        torch.cuda.synchronize()
        for i, (s, h, st, p) in enumerate(zip(SHAPES, host, states, prot)):
            tag = f"{kind} {policy} step {t} {s.name}"
            compare_params(to_np(st.param, s.n), h["p"], 1e-5 * t, tag)
            for name in ("m", "v", "vr", "vc", "cr", "cc"):
                hs = h.get(name)
                if hs is None:
                    continue
                if p:
                    assert hs.codec == oracle.FP32, tag
                _cmp(getattr(st, name), getattr(st, name + "_meta"), hs, f"{tag} {name}")
