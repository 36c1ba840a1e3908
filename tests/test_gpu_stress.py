"""Stress inputs for the fused steps (the state statistics of section 3.3): gradients whose
magnitudes are log-uniform over tens of binary orders (so block log-ranges reach tens of bits
and cross the log floor), embedding-like tensors with most rows exactly zero, ragged shapes; for
AdamW also gradients large enough to push the second moment past the 2^126 cap. GPU against
the oracle, codes bit-exact up to the near-boundary rule."""
import math

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import synth
from paper_2608_22322_amd.workloads import Shape

from .gpu_util import compare_bits, compare_codes, compare_params, log, require_gpu, to_np

pytestmark = pytest.mark.gpu

SHAPES = [Shape("emb", 300, 256), Shape("w", 37, 130), Shape("n", 1, 1000)]
F = lambda x: float(np.float32(x))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _grad(i, s, t, lo, hi, zero_rows, bf16):
    rng = np.random.default_rng(1000 * i + 17 * t + 3)
    mag = np.exp2(rng.uniform(lo, hi, s.n))
    g = (mag * np.where(rng.random(s.n) < 0.5, -1.0, 1.0)).astype(np.float32)
    if s.rows > 1 and zero_rows:
        rows = np.random.default_rng(99 + i).random(s.rows) < zero_rows  # fixed per tensor
        g.reshape(s.rows, s.cols)[rows, :] = 0.0
    return synth.to_bf16_bits(g) if bf16 else g


def _upload(dev, g):
    import torch

    if g.dtype == np.uint16:
        t = torch.from_numpy(np.concatenate([g, np.zeros(8, np.uint16)]).view(np.int16)).to(dev)
    else:
        t = torch.from_numpy(np.concatenate([g, np.zeros(8, np.float32)])).to(dev)
    return t


def _p0(i, s):
    return synth.normal_f32(synth.param_key(i), s.n, 0.02) if s.rows > 1 else np.ones(s.n, np.float32)


def _cmp(codes, meta, hs, tag):
    if hs.codec == oracle.FP32:
        compare_bits(to_np(codes, hs.n), hs.codes, tag)
        return 0
    g = to_np(codes, hs.codes.shape[0])
    if hs.codec == oracle.UF8:
        g = g.astype(np.int8)
    near = compare_codes(g, hs.codes, hs.y, tag)
    assert np.array_equal(g[: hs.n] == 0, hs.codes[: hs.n] == 0), tag + " zero set"
    compare_bits(to_np(meta, hs.meta.shape[0]), hs.meta, tag + " meta")
    return near


@pytest.mark.parametrize("regime", ["wide", "extreme"])
@pytest.mark.parametrize("vc,block", [("AL8", 64), ("AL8", 256), ("AL8", 2048), ("AL16", 128)])
def test_adamw_stress(dev, regime, vc, block):
    import torch

    import paper_2608_22322_amd as al

    lo, hi = (-60, -1) if regime == "wide" else (-70, 68)
    mspec = al.Spec(al.UF8, 256)
    vspec = al.Spec(getattr(al, vc), block, F(2 * math.log2(1e-8)))
    cfg = al.adamw_cfg(grad_bf16=True, m=mspec, v=vspec)
    states, host = [], []
    for i, s in enumerate(SHAPES):
        p = torch.from_numpy(np.concatenate([_p0(i, s), np.zeros(4, np.float32)])).to(dev)
        m, mm = al.alloc_state(s.n, mspec, dev)
        v, vm = al.alloc_state(s.n, vspec, dev)
        states.append(al.ParamState(p, None, s.rows, s.cols, m=m, m_meta=mm, v=v, v_meta=vm))
        host.append(dict(p=_p0(i, s), m=oracle.State(mspec.codec, s.n, 256),
                         v=oracle.State(vspec.codec, s.n, block, vspec.log_floor)))
    near = 0
    for t in (1, 2, 3):
        gs = [_grad(i, s, t, lo, hi, 0.6, True) for i, s in enumerate(SHAPES)]
        for st, g in zip(states, gs):
            st.grad = _upload(dev, g)
        al.adamw_step(states, cfg, t, al.workspace(al.adamw_workspace_bytes(states, cfg), dev))
        torch.cuda.synchronize()
        for i, (s, h, g, st) in enumerate(zip(SHAPES, host, gs, states)):
            oracle.adamw_step(h["p"], g, h["m"], h["v"], t)
            tag = f"{regime} {vc} B{block} step {t} {s.name}"
            near += _cmp(st.m, st.m_meta, h["m"], tag + " m")
            near += _cmp(st.v, st.v_meta, h["v"], tag + " v")
            compare_params(to_np(st.param, s.n), h["p"], 1e-5 * t, tag + " p")
    if regime == "extreme":
        # the second moment reached the cap region and the floor region
        vmax = max(float(np.max(h["v"].meta[0::2] + h["v"].meta[1::2])) for h in host if h["v"].codec != oracle.FP32)
        vmin = min(float(np.min(h["v"].meta[0::2][h["v"].meta[1::2] > 0])) for h in host)
        log(f"extreme: block log-interval ends span [{vmin:.1f}, {vmax:.1f}]")
        assert vmax >= 100 and vmin <= -53
    log(f"AdamW stress {regime} {vc} B{block}: near-boundary differences {near}")


@pytest.mark.parametrize("came", [False, True])
@pytest.mark.parametrize("vc,block", [("AL8", 256), ("AL16", 128)])
def test_factored_stress(dev, came, vc, block):
    import torch

    import paper_2608_22322_amd as al

    f1, f2 = F(math.log2(1e-30)), F(math.log2(1e-16))
    vspec = al.Spec(getattr(al, vc), block, f1)
    mspec, cspec = al.Spec(al.UF8, 256), al.Spec(getattr(al, vc), block, f2)
    states, host = [], []
    for i, s in enumerate(SHAPES):
        p = torch.from_numpy(np.concatenate([_p0(i, s), np.zeros(4, np.float32)])).to(dev)
        st = al.ParamState(p, None, s.rows, s.cols)
        h = dict(p=_p0(i, s))
        mk = lambda sp, n: oracle.State(sp.codec, n, sp.block, sp.log_floor)
        if s.rows > 1:
            st.vr, st.vr_meta = al.alloc_state(s.rows, vspec, dev)
            st.vc, st.vc_meta = al.alloc_state(s.cols, vspec, dev)
            h.update(vr=mk(vspec, s.rows), vc=mk(vspec, s.cols), v=None)
            if came:
                st.cr, st.cr_meta = al.alloc_state(s.rows, cspec, dev)
                st.cc, st.cc_meta = al.alloc_state(s.cols, cspec, dev)
                h.update(cr=mk(cspec, s.rows), cc=mk(cspec, s.cols))
        else:
            st.v, st.v_meta = al.alloc_state(s.n, vspec, dev)
            h.update(vr=None, vc=None, v=mk(vspec, s.n), cr=None, cc=None)
        if came:
            st.m, st.m_meta = al.alloc_state(s.n, mspec, dev)
            h["m"] = mk(mspec, s.n)
        states.append(st)
        host.append(h)
    cfg = al.came_cfg(m=mspec, v=vspec, conf=cspec) if came else al.adafactor_cfg(v=vspec)
    for i, (s, st) in enumerate(zip(SHAPES, states)):  # gradients are set per step; size the workspace first
        st.grad = _upload(dev, _grad(i, s, 1, -60, -1, 0.6, True))
    nbytes = (al.came_workspace_bytes if came else al.adafactor_workspace_bytes)(states, cfg)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    near = 0
    for t in (1, 2, 3):
        gs = [_grad(i, s, t, -60, -1, 0.6, True) for i, s in enumerate(SHAPES)]
        for st, g in zip(states, gs):
            st.grad = _upload(dev, g)
        (al.came_step if came else al.adafactor_step)(states, cfg, t, ws)
        torch.cuda.synchronize()
        for i, (s, h, g, st) in enumerate(zip(SHAPES, host, gs, states)):
            if came:
                oracle.came_step(h["p"], g, s.rows, s.cols, h["m"], h["vr"], h["vc"], h["v"], h["cr"], h["cc"], t)
            else:
                oracle.adafactor_step(h["p"], g, s.rows, s.cols, h["vr"], h["vc"], h["v"], t)
            tag = f"{'CAME' if came else 'Adafactor'} {vc} B{block} step {t} {s.name}"
            for name in ("m", "v", "vr", "vc", "cr", "cc"):
                if h.get(name) is not None:
                    near += _cmp(getattr(st, name), getattr(st, name + "_meta"), h[name], f"{tag} {name}")
            compare_params(to_np(st.param, s.n), h["p"], 1e-5 * t, tag + " p")
    log(f"factored stress came={came} {vc} B{block}: near-boundary differences {near}")
