"""Bounds and determinism of every entry point on the GPU.

Bounds: every buffer a call touches -- parameters, gradients, padded code arrays and their block
metadata, factored vectors, APOLLO's projection and limiter slot, and the workspace at exactly its
queried size -- is allocated with 256 guard bytes of a fixed pattern behind it; after the calls
the guards must be unchanged, and the padding codes of a partial last block must be zero. (A
write past a buffer lands in its own guard, inside the allocation.)

Determinism: the same calls on fresh copies of the same inputs give bit-identical parameters,
codes and metadata (sums are merged in a fixed order; no atomics decide a value).
"""
import math

import numpy as np
import pytest

from paper_2608_22322_amd import synth

from .gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

GUARD = 256
PATTERN = 0xA5
V_FLOOR = float(np.float32(2 * math.log2(1e-8)))
F1 = float(np.float32(math.log2(1e-30)))
F2 = float(np.float32(math.log2(1e-16)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


class Arena:
    """Device buffers each followed by a guard region."""

    def __init__(self, dev):
        self.dev, self.bufs = dev, []

    def alloc(self, nbytes: int, dtype, fill=None):
        import torch

        nbytes = max(int(nbytes), 16)
        nbytes = (nbytes + 15) // 16 * 16
        raw = torch.full((nbytes + GUARD,), PATTERN, dtype=torch.uint8, device=self.dev)
        view = raw[:nbytes].view(dtype)
        if fill is None:
            view.zero_()
        else:
            src = torch.from_numpy(np.ascontiguousarray(fill)).to(self.dev).view(-1).view(dtype)
            view[: src.numel()].copy_(src)
            view[src.numel():].zero_()
        self.bufs.append((raw, nbytes))
        return view

    def check(self, what: str) -> None:
        for k, (raw, nbytes) in enumerate(self.bufs):
            g = raw[nbytes:].cpu().numpy()
            assert np.all(g == PATTERN), f"{what}: buffer {k} guard overwritten at {np.nonzero(g != PATTERN)[0][:8]}"


def _state(ar, al, n, spec):
    import torch

    if spec.codec == al.FP32:
        return ar.alloc(4 * n, torch.float32), None
    dt = {al.AL8: torch.uint8, al.AL16: torch.int16, al.UF8: torch.int8}[spec.codec]
    codes = ar.alloc(al.code_bytes(spec.codec, n, spec.block), dt)
    meta = ar.alloc(4 * al.meta_floats(spec.codec, n, spec.block), torch.float32)
    return codes, meta


def _pad_zero(al, codes, n, spec, what):
    if spec.codec == al.FP32:
        return
    elem = 2 if spec.codec == al.AL16 else 1
    total = al.code_bytes(spec.codec, n, spec.block) // elem
    tail = codes[n:total].cpu().numpy()
    assert np.all(tail == 0), f"{what}: padding codes not zero"


def _grad(ar, i, t, n, bf16):
    import torch

    g = synth.normal_f32(synth.grad_key(i, t), n, 1e-3, synth.mask_key(i), 0.02)
    if bf16:
        return ar.alloc(2 * n, torch.int16, synth.to_bf16_bits(g).view(np.int16))
    return ar.alloc(4 * n, torch.float32, g)


def _snapshot(bufs):
    return [b.detach().cpu().numpy().copy() for b in bufs if b is not None]


def _adamw_run(dev, shapes, bv, bf16):
    import torch

    import paper_2608_22322_amd as al

    ar = Arena(dev)
    ms, vs = al.Spec(al.UF8, 256), al.Spec(al.AL8, bv, V_FLOOR)
    states = []
    for i, n in enumerate(shapes):
        p = ar.alloc(4 * n, torch.float32, synth.normal_f32(synth.param_key(i), n, 0.02))
        m, mm = _state(ar, al, n, ms)
        v, vm = _state(ar, al, n, vs)
        states.append(al.ParamState(p, None, 1, n, m=m, m_meta=mm, v=v, v_meta=vm))
    cfg = al.adamw_cfg(m=ms, v=vs, grad_bf16=bf16)
    for t in (1, 2):
        for i, (st, n) in enumerate(zip(states, shapes)):
            st.grad = _grad(ar, i, t, n, bf16)
        ws = ar.alloc(al.adamw_workspace_bytes(states, cfg), torch.uint8)
        al.adamw_step(states, cfg, t, ws)
    torch.cuda.synchronize()
    ar.check(f"adamw B_V {bv}")
    for st, n in zip(states, shapes):
        _pad_zero(al, st.m, n, ms, "adamw m")
        _pad_zero(al, st.v, n, vs, "adamw v")
    return _snapshot([x for st in states for x in (st.param, st.m, st.m_meta, st.v, st.v_meta)])


@pytest.mark.parametrize("bv", [64, 128, 256, 512, 1024, 2048])
@pytest.mark.parametrize("bf16", [True, False])
def test_adamw_bounds_and_determinism(dev, bv, bf16):
    shapes = [33, 1000, 2049, 70_001, 3 * 2048]
    a = _adamw_run(dev, shapes, bv, bf16)
    b = _adamw_run(dev, shapes, bv, bf16)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    log(f"adamw B_V {bv} bf16 {bf16}: guards intact, runs identical")


def _factored_run(dev, came, shapes, bf16):
    import torch

    import paper_2608_22322_amd as al

    ar = Arena(dev)
    if came:
        vs, ms, cs = al.Spec(al.AL16, 128, F1), al.Spec(al.UF8, 256), al.Spec(al.AL16, 128, F2)
        cfg = al.came_cfg(m=ms, v=vs, conf=cs, grad_bf16=bf16)
    else:
        vs = al.Spec(al.AL8, 256, F1)
        cfg = al.adafactor_cfg(v=vs, grad_bf16=bf16)
    states = []
    for i, (rows, cols) in enumerate(shapes):
        n = rows * cols
        st = al.ParamState(ar.alloc(4 * n, torch.float32, synth.normal_f32(synth.param_key(i), n, 0.02)), None,
                           rows, cols)
        if rows > 1:
            st.vr, st.vr_meta = _state(ar, al, rows, vs)
            st.vc, st.vc_meta = _state(ar, al, cols, vs)
            if came:
                st.cr, st.cr_meta = _state(ar, al, rows, cs)
                st.cc, st.cc_meta = _state(ar, al, cols, cs)
        else:
            st.v, st.v_meta = _state(ar, al, n, vs)
        if came:
            st.m, st.m_meta = _state(ar, al, n, ms)
        states.append(st)
    for t in (1, 2):
        for i, (st, (rows, cols)) in enumerate(zip(states, shapes)):
            st.grad = _grad(ar, i, t, rows * cols, bf16)
        arr = al.tensor_array(states)
        nbytes = (al.came_workspace_bytes if came else al.adafactor_workspace_bytes)(states, cfg, arr=arr)
        ws = ar.alloc(nbytes, torch.uint8)
        (al.came_step if came else al.adafactor_step)(states, cfg, t, ws, arr=arr)
    torch.cuda.synchronize()
    ar.check("came" if came else "adafactor")
    roles = ("m", "v", "vr", "vc", "cr", "cc")
    return _snapshot([st.param for st in states] + [getattr(st, r) for st in states for r in roles] +
                     [getattr(st, r + "_meta") for st in states for r in roles])


@pytest.mark.parametrize("bf16", [True, False])
@pytest.mark.parametrize("came", [False, True])
def test_factored_bounds_and_determinism(dev, came, bf16):
    shapes = [(300, 257), (37, 130), (256, 512), (1, 700), (513, 64), (512, 256)]
    a = _factored_run(dev, came, shapes, bf16)
    b = _factored_run(dev, came, shapes, bf16)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    log(f"{'came' if came else 'adafactor'}: guards intact, runs identical")


def _apollo_run(dev, shapes, rank):
    import torch

    import paper_2608_22322_amd as al
    from oracle import apollo as oap

    ar = Arena(dev)
    ms, vs = al.Spec(al.UF8, 256), al.Spec(al.AL8, 2048, V_FLOOR)
    cfg = al.apollo_cfg(rank=rank, m=ms, v=vs)
    items = []
    for i, (rows, cols) in enumerate(shapes):
        right, C, L = oap.layout(rows, cols)
        n = rows * cols
        p = ar.alloc(4 * n, torch.float32, synth.normal_f32(synth.param_key(i), n, 0.02))
        pj = ar.alloc(4 * L * rank, torch.float32, synth.proj_matrix(i, 0, L, rank))
        m, mm = _state(ar, al, C * rank, ms)
        v, vm = _state(ar, al, C * rank, vs)
        ns = ar.alloc(4, torch.float32)
        items.append([p, None, rows, cols, pj, m, mm, v, vm, ns])
    for t in (1, 2):
        for i, it in enumerate(items):
            it[1] = _grad(ar, i, t, it[2] * it[3], True)
        arr = al.apollo_tensor_array([tuple(it) for it in items])
        ws = ar.alloc(al.apollo_workspace_bytes(arr, len(items), cfg), torch.uint8)
        al.apollo_step(arr, len(items), cfg, t, ws)
    torch.cuda.synchronize()
    ar.check("apollo")
    return _snapshot([x for it in items for x in (it[0], it[5], it[6], it[7], it[8], it[9])])


def test_apollo_bounds_and_determinism(dev):
    shapes = [(70, 33), (40, 300), (256, 512), (129, 64), (5, 700), (512, 256)]
    a = _apollo_run(dev, shapes, 64)
    b = _apollo_run(dev, shapes, 64)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    log("apollo: guards intact, runs identical")


@pytest.mark.parametrize("codec,block", [("AL8", 64), ("AL16", 2048), ("UF8", 256)])
def test_codec_bounds(dev, codec, block):
    import torch

    import paper_2608_22322_amd as al

    c = getattr(al, codec)
    ar = Arena(dev)
    for n in (1, 63, 1000, 5000 + 17):
        x = synth.normal_f32(synth.grad_key(9, n), n, 1e-3)
        if c != al.UF8:
            x = np.abs(x)
        xd = ar.alloc(4 * n, torch.float32, x)
        spec = al.Spec(c, block, V_FLOOR)
        codes, meta = _state(ar, al, n, spec)
        al.quantize(c, xd[:n], block, V_FLOOR, codes, meta)
        out = ar.alloc(4 * n, torch.float32)
        al.dequantize(c, codes, meta, n, block, out)
        torch.cuda.synchronize()
        _pad_zero(al, codes, n, spec, f"{codec} n={n}")
    ar.check(f"{codec} B{block}")
