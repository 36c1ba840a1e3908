"""GPU parity of the factored optimizer steps (al_adafactor_step, al_came_step)
against the CPU oracle.

* ragged tensor lists (partial 64x64 tiles, odd column counts, 1-D tensors,
  and tensors of whole 256x256 units) over codec / block combinations, bf16
  and fp32 grads, 3 steps;
* 50-step trajectories on TinyLlama-shaped tensors (AL8 B256 Adafactor;
  AL16 B128 + UF8 CAME);
* the full TinyLlama-1.1B list stepped on the GPU in one call, with whole
  small tensors (k/v projections, norms) recomputed by the oracle: the
  factored step couples elements only within a tensor.
"""
import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import data
from paper_2608_22322_amd.workloads import Shape, Workload, llama7b_shapes, tinyllama_shapes

from .gpu_util import compare_bits, compare_codes, compare_params, log, require_gpu, to_np

pytestmark = pytest.mark.gpu

F1 = float(np.float32(math.log2(1e-30)))
F2 = float(np.float32(math.log2(1e-16)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _spec(al, codec, block, floor):
    return al.Spec({"FP32": al.FP32, "AL8": al.AL8, "AL16": al.AL16, "UF8": al.UF8}[codec], block, floor)


class FacPair:
    """A tensor list held on the GPU (library) and on the host (oracle) for Adafactor or CAME."""

    def __init__(self, dev, shapes, w, came, vspec, mspec=None, cspec=None, sample=None, exact=False):
        import torch

        import paper_2608_22322_amd as al

        self.al, self.w, self.shapes, self.came = al, w, shapes, came
        self.vspec, self.mspec, self.cspec = vspec, mspec, cspec
        self.sample = list(range(len(shapes))) if sample is None else sample
        self.states, self.host = [], {}
        for i, s in enumerate(shapes):
            st = al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols)
            if s.rows > 1:
                st.vr, st.vr_meta = al.alloc_state(s.rows, vspec, dev)
                st.vc, st.vc_meta = al.alloc_state(s.cols, vspec, dev)
                if came:
                    st.cr, st.cr_meta = al.alloc_state(s.rows, cspec, dev)
                    st.cc, st.cc_meta = al.alloc_state(s.cols, cspec, dev)
            else:
                st.v, st.v_meta = al.alloc_state(s.n, vspec, dev)
            if came:
                st.m, st.m_meta = al.alloc_state(s.n, mspec, dev)
            self.states.append(st)
        for i in self.sample:
            s = shapes[i]
            h = dict(p=data.host_param(i, s, np.arange(s.n)))
            st = lambda sp, n: oracle.State(sp.codec, n, sp.block, sp.log_floor)
            if s.rows > 1:
                h["vr"], h["vc"], h["v"] = st(vspec, s.rows), st(vspec, s.cols), None
                if came:
                    h["cr"], h["cc"] = st(cspec, s.rows), st(cspec, s.cols)
            else:
                h["vr"], h["vc"], h["v"] = None, None, st(vspec, s.n)
                h["cr"], h["cc"] = None, None
            if came:
                h["m"] = st(mspec, s.n)
            self.host[i] = h
        if came:
            self.cfg = al.came_cfg(grad_bf16=w.grad_bf16, m=mspec, v=vspec, conf=cspec, exact_sums=exact)
            nbytes = al.came_workspace_bytes(self.states, self.cfg)
        else:
            self.cfg = al.adafactor_cfg(grad_bf16=w.grad_bf16, v=vspec, exact_sums=exact)
            nbytes = al.adafactor_workspace_bytes(self.states, self.cfg)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        self.arr = al.tensor_array(self.states)

    def step(self, t):
        import torch

        for i, (s, st) in enumerate(zip(self.shapes, self.states)):
            data.fill_grad(st.grad, i, s, self.w, t)
        if self.came:
            self.al.came_step(self.states, self.cfg, t, self.ws, arr=self.arr)
        else:
            self.al.adafactor_step(self.states, self.cfg, t, self.ws, arr=self.arr)

        def host_step(i):
            s, h = self.shapes[i], self.host[i]
            g = data.host_grad(i, self.w, t, np.arange(s.n))
            if self.came:
                oracle.came_step(h["p"], g, s.rows, s.cols, h["m"], h["vr"], h["vc"], h["v"], h["cr"], h["cc"], t)
            else:
                oracle.adafactor_step(h["p"], g, s.rows, s.cols, h["vr"], h["vc"], h["v"], t)

        # the sampled tensors are independent: their oracle steps run side by side (the C oracle releases
        # the interpreter lock), largest first
        order = sorted(self.sample, key=lambda i: -self.shapes[i].n)
        with ThreadPoolExecutor(min(8, max(1, len(order)))) as ex:
            list(ex.map(host_step, order))
        torch.cuda.synchronize()

    def compare(self, t, rtol):
        near = 0
        for i in self.sample:
            s, h, st = self.shapes[i], self.host[i], self.states[i]
            tag = f"step {t} tensor {i} {s.name} [{s.rows}x{s.cols}]"
            slots = [("vr", st.vr, st.vr_meta), ("vc", st.vc, st.vc_meta), ("v", st.v, st.v_meta)]
            if self.came:
                slots += [("cr", st.cr, st.cr_meta), ("cc", st.cc, st.cc_meta), ("m", st.m, st.m_meta)]
            for name, codes, meta in slots:
                hs = h.get(name)
                if hs is None:
                    continue
                near += _cmp_state(codes, meta, hs, f"{tag} {name}")
            compare_params(to_np(st.param, s.n), h["p"], rtol, tag + " p")
        return near


def _cmp_state(codes, meta, hs, tag):
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


# ragged shapes (partial units, odd widths, 1-D) and two tensors of whole 256x256 units (w, x: the
# streaming kernels), so every codec combination and both gradient types cover both kernel families
RAGGED = [Shape("a", 5, 7), Shape("b", 64, 256), Shape("w", 256, 512), Shape("c", 130, 513), Shape("d", 300, 66),
          Shape("e", 2, 1030), Shape("f", 1, 1), Shape("x", 512, 256), Shape("g", 1, 777), Shape("h", 257, 3),
          Shape("i", 1, 2048)]


@pytest.mark.parametrize("grad_bf16", [True, False])
@pytest.mark.parametrize("vc,block", [("AL8", 256), ("AL8", 64), ("AL8", 2048), ("AL16", 128), ("FP32", 256)])
def test_adafactor_ragged_lists(dev, grad_bf16, vc, block):
    import paper_2608_22322_amd as al

    w = Workload("ragged", RAGGED, grad_bf16=grad_bf16, zero_frac=0.05, steps=3)
    pair = FacPair(dev, RAGGED, w, False, _spec(al, vc, block, F1))
    for t in (1, 2, 3):
        pair.step(t)
        pair.compare(t, 1e-5 * t)


@pytest.mark.parametrize("grad_bf16", [True, False])
@pytest.mark.parametrize("mc,vc,vb,cc,cb", [("UF8", "AL16", 128, "AL16", 128), ("UF8", "AL8", 2048, "AL8", 2048),
                                            ("UF8", "AL8", 256, "FP32", 256), ("FP32", "FP32", 256, "FP32", 256),
                                            ("UF8", "AL16", 64, "AL8", 512)])
def test_came_ragged_lists(dev, grad_bf16, mc, vc, vb, cc, cb):
    import paper_2608_22322_amd as al

    w = Workload("ragged", RAGGED, grad_bf16=grad_bf16, zero_frac=0.05, steps=3)
    pair = FacPair(dev, RAGGED, w, True, _spec(al, vc, vb, F1), mspec=_spec(al, mc, 256, 0.0),
                   cspec=_spec(al, cc, cb, F2))
    for t in (1, 2, 3):
        pair.step(t)
        pair.compare(t, 1e-5 * t)


# a q projection (8 x 8 whole units: column sums merged over unit rows), a k projection (one unit row), a
# norm (1-D) and a ragged slab (the per-unit kernels)
TL_SUBSET = [Shape("q", 2048, 2048), Shape("k", 256, 2048), Shape("attn_norm", 1, 2048),
             Shape("down_slab", 96, 5632)]


def test_adafactor_100_steps(dev):
    """Independent 100-step trajectories (the TinyLlama Adafactor configuration's length) on a
    subset of its shapes, a full q projection among them: states and parameters compared along the way."""
    import paper_2608_22322_amd as al

    w = Workload("tl-subset", TL_SUBSET, zero_frac=0.0, steps=100)
    pair = FacPair(dev, TL_SUBSET, w, False, _spec(al, "AL8", 256, F1))
    near = 0
    for t in range(1, 101):
        pair.step(t)
        if t in (1, 2, 10, 25, 50, 75, 100):
            near += pair.compare(t, 1e-5 if t == 1 else 1e-4)
    log(f"Adafactor 100 steps: near-boundary code differences {near}")


def test_came_100_steps(dev):
    """As test_adafactor_100_steps, for the TinyLlama CAME configuration."""
    import paper_2608_22322_amd as al

    w = Workload("tl-subset", TL_SUBSET, zero_frac=0.02, steps=100)
    pair = FacPair(dev, TL_SUBSET, w, True, _spec(al, "AL16", 128, F1), mspec=_spec(al, "UF8", 256, 0.0),
                   cspec=_spec(al, "AL16", 128, F2))
    near = 0
    for t in range(1, 101):
        pair.step(t)
        if t in (1, 2, 10, 25, 50, 75, 100):
            near += pair.compare(t, 1e-5 if t == 1 else 1e-4)
    log(f"CAME 100 steps: near-boundary code differences {near}")


@pytest.mark.parametrize("came", [False, True])
def test_full_tinyllama_list_sampled(dev, came):
    """The whole 201-tensor TinyLlama list in one call; whole small tensors recomputed by the oracle."""
    import torch

    import paper_2608_22322_amd as al

    shapes = tinyllama_shapes()
    w = Workload("tinyllama", shapes, zero_frac=0.02 if came else 0.0, steps=2)
    sample = [i for i, s in enumerate(shapes) if s.name in ("embed", "layer0.k", "layer0.attn_norm", "layer3.gate",
                                                             "layer7.v", "layer12.down", "layer21.mlp_norm",
                                                             "norm")]
    if came:
        pair = FacPair(dev, shapes, w, True, _spec(al, "AL16", 128, F1), mspec=_spec(al, "UF8", 256, 0.0),
                       cspec=_spec(al, "AL16", 128, F2), sample=sample)
    else:
        pair = FacPair(dev, shapes, w, False, _spec(al, "AL8", 256, F1), sample=sample)
    log(f"TinyLlama full list, {'CAME' if came else 'Adafactor'}, sampled tensors {sample}")
    for t in (1, 2):
        pair.step(t)
        pair.compare(t, 1e-5 * t)
    del pair
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("came", [False, True])
def test_full_llama7b_list_sampled(dev, came):
    """The whole 291-tensor Llama-7B list in one call, in the configuration the benchmark times (Adafactor:
    AL8 B256, no zero mask; CAME: AL16 B128 factors and confidence, UF8 momentum, 2% zeros); the LM head
    [32000 x 4096] (125 row units in the finalize merge), an FFN up projection [11008 x 4096], a down
    projection [4096 x 11008] and two norms recomputed whole by the oracle, 2 steps."""
    import torch

    import paper_2608_22322_amd as al

    shapes = llama7b_shapes()
    w = Workload("llama-7b", shapes, zero_frac=0.02 if came else 0.0, steps=2)
    sample = [i for i, s in enumerate(shapes) if s.name in ("layer0.attn_norm", "layer17.down", "layer31.up",
                                                             "norm", "lm_head")]
    assert len(sample) == 5
    if came:
        pair = FacPair(dev, shapes, w, True, _spec(al, "AL16", 128, F1), mspec=_spec(al, "UF8", 256, 0.0),
                       cspec=_spec(al, "AL16", 128, F2), sample=sample)
    else:
        pair = FacPair(dev, shapes, w, False, _spec(al, "AL8", 256, F1), sample=sample)
    log(f"Llama-7B full list, {'CAME' if came else 'Adafactor'}, sampled tensors "
        f"{[(shapes[i].name, shapes[i].rows, shapes[i].cols) for i in sample]}")
    near = 0
    for t in (1, 2):
        pair.step(t)
        near += pair.compare(t, 1e-5 * t)
        log(f"step {t} compared")
    log(f"near-boundary code differences: {near}")
    del pair
    torch.cuda.empty_cache()


@pytest.mark.parametrize("came", [False, True])
def test_exact_sums_flag_gives_identical_states(dev, came):
    """The marginal kernels' fast sums are kept only where they provably round like the exact ones. Stepping
    the same list with AL_FLAG_EXACT_SUMS (every row and column mean summed again exactly in the finalize
    step) must give the same codes, metadata and parameters bit for bit, and both match the oracle:
    TinyLlama-shaped tensors and ragged ones, 6 steps."""
    import torch

    import paper_2608_22322_amd as al

    shapes = [Shape("k", 256, 2048), Shape("norm", 1, 2048), Shape("slab", 300, 513), Shape("tall", 1030, 64)]
    w = Workload("exact-vs-fast", shapes, zero_frac=0.02, steps=6)
    if came:
        kw = dict(vspec=_spec(al, "AL16", 128, F1), mspec=_spec(al, "UF8", 256, 0.0), cspec=_spec(al, "AL16", 128, F2))
    else:
        kw = dict(vspec=_spec(al, "AL8", 256, F1))
    fast = FacPair(dev, shapes, w, came, **kw)
    exact = FacPair(dev, shapes, w, came, exact=True, sample=[], **kw)
    for t in range(1, 7):
        fast.step(t)
        exact.step(t)
        fast.compare(t, 1e-5 if t == 1 else 1e-4)
        for i, (a, b) in enumerate(zip(fast.states, exact.states)):
            for name in ("param", "m", "m_meta", "v", "v_meta", "vr", "vr_meta", "vc", "vc_meta", "cr", "cr_meta",
                         "cc", "cc_meta"):
                x, y = getattr(a, name), getattr(b, name)
                if x is None:
                    continue
                assert torch.equal(x, y), f"step {t} tensor {i} {name}: exact-sums path differs"
    log(f"{'CAME' if came else 'Adafactor'}: fast and exact-sum paths identical over 6 steps")
