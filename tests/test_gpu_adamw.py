"""GPU parity of the fused AdamW step (al_adamw_step) against the CPU oracle.

* ragged multi-tensor lists (1 .. 3 tiles, partial blocks) over every codec
  combination and block size, 3 steps;
* the 1024x1024 workload (fp32 grads, 5% dormant entries held at zero for five
  steps), 10 steps, compared at every step;
* 100-step trajectories on TinyLlama-shaped tensors (bf16 grads, 2% zeros);
* full-size TinyLlama-1.1B and Llama-7B lists in the launch configuration the
  benchmark times, checked on sampled tiles that the oracle recomputes.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import data, synth
from paper_2608_22322_amd.workloads import Shape, Workload, llama7b_shapes, tinyllama_shapes, workload_1024

from .gpu_util import compare_bits, compare_codes, compare_params, log, require_gpu, to_np

pytestmark = pytest.mark.gpu

V_FLOOR = float(np.float32(2 * math.log2(1e-8)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


class Pair:
    """A tensor list held both on the GPU (library path) and on the host (oracle)."""

    def __init__(self, dev, shapes, w: Workload, mspec, vspec):
        import paper_2608_22322_amd as al

        self.al, self.w, self.shapes = al, w, shapes
        self.mspec, self.vspec = mspec, vspec
        self.states, self.hp, self.hm, self.hv, self.grads = [], [], [], [], []
        for i, s in enumerate(shapes):
            p = data.device_param(i, s, dev)
            g = data.device_grad_buffer(s, w, dev)
            m, mm = al.alloc_state(s.n, mspec, dev)
            v, vm = al.alloc_state(s.n, vspec, dev)
            self.states.append(al.ParamState(p, g, s.rows, s.cols, m=m, m_meta=mm, v=v, v_meta=vm))
            self.hp.append(data.host_param(i, s, np.arange(s.n)))
            self.hm.append(oracle.State(mspec.codec, s.n, mspec.block, mspec.log_floor))
            self.hv.append(oracle.State(vspec.codec, s.n, vspec.block, vspec.log_floor))
        self.cfg = al.adamw_cfg(grad_bf16=w.grad_bf16, m=mspec, v=vspec)
        self.arr = al.tensor_array(self.states)
        self.ws = al.workspace(al.adamw_workspace_bytes(self.states, self.cfg, arr=self.arr), dev)

    def step(self, t):
        import torch

        for i, (s, st) in enumerate(zip(self.shapes, self.states)):
            data.fill_grad(st.grad, i, s, self.w, t)
        self.al.adamw_step(self.states, self.cfg, t, self.ws, arr=self.arr)
        for i, s in enumerate(self.shapes):
            g = data.host_grad(i, self.w, t, np.arange(s.n))
            oracle.adamw_step(self.hp[i], g, self.hm[i], self.hv[i], t)
        torch.cuda.synchronize()

    def compare(self, t, rtol):
        near = 0
        for i, (s, st) in enumerate(zip(self.shapes, self.states)):
            tag = f"step {t} tensor {i} {s.name} n{s.n}"
            near += self._cmp_state(st.m, st.m_meta, self.hm[i], tag + " m")
            near += self._cmp_state(st.v, st.v_meta, self.hv[i], tag + " v")
            compare_params(to_np(st.param, s.n), self.hp[i], rtol, tag + " p")
        return near

    def _cmp_state(self, codes, meta, hs, tag):
        if hs.codec == oracle.FP32:
            compare_bits(to_np(codes, hs.n), hs.codes, tag)
            return 0
        nc = hs.codes.shape[0]
        g = to_np(codes, nc)
        if hs.codec == oracle.UF8:
            g = g.astype(np.int8)
        near = compare_codes(g, hs.codes, hs.y, tag)
        assert np.array_equal(g[: hs.n] == 0, hs.codes[: hs.n] == 0), tag + " zero set"
        compare_bits(to_np(meta, hs.meta.shape[0]), hs.meta, tag + " meta")
        return near


RAGGED = [Shape("a", 1, 1), Shape("b", 1, 3), Shape("c", 1, 255), Shape("d", 2, 128), Shape("e", 1, 257),
          Shape("f", 3, 1000), Shape("g", 17, 256), Shape("h", 2048 * 3 + 5, 1), Shape("i", 8, 1024),
          Shape("j", 1, 64 * 5 + 1)]


def _spec(al, name, block):
    if name == "AL8":
        return al.Spec(al.AL8, block, V_FLOOR)
    if name == "AL16":
        return al.Spec(al.AL16, block, V_FLOOR)
    return al.Spec(al.FP32, 256)


@pytest.mark.parametrize("grad_bf16", [True, False])
@pytest.mark.parametrize("mc", ["UF8", "FP32"])
@pytest.mark.parametrize("vc,block", [("AL8", 64), ("AL8", 128), ("AL8", 256), ("AL8", 512), ("AL8", 1024),
                                      ("AL8", 2048), ("AL16", 128), ("AL16", 2048), ("FP32", 256)])
def test_adamw_ragged_lists(dev, grad_bf16, mc, vc, block):
    import paper_2608_22322_amd as al

    w = Workload("ragged", RAGGED, grad_bf16=grad_bf16, zero_frac=0.1, steps=3)
    mspec = al.Spec(al.UF8, 256) if mc == "UF8" else al.Spec(al.FP32, 256)
    pair = Pair(dev, RAGGED, w, mspec, _spec(al, vc, block))
    for t in (1, 2, 3):
        pair.step(t)
        pair.compare(t, 1e-5 * t)


def test_adamw_1024_workload(dev):
    """1024x1024 fp32 params/grads, 5% dormant entries for steps 1-5, AL8 v + UF8 m, block 256, 10 steps."""
    import paper_2608_22322_amd as al

    w = workload_1024()
    pair = Pair(dev, w.shapes, w, al.Spec(al.UF8, 256), al.Spec(al.AL8, 256, V_FLOOR))
    n = w.shapes[0].n
    dormant = np.ones(n, bool)  # every gradient so far exactly zero (the 5% mask, plus rare natural zeros)
    near = 0
    for t in range(1, w.steps + 1):
        pair.step(t)
        near += pair.compare(t, 1e-5 if t == 1 else 1e-4)
        dormant &= data.host_grad(0, w, t, np.arange(n)) == 0
        v = to_np(pair.states[0].v, n)
        m = to_np(pair.states[0].m, n)
        # exact zero (section 4.2): v code 0 exactly on entries that never saw a gradient
        assert np.array_equal(v == 0, dormant), t
        assert np.all(m[dormant] == 0), t
        if t <= 5:
            assert 0.045 < dormant.mean() < 0.055
        else:
            assert dormant.sum() < 5
    log(f"1024x1024: near-boundary code differences over 10 steps: {near}")


@pytest.mark.parametrize("block", [256, 2048])
def test_adamw_100_steps_tinyllama_shapes(dev, block):
    """100-step trajectory on a TinyLlama-shaped subset (a k/v projection, a norm, a ragged slab)."""
    import paper_2608_22322_amd as al

    shapes = [Shape("k", 256, 2048), Shape("attn_norm", 1, 2048), Shape("slab", 37, 999)]
    w = Workload("tl-subset", shapes, zero_frac=0.02, steps=100)
    pair = Pair(dev, shapes, w, al.Spec(al.UF8, 256), al.Spec(al.AL8, block, V_FLOOR))
    near = 0
    for t in range(1, 101):
        pair.step(t)
        if t in (1, 2, 5, 10, 25, 50, 75, 100):
            near += pair.compare(t, 1e-5 if t == 1 else 1e-4)
    log(f"100 steps B{block}: near-boundary code differences at checked steps: {near}")


def _sampled_full_size(dev, shapes, w, block, n_samples, steps, seed):
    """Run the full list on the GPU; recompute sampled whole tiles with the oracle from regenerated inputs."""
    T = max(block, 256)
    rng = np.random.default_rng(seed)
    picks = []
    for _ in range(n_samples):
        i = int(rng.integers(len(shapes)))
        ntiles = (shapes[i].n + T - 1) // T
        k = int(rng.integers(ntiles))
        picks.append((i, k))
    picks += [(0, 0), (len(shapes) - 1, (shapes[-1].n + T - 1) // T - 1)]
    return _sampled_full_size_picks(dev, shapes, w, block, steps, picks)


def _sampled_full_size_picks(dev, shapes, w, block, steps, picks):
    """As _sampled_full_size, for the given (tensor, tile) picks; a tile is max(B_V, 256) elements."""
    import torch

    import paper_2608_22322_amd as al

    T = max(block, 256)
    mspec, vspec = al.Spec(al.UF8, 256), al.Spec(al.AL8, block, V_FLOOR)
    states = []
    for i, s in enumerate(shapes):
        p = data.device_param(i, s, dev)
        g = data.device_grad_buffer(s, w, dev)
        m, mm = al.alloc_state(s.n, mspec, dev)
        v, vm = al.alloc_state(s.n, vspec, dev)
        states.append(al.ParamState(p, g, s.rows, s.cols, m=m, m_meta=mm, v=v, v_meta=vm))
    cfg = al.adamw_cfg(grad_bf16=True, m=mspec, v=vspec)
    arr = al.tensor_array(states)
    ws = al.workspace(al.adamw_workspace_bytes(states, cfg, arr=arr), dev)
    host = {}
    for (i, k) in picks:
        s = shapes[i]
        lo, hi = k * T, min(s.n, (k + 1) * T)
        L = hi - lo
        host[(i, k)] = dict(p=data.host_param(i, s, np.arange(lo, hi)),
                            m=oracle.State(mspec.codec, L, 256), v=oracle.State(vspec.codec, L, block, V_FLOOR))
    for t in range(1, steps + 1):
        for i, (s, st) in enumerate(zip(shapes, states)):
            data.fill_grad(st.grad, i, s, w, t)
        al.adamw_step(states, cfg, t, ws, arr=arr)
        for (i, k), h in host.items():
            lo, hi = k * T, min(shapes[i].n, (k + 1) * T)
            oracle.adamw_step(h["p"], data.host_grad(i, w, t, np.arange(lo, hi)), h["m"], h["v"], t)
        torch.cuda.synchronize()
    near = 0
    for (i, k), h in host.items():
        s, st = shapes[i], states[i]
        lo, hi = k * T, min(s.n, (k + 1) * T)
        tag = f"{s.name} tile {k}"
        compare_params(to_np(st.param[lo:hi]), h["p"], 1e-5 * steps, tag)
        mc = to_np(st.m[lo:lo + h["m"].codes.shape[0]]).astype(np.int8)
        near += compare_codes(mc, h["m"].codes, h["m"].y, tag + " m")
        compare_bits(to_np(st.m_meta[lo // 256: lo // 256 + h["m"].meta.shape[0]]), h["m"].meta, tag + " m meta")
        vc = to_np(st.v[lo:lo + h["v"].codes.shape[0]])
        near += compare_codes(vc, h["v"].codes, h["v"].y, tag + " v")
        nb = h["v"].meta.shape[0]
        compare_bits(to_np(st.v_meta[2 * (lo // block): 2 * (lo // block) + nb]), h["v"].meta, tag + " v meta")
    return near


@pytest.mark.parametrize("block", [256, 2048])
def test_adamw_full_size_tinyllama_sampled(dev, block):
    w = Workload("tinyllama", tinyllama_shapes(), zero_frac=0.02, steps=3)
    log(f"TinyLlama-1.1B full size, B_V {block}")
    near = _sampled_full_size(dev, w.shapes, w, block, 48, 3, 5)
    log(f"near-boundary code differences: {near}")


@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024, 2048])
def test_adamw_full_size_llama7b_sampled(dev, block):
    import torch

    w = Workload("llama-7b", llama7b_shapes(), zero_frac=0.01, steps=2)
    log(f"Llama-7B full size, B_V {block}")
    near = _sampled_full_size(dev, w.shapes, w, block, 32, 2, 9)
    log(f"near-boundary code differences: {near}")
    torch.cuda.empty_cache()


@pytest.mark.parametrize("block", [64, 2048])
def test_adamw_tensor_beyond_2_31_elements(dev, block):
    """One tensor of 2^31 + 3 * 2048 + 778 elements (64-bit offsets, ragged last chunk); sampled
    tiles below and above 2^31 recomputed by the oracle."""
    import torch

    cols = 2**30 + 3 * 1024 + 389
    n = 2 * cols
    shapes = [Shape("huge", 2, cols)]
    w = Workload("huge", shapes, zero_frac=0.01, steps=2)
    log(f"one tensor of {n} elements, B_V {block}")
    T = max(block, 256)
    near = _sampled_full_size_picks(dev, shapes, w, block, 2, [(0, 0), (0, 2**31 // T - 1), (0, 2**31 // T),
                                                               (0, 2**31 // T + 1), (0, (n + T - 1) // T - 1)])
    log(f"near-boundary code differences: {near}")
    torch.cuda.empty_cache()
