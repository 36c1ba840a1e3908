"""GPU parity of the APOLLO projected-state step (al_apollo_step) against the CPU oracle
(oracle/apollo.py).

* ragged tensor lists on both projection sides (rows >= cols: channels are rows; rows < cols:
  channels are columns), partial 32-channel projection tiles, partial 256x256 update units,
  projected lengths below and above the rank;
* the projection's slice and tile edges: projected lengths of one 16-input slice, one slice and
  one input, an odd number of slices, and channel counts one past a tile, at every rank;
* ranks 64, 128 and 256, bf16 and fp32 gradients, UF8 + AL8 B2048 codes and FP32 states;
* three steps with the norm-growth limiter on, an all-zero gradient channel;
* the ApolloStep driver over a small named list (projected and full-AdamW tensors).

Rules: the projected moments' codes follow the code rule (bit-exact except an element whose oracle
position lies within 1e-4 of a rounding boundary); fp32 states bit-exact; the limiter state and the
parameters to 1e-5 relative (the direction on the projected space is fp32 on the GPU, binary64 then
fp32 in the oracle, so the channel scales agree to a few fp32 ulps).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import apollo as oap
from paper_2608_22322_amd import synth

from .gpu_util import compare_bits, compare_codes, compare_params, log, require_gpu, to_np

pytestmark = pytest.mark.gpu

FLOOR = float(np.float32(2 * math.log2(1e-8)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def _grad(i, t, rows, cols, bf16, zero_channel=None):
    g = synth.normal_f32(synth.grad_key(i, t), rows * cols, 1e-3, synth.mask_key(i), 0.02).reshape(rows, cols)
    if zero_channel is not None:
        if rows >= cols:
            g[zero_channel, :] = 0.0
        else:
            g[:, zero_channel] = 0.0
    g = g.ravel()
    return synth.to_bf16_bits(g) if bf16 else g


def _run(dev, shapes, rank, bf16, coded, steps=3, gamma=1.01, zero_channel=None):
    import torch

    import paper_2608_22322_amd as al

    mspec = al.Spec(al.UF8, 256) if coded else al.Spec(al.FP32, 256)
    vspec = al.Spec(al.AL8, 2048, FLOOR) if coded else al.Spec(al.FP32, 2048)
    cfg = al.apollo_cfg(lr=1e-4, gamma=gamma, rank=rank, grad_bf16=bf16, m=mspec, v=vspec)
    items, host = [], []
    for i, (rows, cols) in enumerate(shapes):
        right, C, L = oap.layout(rows, cols)
        p0 = synth.normal_f32(synth.param_key(i), rows * cols, 0.02)
        P = synth.proj_matrix(i, 0, L, rank)
        p = torch.from_numpy(p0.copy()).to(dev)
        g = torch.empty(rows * cols, dtype=torch.bfloat16 if bf16 else torch.float32, device=dev)
        m, mm = al.alloc_state(C * rank, mspec, dev)
        v, vm = al.alloc_state(C * rank, vspec, dev)
        pj = torch.empty(L * rank, dtype=torch.float32, device=dev)
        al.synth_normal(pj, synth.proj_key(i, 0), 1.0 / math.sqrt(rank))
        ns = torch.zeros(4, dtype=torch.float32, device=dev)
        items.append((p, g, rows, cols, pj, m, mm, v, vm, ns))
        hm = oracle.State(mspec.codec, C * rank, 256)
        hv = oracle.State(vspec.codec, C * rank, 2048, FLOOR)
        host.append(dict(p=p0.copy(), P=P, m=hm, v=hv, prev=np.zeros(1, np.float32), pj=pj))
    arr = al.apollo_tensor_array(items)
    ws = torch.empty(al.apollo_workspace_bytes(arr, len(items), cfg), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    for i, h in enumerate(host):  # the device projection is the host's, bit for bit
        assert np.array_equal(to_np(h["pj"]), h["P"].ravel())
    for t in range(1, steps + 1):
        for i, (rows, cols) in enumerate(shapes):
            gh = _grad(i, t, rows, cols, bf16, zero_channel)
            gd = torch.from_numpy(gh.view(np.int16) if bf16 else gh).to(dev)
            items[i][1].copy_(gd.view(torch.bfloat16) if bf16 else gd)
            h = host[i]
            oap.apollo_step(h["p"], gh, rows, cols, h["P"], h["m"], h["v"], t, h["prev"], lr=1e-4, gamma=gamma)
        al.apollo_step(arr, len(items), cfg, t, ws)
        torch.cuda.synchronize()
        near = 0
        for i, (rows, cols) in enumerate(shapes):
            right, C, L = oap.layout(rows, cols)
            n = C * rank
            h, it = host[i], items[i]
            what = f"{(rows, cols)} r{rank} t{t}"
            compare_params(to_np(it[0]), h["p"], 1e-5, f"{what} param")
            if coded:
                near += compare_codes(to_np(it[5], n), h["m"].codes[:n], h["m"].y, f"{what} m codes")
                near += compare_codes(to_np(it[7], n), h["v"].codes[:n], h["v"].y, f"{what} v codes")
                if near == 0:
                    compare_bits(to_np(it[6])[:len(h["m"].meta)], h["m"].meta, f"{what} m meta")
                    compare_bits(to_np(it[8])[:len(h["v"].meta)], h["v"].meta, f"{what} v meta")
            else:
                compare_bits(to_np(it[5], n), h["m"].codes[:n], f"{what} m")
                compare_bits(to_np(it[7], n), h["v"].codes[:n], f"{what} v")
            if gamma > 0:
                ns = float(to_np(it[9])[0])
                assert math.isclose(ns, float(h["prev"][0]), rel_tol=1e-5), (what, ns, float(h["prev"][0]))
        log(f"apollo {shapes} rank {rank} bf16 {bf16} coded {coded} t{t}: near-boundary code diffs {near}")


RAGGED = [(70, 33), (40, 300), (300, 40), (256, 256), (5, 700), (129, 64)]


@pytest.mark.parametrize("rank", [64, 128, 256])
@pytest.mark.parametrize("bf16", [True, False])
def test_apollo_coded_ragged(dev, rank, bf16):
    _run(dev, RAGGED, rank, bf16, coded=True)


# (rows, cols) -> (channels, projected length): (33, 16) 33 x 16, (32, 17) 32 x 17, (64, 32) 64 x 32,
# (65, 48) 65 x 48, (16, 100) 100 x 16, (17, 96) 96 x 17, (31, 48) 48 x 31
EDGES = [(33, 16), (32, 17), (64, 32), (65, 48), (16, 100), (17, 96), (31, 48)]


@pytest.mark.parametrize("rank", [64, 128, 256])
@pytest.mark.parametrize("bf16", [True, False])
def test_apollo_projection_slice_and_tile_edges(dev, rank, bf16):
    _run(dev, EDGES, rank, bf16, coded=True, steps=2)


def test_apollo_fp32_states(dev):
    _run(dev, [(96, 40), (33, 130)], 64, True, coded=False)


def test_apollo_zero_channel_and_no_limiter(dev):
    _run(dev, [(80, 48), (48, 80)], 64, True, coded=True, gamma=0.0, zero_channel=7)


def test_apollo_tinyllama_layer_shapes(dev):
    # one TinyLlama decoder layer's projected tensors (q, k, o, gate, down) at rank 256
    _run(dev, [(2048, 2048), (256, 2048), (5632, 2048), (2048, 5632)], 256, True, coded=True, steps=2)


def test_apollo_driver_mixed_list(dev):
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import apollo

    names = ["embed", "layer0.q", "layer0.down", "layer0.attn_norm"]
    shapes = [(64, 40), (48, 48), (40, 96), (1, 48)]
    states, host = [], []
    for i, (rows, cols) in enumerate(shapes):
        p0 = synth.normal_f32(synth.param_key(i), rows * cols, 0.02)
        st = al.ParamState(torch.from_numpy(p0.copy()).to(dev), torch.empty(rows * cols, dtype=torch.bfloat16,
                                                                               device=dev), rows, cols)
        states.append(st)
        host.append(p0.copy())
    cfg = al.apollo_cfg(rank=64)
    drv = apollo.ApolloStep(states, names, cfg, gap=2)
    hs = []
    for i, (rows, cols) in enumerate(shapes):
        if apollo.projected(names[i], rows, cols):
            right, C, L = oap.layout(rows, cols)
            hs.append((oracle.State(oracle.UF8, C * 64, 256), oracle.State(oracle.AL8, C * 64, 2048, FLOOR),
                       np.zeros(1, np.float32)))
        else:
            hs.append((oracle.State(oracle.UF8, rows * cols, 256), oracle.State(oracle.AL8, rows * cols, 2048, FLOOR),
                       None))
    for t in range(1, 4):  # the projection is redrawn at step 3 (gap 2)
        for i, (rows, cols) in enumerate(shapes):
            gh = _grad(i, t, rows, cols, True)
            states[i].grad.copy_(torch.from_numpy(gh.view(np.int16)).to(dev).view(torch.bfloat16))
            m, v, prev = hs[i]
            if prev is not None:
                right, C, L = oap.layout(rows, cols)
                P = synth.proj_matrix(i, (t - 1) // 2, L, 64)
                oap.apollo_step(host[i], gh, rows, cols, P, m, v, t, prev, lr=1e-4)
            else:
                oracle.adamw_step(host[i], gh, m, v, t, lr=1e-4, wd=0.0)
        drv.step(t)
        torch.cuda.synchronize()
        for i in range(len(shapes)):
            compare_params(to_np(states[i].param)[:host[i].shape[0]], host[i], 1e-5, f"{names[i]} t{t}")


def test_apollo_full_tinyllama_list_sampled(dev):
    """The whole 201-tensor TinyLlama list through ApolloStep (the bench's configuration: 154 projected
    layer matrices at rank 256, embedding/head/norms under AdamW); whole small tensors recomputed by the
    oracle -- projected ones (left and right) and 1-D ones -- after each of two steps."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd import apollo, data
    from paper_2608_22322_amd.workloads import tinyllama_shapes, workload_tinyllama

    shapes = tinyllama_shapes()
    w = workload_tinyllama(zero_frac=0.02)
    states = []
    for i, s in enumerate(shapes):
        states.append(al.ParamState(data.device_param(i, s, dev), data.device_grad_buffer(s, w, dev), s.rows, s.cols))
    drv = apollo.ApolloStep(states, [s.name for s in shapes], al.apollo_cfg(), device=dev)
    names = ("layer0.k", "layer7.v", "layer3.q", "layer0.attn_norm", "norm")
    sample = [i for i, s in enumerate(shapes) if s.name in names]
    host = {}
    for i in sample:
        s = shapes[i]
        p0 = data.host_param(i, s, np.arange(s.n))
        if apollo.projected(s.name, s.rows, s.cols):
            right, C, L = oap.layout(s.rows, s.cols)
            host[i] = dict(p=p0.copy(), P=synth.proj_matrix(i, 0, L, 256), m=oracle.State(oracle.UF8, C * 256, 256),
                           v=oracle.State(oracle.AL8, C * 256, 2048, FLOOR), prev=np.zeros(1, np.float32),
                           k=drv.proj_idx.index(i))
        else:
            host[i] = dict(p=p0.copy(), m=oracle.State(oracle.UF8, s.n, 256), v=oracle.State(oracle.AL8, s.n, 2048, FLOOR))
    log(f"APOLLO full TinyLlama list, sampled tensors {[shapes[i].name for i in sample]}")
    for t in (1, 2):
        for i, s in enumerate(shapes):
            data.fill_grad(states[i].grad, i, s, w, t)
        drv.step(t)
        torch.cuda.synchronize()
        for i in sample:
            s, h = shapes[i], host[i]
            gh = data.host_grad(i, w, t, np.arange(s.n))
            what = f"{s.name} t{t}"
            if "P" in h:
                oap.apollo_step(h["p"], gh, s.rows, s.cols, h["P"], h["m"], h["v"], t, h["prev"], lr=1e-4)
                it = drv.items[h["k"]]
                n = oap.layout(s.rows, s.cols)[1] * 256
                compare_codes(to_np(it[5], n), h["m"].codes[:n], h["m"].y, f"{what} m codes")
                compare_codes(to_np(it[7], n), h["v"].codes[:n], h["v"].y, f"{what} v codes")
                assert math.isclose(float(to_np(it[9])[0]), float(h["prev"][0]), rel_tol=1e-5), what
            else:
                oracle.adamw_step(h["p"], gh, h["m"], h["v"], t, lr=1e-4, wd=0.0)
                compare_codes(to_np(states[i].m, s.n), h["m"].codes[:s.n], h["m"].y, f"{what} m codes")
                compare_codes(to_np(states[i].v, s.n), h["v"].codes[:s.n], h["v"].y, f"{what} v codes")
            compare_params(to_np(states[i].param)[:s.n], h["p"], 1e-5, f"{what} param")
    del drv, states
    torch.cuda.empty_cache()
