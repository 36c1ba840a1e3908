"""GPU parity of the standalone codecs (al_quantize / al_dequantize) and of the
synthetic-input fill against the CPU oracle / host generator."""
import math

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import synth

from .gpu_util import compare_bits, compare_codes, log, require_gpu, to_np

pytestmark = pytest.mark.gpu

CODECS = {"AL8": 1, "AL16": 2, "UF8": 3}


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def test_synth_fill_matches_host(dev):
    import torch

    import paper_2608_22322_amd as al

    for n, dt, frac in ((1_000_003, torch.bfloat16, 0.02), (65_537, torch.float32, 0.05), (13, torch.float32, 0.0)):
        key, mk = synth.grad_key(3, 7), synth.mask_key(3)
        buf = torch.empty(n + 8, dtype=dt, device=dev)
        al.synth_normal(buf[:n], key, 1e-3, mk, frac)
        torch.cuda.synchronize()
        host = synth.normal_f32(key, n, 1e-3, mk, frac)
        if dt == torch.bfloat16:
            assert np.array_equal(to_np(buf, n), synth.to_bf16_bits(host))
        else:
            compare_bits(to_np(buf, n), host, "synth f32")
        if frac:
            assert abs((host == 0).mean() - frac) < 0.01


def _inputs(kind: str, n: int, rng) -> np.ndarray:
    if kind == "uf8":
        x = rng.normal(0, 1e-3, n).astype(np.float32)
        x[rng.random(n) < 0.05] = 0.0
        return x
    if kind == "narrow":
        x = np.exp2(rng.uniform(-22, -20.5, n))
    elif kind == "wide":
        x = np.exp2(rng.uniform(-140, 100, n))  # includes subnormals and values near the cap
    elif kind == "embed":  # 40-85% exact zeros, wide range (section 3.3 statistics)
        x = np.exp2(rng.uniform(-90, -10, n))
        x[rng.random(n) < rng.uniform(0.4, 0.85)] = 0.0
    else:
        raise ValueError(kind)
    x = x.astype(np.float32)
    x[rng.random(n) < 0.03] = 0.0
    return x


def _run_codec(dev, codec, block, x, lf):
    import torch

    import paper_2608_22322_amd as al

    n = x.shape[0]
    xd = torch.from_numpy(np.concatenate([x, np.zeros(4, np.float32)])).to(dev)
    codes, meta = al.alloc_state(n, al.Spec(codec, block), dev)
    codes.fill_(0x55 if codec != 2 else 0x5555)  # padding must be rewritten as 0
    al.quantize(codec, xd[:n], block, lf, codes, meta)
    out = torch.empty(n + 4, dtype=torch.float32, device=dev)
    al.dequantize(codec, codes, meta, n, block, out)
    torch.cuda.synchronize()
    nc = al.code_bytes(codec, n, block) // (2 if codec == 2 else 1)
    return to_np(codes, nc), to_np(meta, al.meta_floats(codec, n, block)), to_np(out, n)


@pytest.mark.parametrize("codec", ["AL8", "AL16", "UF8"])
@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024, 2048])
def test_quantize_dequantize_parity(dev, codec, block):
    c = CODECS[codec]
    rng = np.random.default_rng(block * 7 + c)
    kinds = ["uf8"] if codec == "UF8" else ["narrow", "wide", "embed"]
    near = 0
    for kind in kinds:
        for n in (block * 9 + 2048 * 3 + 5, 2048 * 7, 3, 0, block - 1, 4 * 2048 + 257):
            x = _inputs(kind, n, rng)
            lf = float(np.float32(-53.150849518197795 if kind != "wide" else -126.0))
            g_codes, g_meta, g_out = _run_codec(dev, c, block, x, lf)
            if codec == "UF8":
                o_codes, o_meta, y = oracle.uf8_quantize(x, block)
                o_out = oracle.uf8_dequantize(o_codes, o_meta, n, block)
            else:
                bits = 8 if codec == "AL8" else 16
                o_codes, o_meta, y = oracle.al_quantize(bits, x, block, lf)
                o_out = oracle.al_dequantize(bits, o_codes, o_meta, n, block)
            tag = f"{codec} B{block} {kind} n{n}"
            near += compare_codes(g_codes, o_codes, y, tag)
            compare_bits(g_meta, o_meta, tag + " meta")
            # decode from the GPU's own codes so a near-boundary code difference does not cascade
            if codec == "UF8":
                ref = oracle.uf8_dequantize(g_codes.astype(np.int8), g_meta, n, block)
            else:
                ref = oracle.al_dequantize(bits, g_codes, g_meta, n, block)
            compare_bits(g_out, ref, tag + " decode")
            if near == 0:
                compare_bits(g_out, o_out, tag + " decode vs oracle codes")
    log(f"{codec} B{block}: near-boundary code differences: {near}")


def test_degenerate_blocks(dev):
    """All-zero, coincident, below-floor and near-cap blocks (section 4.1 rules)."""
    B = 256
    blocks = [
        np.zeros(B, np.float32),
        np.full(B, 3.0, np.float32),
        np.where(np.arange(B) % 3 == 0, 0.0, 7.5e-20).astype(np.float32),
        np.exp2(np.linspace(-80, -60, B)).astype(np.float32),
        np.exp2(np.linspace(100, 127.9, B)).astype(np.float32),
        np.where(np.arange(B) == 5, 1e-45, 0.0).astype(np.float32),
        np.where(np.arange(B) < 2, np.float32(1.0), np.float32(np.nextafter(np.float32(1), np.float32(2)))),
    ]
    x = np.concatenate(blocks).astype(np.float32)
    for codec, bits in (("AL8", 8), ("AL16", 16)):
        g_codes, g_meta, g_out = _run_codec(dev, CODECS[codec], B, x, -53.0)
        o_codes, o_meta, y = oracle.al_quantize(bits, x, B, -53.0)
        compare_codes(g_codes, o_codes, y, codec + " degenerate")
        compare_bits(g_meta, o_meta, codec + " degenerate meta")
        compare_bits(g_out, oracle.al_dequantize(bits, o_codes, o_meta, x.shape[0], B), codec + " degenerate decode")
        assert np.array_equal(g_codes[: x.shape[0]] == 0, x == 0)


@pytest.mark.parametrize("codec", ["AL8", "UF8"])
def test_quantize_beyond_2_31_elements(dev, codec):
    """al_quantize / al_dequantize over 2^31 + 2048 + 333 elements (64-bit offsets, partial last
    block); blocks below and above 2^31 recomputed by the oracle from regenerated inputs."""
    import torch

    import paper_2608_22322_amd as al

    B = 256
    n = 2**31 + 2048 + 333
    key = synth.grad_key(77, 1)
    xd = torch.empty(n + 4, dtype=torch.float32, device=dev)
    al.synth_normal(xd[:n], key, 1e-3)
    if codec == "AL8":
        xd.abs_()
    c = CODECS[codec]
    codes, meta = al.alloc_state(n, al.Spec(c, B), dev)
    al.quantize(c, xd[:n], B, -53.0, codes, meta)
    out = torch.empty(n + 4, dtype=torch.float32, device=dev)
    al.dequantize(c, codes, meta, n, B, out)
    torch.cuda.synchronize()
    nb = (n + B - 1) // B
    near = 0
    for b in (0, 2**31 // B - 1, 2**31 // B, 2**31 // B + 1, nb - 1):
        lo, hi = b * B, min(n, (b + 1) * B)
        x = synth.normal_f32(key, np.arange(lo, hi), 1e-3)
        if codec == "AL8":
            x = np.abs(x)
        g_codes = to_np(codes[lo:lo + B])
        if codec == "UF8":
            o_codes, o_meta, y = oracle.uf8_quantize(x, B)
            g_codes = g_codes.astype(np.int8)
            compare_bits(to_np(meta[b:b + 1]), o_meta, f"{codec} block {b} meta")
            ref = oracle.uf8_dequantize(g_codes, o_meta, hi - lo, B)
        else:
            o_codes, o_meta, y = oracle.al_quantize(8, x, B, -53.0)
            compare_bits(to_np(meta[2 * b:2 * b + 2]), o_meta, f"{codec} block {b} meta")
            ref = oracle.al_dequantize(8, g_codes, o_meta, hi - lo, B)
        near += compare_codes(g_codes, o_codes, y, f"{codec} block {b}")
        compare_bits(to_np(out[lo:hi]), ref, f"{codec} block {b} decode")
    log(f"{codec} beyond 2^31: near-boundary code differences {near}")
    del xd, out, codes, meta
    torch.cuda.empty_cache()
