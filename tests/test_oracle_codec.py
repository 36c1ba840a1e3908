"""Pins for the oracle's codec: what the paper and the mathematics fix.

Each test checks the CPU oracle against something other than itself: hand-
derived worked examples, the exact-zero invariant (section 4.2), the endpoint
codes implied by Eq. al_quant at z = 0 and z = 1, brute-force nearest-level
search on tiny blocks, the half-step round-trip bound, level coverage, and
Python's math.fsum for the exact summation.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "al_worked_examples.json")


def _f32(x):
    return np.asarray(x, dtype=np.float32)


# ---------------------------------------------------------------- worked examples
def test_worked_examples_al():
    ex = json.load(open(GOLD))["al"]
    for e in ex:
        codes, meta, _ = oracle.al_quantize(e["bits"], _f32(e["x"]), e["block"], e["log_floor"])
        assert codes.tolist() == e["codes"], e["name"]
        if "meta" in e:
            assert meta.tolist() == e["meta"], e["name"]
        else:
            assert meta[0] == np.float32(math.log2(e["meta_lmin_is_fl32_log2_of"])), e["name"]
            assert meta[1] == np.float32(e["meta_delta"]), e["name"]
        if "decoded" in e:
            dec = oracle.al_dequantize(e["bits"], codes, meta, len(e["x"]), e["block"])
            assert dec.tolist() == e["decoded"], e["name"]


def test_worked_examples_uf8():
    for e in json.load(open(GOLD))["uf8"]:
        codes, meta, _ = oracle.uf8_quantize(_f32(e["x"]), e["block"])
        assert codes.tolist() == e["codes"], e["name"]
        assert meta.tolist() == e["meta"]
        dec = oracle.uf8_dequantize(codes, meta, len(e["x"]), e["block"])
        want = np.array(e["decoded_num_over_127"], dtype=np.float64) / 127.0
        np.testing.assert_allclose(dec, want, rtol=1e-7, atol=0)


# ---------------------------------------------------------------- exact zero
def _random_positive(rng, n):
    """Positive fp32 values over a wide log range, some subnormal."""
    e = rng.uniform(-140.0, 60.0, n)
    return _f32(np.exp2(e) * rng.uniform(1.0, 2.0, n))


@pytest.mark.parametrize("bits", [8, 16])
def test_exact_zero_invariant_exhaustive_masks(bits):
    """q = 0 <=> x = 0 over all 2^8 zero patterns of an 8-element block (Eq. exact_zero)."""
    rng = np.random.default_rng(1)
    for mask in range(256):
        for trial in range(4):
            x = _random_positive(rng, 8)
            zero = np.array([(mask >> i) & 1 for i in range(8)], dtype=bool)
            x[zero] = np.where(rng.random(zero.sum()) < 0.5, 0.0, -0.0).astype(np.float32)
            floor = float(rng.choice([-126.0, -53.0, -20.0]))
            codes, meta, _ = oracle.al_quantize(bits, x, 8, floor)
            assert np.array_equal(codes == 0, zero), (mask, x)
            dec = oracle.al_dequantize(bits, codes, meta, 8, 8)
            assert np.array_equal(dec == 0, zero), (mask, x, dec)
            assert np.all(dec[~zero] > 0)


# ---------------------------------------------------------------- endpoints
@pytest.mark.parametrize("bits", [8, 16])
@pytest.mark.parametrize("block", [64, 256, 2048])
def test_endpoint_codes(bits, block):
    """Non-degenerate blocks inside [2^floor, 2^126]: min -> code 1, max -> code L-1."""
    rng = np.random.default_rng(block + bits)
    top = (1 << bits) - 1
    for trial in range(20):
        width = float(rng.choice([1e-3, 0.5, 4.0, 40.0]))
        lo = rng.uniform(-50.0, 20.0)
        x = _f32(np.exp2(lo + width * rng.random(block)))
        x[rng.random(block) < 0.1] = 0.0
        codes, meta, _ = oracle.al_quantize(bits, x, block, -53.0)
        pos = x > 0
        if x[pos].min() == x[pos].max():
            continue
        assert codes[np.argmin(np.where(pos, x, np.inf))] == 1
        assert codes[np.argmax(x)] == top
        assert codes[pos].min() == 1 and codes[pos].max() == top


# ---------------------------------------------------------------- brute force
@pytest.mark.parametrize("bits", [8, 16])
def test_bruteforce_nearest_level(bits):
    """For 8-element blocks the closed-form code is the level nearest in log2 among
    all L-1 positive levels l_min + (k-1) * delta / (L-2) (ties excluded)."""
    rng = np.random.default_rng(7 + bits)
    L2 = (1 << bits) - 2
    k = np.arange(1, L2 + 2, dtype=np.float64)
    checked = 0
    for trial in range(300):
        span = float(rng.choice([0.01, 1.0, 8.0, 90.0]))
        x = _f32(np.exp2(rng.uniform(-40, -40 + span, 8)))
        x[rng.random(8) < 0.2] = 0.0
        floor = float(rng.choice([-126.0, -53.0, -35.0]))
        codes, meta, y = oracle.al_quantize(bits, x, 8, floor)
        pos = x > 0
        if pos.sum() < 2 or x[pos].min() == x[pos].max():
            continue
        # brute force from the fitted interval recomputed independently here
        lmin = max(floor, math.log2(float(x[pos].min())))
        lmax = min(math.log2(float(x[pos].max())), 126.0)
        delta = max(lmax - lmin, 1e-12)
        levels = lmin + (k - 1.0) * delta / L2
        for i in np.nonzero(pos)[0]:
            t = math.log2(float(x[i]))
            dist = np.abs(levels - t)
            best = int(k[np.argmin(dist)])
            frac = y[i] - math.floor(y[i])
            if abs(frac - 0.5) < 1e-9:
                continue
            assert codes[i] == best, (trial, i, codes[i], best)
            checked += 1
    assert checked > 500


# ---------------------------------------------------------------- round trip
@pytest.mark.parametrize("bits", [8, 16])
def test_round_trip_half_step(bits):
    """|log2 xhat - log2 x| <= delta / (2 (L-2)) + metadata/output rounding, for x in the interval."""
    rng = np.random.default_rng(11 + bits)
    L2 = (1 << bits) - 2
    for trial in range(50):
        B = 256
        span = float(rng.choice([0.3, 3.0, 30.0]))
        x = _f32(np.exp2(rng.uniform(-30, -30 + span, B)))
        codes, meta, _ = oracle.al_quantize(bits, x, B, -126.0)
        dec = oracle.al_dequantize(bits, codes, meta, B, B)
        lmin, delta = float(meta[0]), float(meta[1])
        ulp = lambda v: float(np.spacing(np.float32(abs(v))))
        bound = delta / (2 * L2) + 0.5 * ulp(lmin) + 0.5 * ulp(delta) + 2.0**-23 + 1e-12
        err = np.abs(np.log2(dec.astype(np.float64)) - np.log2(x.astype(np.float64)))
        assert err.max() <= bound, (trial, err.max(), bound)


def test_al8_uses_every_level():
    """AL8 has 255 positive levels (section 4.1); a dense random block set hits all of them."""
    rng = np.random.default_rng(3)
    x = _f32(np.exp2(rng.uniform(-20, -10, 256 * 400)))
    codes, _, _ = oracle.al_quantize(8, x, 256, -126.0)
    assert set(np.unique(codes).tolist()) == set(range(1, 256))


def test_al16_uses_every_level():
    """AL16 has 65,535 positive levels (section 4.1). Blocks with endpoints 1 and 2 (l_min 0, width 1)
    and interior values placed on the level grid reach every code exactly once per level."""
    L2 = 65534
    B = 2048
    levels = np.arange(L2 + 1, dtype=np.float64)  # code - 1
    per = B - 2
    nblk = -(-levels.shape[0] // per)
    x = np.empty(nblk * B, np.float32)
    for b in range(nblk):
        k = levels[b * per:(b + 1) * per]
        k = np.concatenate([k, np.full(per - k.shape[0], k[-1])])
        x[b * B:(b + 1) * B] = _f32(np.concatenate([[1.0, 2.0], np.exp2(k / L2)]))
    codes, meta, _ = oracle.al_quantize(16, x, B, -126.0)
    assert np.all(meta[0::2] == 0.0) and np.all(meta[1::2] == 1.0)
    assert set(np.unique(codes).tolist()) == set(range(1, 65536))
    interior = codes.reshape(nblk, B)[:, 2:].reshape(-1)[: levels.shape[0]]
    assert np.array_equal(interior.astype(np.int64), levels.astype(np.int64) + 1)


def test_block_below_floor_decodes_to_floor():
    """Every value below the floor: interval width clamps, all codes 1, decode 2^floor."""
    x = _f32([2.0**-80, 2.0**-70, 2.0**-60])
    codes, meta, _ = oracle.al_quantize(8, x, 8, -53.0)
    assert codes[:3].tolist() == [1, 1, 1]
    assert meta[0] == -53.0 and meta[1] == np.float32(1e-12)
    dec = oracle.al_dequantize(8, codes, meta, 3, 8)
    assert np.all(dec == np.float32(2.0**-53))


def test_partial_last_block_and_padding():
    rng = np.random.default_rng(5)
    n = 64 * 3 + 17
    x = _f32(np.exp2(rng.uniform(-10, 0, n)))
    codes, meta, _ = oracle.al_quantize(8, x, 64, -53.0)
    assert codes.shape[0] == 256 and np.all(codes[n:] == 0) and np.all(codes[:n] > 0)
    # the last block's interval comes from its 17 elements only
    assert meta[6] == np.float32(max(-53.0, math.log2(float(x[192:].min()))))


# ---------------------------------------------------------------- UF8
def test_uf8_properties():
    rng = np.random.default_rng(9)
    x = _f32(rng.normal(0, 1e-3, 256 * 64))
    x[rng.random(x.shape[0]) < 0.05] = 0.0
    codes, meta, _ = oracle.uf8_quantize(x, 256)
    dec = oracle.uf8_dequantize(codes, meta, x.shape[0], 256)
    xb = x.reshape(-1, 256)
    cb = codes.reshape(-1, 256)
    assert np.array_equal(meta, np.abs(xb).max(axis=1))
    for b in range(xb.shape[0]):
        i = np.argmax(np.abs(xb[b]))
        assert abs(int(cb[b, i])) == 127
    assert np.all((codes == 0) == (x == 0) | (np.abs(x) < np.repeat(meta, 256) / 254 * 1.0000001))
    # no sign flips; error at most half a step
    assert np.all(np.sign(dec) * np.sign(x) >= 0)
    step = np.repeat(meta, 256).astype(np.float64) / 127.0
    assert np.all(np.abs(dec.astype(np.float64) - x) <= step / 2 * (1 + 1e-6) + 1e-12)
    assert codes.min() >= -127


def test_uf8_zero_block():
    codes, meta, _ = oracle.uf8_quantize(np.zeros(300, np.float32), 256)
    assert np.all(codes == 0) and np.all(meta == 0)
    assert np.all(oracle.uf8_dequantize(codes, meta, 300, 256) == 0)


# ---------------------------------------------------------------- exact sum
def test_exact_sum_matches_fsum():
    rng = np.random.default_rng(13)
    for trial in range(200):
        n = int(rng.integers(1, 3000))
        kind = trial % 4
        if kind == 0:
            x = rng.normal(size=n)
        elif kind == 1:
            x = np.exp2(rng.uniform(-300, 300, n)) * rng.choice([-1, 1], n)
        elif kind == 2:
            x = rng.normal(size=n) * 1e-3
            x = np.concatenate([x, -x[: n // 2], [1e100, -1e100, 1e-30]])
        else:
            x = np.abs(rng.normal(size=n)) ** 2 + 1e-30
        assert oracle.exact_sum(x) == math.fsum(x.tolist()), trial
