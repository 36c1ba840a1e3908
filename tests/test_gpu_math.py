"""Device math primitives the codes rely on, bounded against the host.

* The hardware fp32 log2 on mantissas in [1/2, 1) (the fast code position):
  its error over all 2^23 mantissas must stay below a quarter of the guard
  band the encoder assumes (kLog2MantErr = 2^-21), so every code decision
  outside the band equals the binary64 one.
* The binary64 exp2 polynomial (decoding): relative error about one ulp.
* binary64 log2, sqrt and 1/sqrt (block endpoints, factored reconstruction):
  sqrt and the division are IEEE correctly rounded, so they must match the
  host bit for bit; log2 within one ulp.
"""
import numpy as np
import pytest

from .gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

GUARD = 2.0**-21


def _run(fn, x):
    import torch

    import paper_2608_22322_amd as al

    xd = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).cuda()
    out = torch.empty_like(xd)
    al.diag_math(fn, xd, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_hw_log2_on_mantissas_is_within_guard():
    require_gpu()
    m = (np.arange(1 << 23, dtype=np.uint32) | np.uint32(0x3F000000)).view(np.float32)  # all of [1/2, 1)
    got = _run(0, m.astype(np.float64))
    ref = np.log2(m.astype(np.float64))
    err = np.abs(got - ref).max()
    log(f"hardware fp32 log2 on [1/2,1): max abs error {err:.3e} = 2^{np.log2(err):.2f}")
    assert err <= GUARD / 4


def test_exp2_polynomial_relative_error():
    require_gpu()
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.uniform(-150, 128, 1 << 20), np.arange(-150, 128, 0.25)])
    got = _run(1, x)
    ld = np.exp2(x.astype(np.longdouble))
    rel = float(np.abs((got.astype(np.longdouble) - ld) / ld).max())
    log(f"exp2 polynomial: max rel error {rel:.3e}")
    assert rel < 2.5e-16
    # rounded to fp32 it agrees with the host's exp2 except within ~1e-16 of a midpoint
    mism = np.count_nonzero(got.astype(np.float32) != np.exp2(x).astype(np.float32))
    assert mism <= 2, mism


def test_log2_sqrt_rsqrt():
    require_gpu()
    rng = np.random.default_rng(2)
    x = np.exp2(rng.uniform(-140, 120, 1 << 20))
    lg = _run(2, x)
    ulp = np.spacing(np.abs(np.log2(x)))
    assert np.all(np.abs(lg - np.log2(x)) <= ulp)
    assert np.array_equal(_run(3, x), np.sqrt(x))
    assert np.array_equal(_run(4, x), 1.0 / np.sqrt(x))


def test_fit_log2_matches_host_log2():
    """The block-endpoint log2 of an fp32 value (fn 8) against the host libm log2 (the oracle's):
    every fp32 significand of the binade [2^-20, 2^-19), every significand of [1/2, 2) (results
    near 0), 2^20 random positive finite fp32 values (subnormals included) and powers of two. Bound:
    one ulp of the result plus 1.5 2^-53 (the small term's roundings); the fp32 roundings, which the
    stored metadata takes, must agree everywhere."""
    require_gpu()
    import math

    sig = (np.arange(1 << 23, dtype=np.uint32) | np.uint32(0x3F800000)).view(np.float32).astype(np.float64)
    rng = np.random.default_rng(8)
    bits = rng.integers(1, 0x7F800000, 1 << 20, dtype=np.uint32)
    x = np.concatenate([sig * 2.0**-20, sig * 0.5, sig, bits.view(np.float32).astype(np.float64),
                        np.exp2(np.arange(-149.0, 128.0))])
    got = _run(8, x)
    ref = np.array([math.log2(v) for v in x])
    err = np.abs(got - ref)
    bound = np.spacing(np.abs(ref)) + 1.5 * 2.0**-53
    worst = float((err / bound).max())
    ndiff = int(np.count_nonzero(got != ref))
    log(f"fit log2: {ndiff} of {x.size:,} differ from the host's (largest error {worst:.3f} of the bound)")
    assert worst <= 1.0
    assert np.array_equal(got.astype(np.float32), ref.astype(np.float32))
    p2 = np.exp2(np.arange(-149.0, 128.0))
    assert np.array_equal(_run(8, p2), np.arange(-149.0, 128.0))  # exact at powers of two


def _fp32_cover():
    """Every fp32 significand (x in [1, 2)), the same significands at the ends of the fp32 range
    (subnormals included, as values), and 2^20 random positive finite fp32 bit patterns."""
    sig = (np.arange(1 << 23, dtype=np.uint32) | np.uint32(0x3F800000)).view(np.float32).astype(np.float64)
    rng = np.random.default_rng(3)
    bits = rng.integers(1, 0x7F800000, 1 << 20, dtype=np.uint32)
    rnd = bits.view(np.float32).astype(np.float64)
    ends = np.concatenate([sig[::97] * 2.0**-149, sig[::89] * 2.0**-127, sig[::83] * 2.0**127])
    return np.concatenate([sig, rnd, ends, [2.0**-149, float(np.finfo(np.float32).max)]])


def test_uf8_division_free_quotients_are_correctly_rounded():
    """x / 127 (UF8 decode step) and 127 / x (encode scale) without the binary64 division equal the
    IEEE quotients bit for bit; scaling x by 2^k scales every step exactly, so the significands of
    [1, 2) cover every fp32 input (the range ends and random patterns check that)."""
    require_gpu()
    x = _fp32_cover()
    q = _run(5, x)
    assert np.array_equal(q, x / 127.0), np.count_nonzero(q != x / 127.0)
    assert np.array_equal(_run(5, -x), -x / 127.0)
    assert _run(5, np.zeros(1))[0] == 0.0
    r = _run(6, x)
    assert np.array_equal(r, 127.0 / x), np.count_nonzero(r != 127.0 / x)
    log(f"x/127 and 127/x exact over {x.size:,} fp32 inputs")


def test_clipped_quotient_matches_division():
    """fl32(x / d) from fl64(x * fl64(1/d)) with the fallback test (the clipped updates of the factored
    steps) equals (float)(x / d) bit for bit: random magnitudes across the fp32 range (subnormal and
    overflowing quotients included) and quotients placed on and beside fp32 rounding midpoints."""
    require_gpu()
    rng = np.random.default_rng(4)
    wide = np.exp2(rng.uniform(-160.0, 130.0, 1 << 20)) * rng.choice([-1.0, 1.0], 1 << 20)
    f = rng.integers(1, 0x7F000000, 1 << 19, dtype=np.uint32).view(np.float32).astype(np.float64)
    nxt = np.nextafter(f.astype(np.float32), np.float32(np.inf)).astype(np.float64)
    mid = (f + nxt) / 2.0  # exact in binary64
    near = np.concatenate([mid * 3.0, np.nextafter(mid * 3.0, np.inf), np.nextafter(mid * 3.0, -np.inf)])
    sub = np.exp2(rng.uniform(-150.0, -124.0, 1 << 18)) * 3.0
    x = np.concatenate([wide, near, sub, [0.0, -0.0, 3.0 * 2.0**-126, 3.0 * (2.0**-126 - 2.0**-150)]])
    got = _run(7, x).astype(np.float32)
    with np.errstate(over="ignore"):
        ref = (x / 3.0).astype(np.float32)
    bad = np.count_nonzero(got.view(np.uint32) != ref.view(np.uint32))
    log(f"clipped quotient: {x.size:,} inputs, {bad} differences")
    assert bad == 0


def test_folded_clipped_quotient_matches_division():
    """The CAME passes' clipped update: q = fl64(fl64(fl64(r * fl64(1/d)) * c) * x) with the decision test over
    eight quotients at a time (two unsigned minima) and the exact fl32(fl64(fl64(r c) x) / d) for the whole
    group when any rounding is undecided, against that division on the host bit for bit. Groups of eight
    normal-range quotients (the fast path), groups with one quotient on or beside an fp32 rounding midpoint
    among seven normal ones, and groups of random magnitudes across the fp32 range (subnormal, underflowing
    and overflowing quotients) with zeros of both signs."""
    require_gpu()
    r, c, d = 0.7310585786300049, 1234.5678901234567, 3.0000000000000004  # the kernel's constants
    rc = r * c
    rng = np.random.default_rng(9)

    def normal(k):
        return np.exp2(rng.uniform(-100.0, 100.0, k)) * rng.choice([-1.0, 1.0], k) * d / rc

    plain = normal(1 << 20)
    f = rng.integers(0x00800000, 0x7F000000, 3 << 16, dtype=np.uint32).view(np.float32).astype(np.float64)
    nxt = np.nextafter(f.astype(np.float32), np.float32(np.inf)).astype(np.float64)
    xm = (f + nxt) / 2.0 * d / rc  # quotients within a few binary64 ulps of a midpoint
    near = np.concatenate([xm[: 1 << 16], np.nextafter(xm[1 << 16: 2 << 16], np.inf),
                           np.nextafter(xm[2 << 16:], -np.inf)])
    mixed = normal(8 * near.size).reshape(-1, 8)
    mixed[np.arange(near.size), rng.integers(0, 8, near.size)] = near
    wide = np.exp2(rng.uniform(-170.0, 130.0, 1 << 18)) * rng.choice([-1.0, 1.0], 1 << 18) * d / rc
    edge = np.array([0.0, -0.0, 2.0**-126 * d / rc, -(2.0**-150) * d / rc, 2.0**128 * d / rc, 1e-320, -1e-310,
                     2.0**-126 * (1 + 2.0**-20) * d / rc])
    x = np.concatenate([plain, mixed.reshape(-1), wide, edge])
    got = _run(9, x).astype(np.float32)
    with np.errstate(over="ignore", under="ignore"):
        ref = ((rc * x) / d).astype(np.float32)
    bad = np.count_nonzero(got.view(np.uint32) != ref.view(np.uint32))
    log(f"folded clipped quotient: {x.size:,} inputs, {bad} differences")
    assert bad == 0


def test_bf16_quotient_midpoint_test_alone():
    """The CAME residual pass with bf16 gradients drops the range test when r_i / clip * min_j c_j >=
    2^7 (1 + 2^-18): every nonzero bf16 has |g| >= 2^-133, so each quotient is zero or in the fp32 normal
    range. At a factor just above that bound (about 2^7 (1 + 2^-17)), every bf16 value (subnormal ones, whose
    quotients land just above FLT_MIN, included), in groups of eight, against the host division bit for
    bit."""
    require_gpu()
    c = float.fromhex("0x1.00008c3a4f91dp7")  # the kernel's constant, about 2^7 (1 + 2^-17)
    bits = np.arange(1 << 16, dtype=np.uint32)
    xf = (bits << 16).view(np.float32)
    x = xf[np.isfinite(xf)].astype(np.float64)
    x = np.concatenate([x, np.zeros((-x.size) % 8)])
    got = _run(10, x).astype(np.float32)
    with np.errstate(over="ignore"):
        ref = ((1.0 * c) * x / 1.0).astype(np.float32)
    assert np.all(np.abs(ref[x != 0]) >= np.float32(2.0**-126))  # the bound the pass relies on
    bad = np.count_nonzero(got.view(np.uint32) != ref.view(np.uint32))
    log(f"bf16 quotients, midpoint test alone: {x.size:,} inputs, {bad} differences")
    assert bad == 0
