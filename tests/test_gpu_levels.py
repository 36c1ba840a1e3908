"""The fused AdamW step's split-table AL8 decode (section 4.1, Eq. al_dequant),
measured level by level through al_diag_levels, which evaluates the step
kernel's own table functions.

For random blocks (l_min over the optimizers' floors and beyond, delta from
2^-8 to 90 bits) every positive level q = 1..255 is decoded through the two-
factor tables (AL8 blocks of 128 and more) and the three-factor tables (blocks
of 64), and compared with
* 2^E in extended precision, E = l32 + (q - 1) delta32 / 254: the binary64
  value must lie within (ln 2 (|l32| + 3 (q - 1) st) + c) 2^-53 relative of
  it, st = delta32 / 254 (the binary64 roundings of st and of the factors'
  arguments, which grow with their size, and of the evaluations and products;
  c = 5 for two factors, 7 for three);
* the oracle's level fl32(exp2(E)): the fp32 roundings must agree, except
  where 2^E lies within that bound of an fp32 rounding midpoint (then the two
  differ by one fp32 ulp).
"""
import math

import numpy as np
import pytest

import oracle

from .gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

U = 2.0**-53


def _blocks(nb, seed):
    rng = np.random.default_rng(seed)
    lmin = rng.uniform(-110.0, 40.0, nb).astype(np.float32)
    delta = np.exp2(rng.uniform(-8.0, math.log2(90.0), nb)).astype(np.float32)
    return lmin, delta


@pytest.mark.parametrize("kind,c", [(0, 5.0), (1, 7.0)])
def test_split_table_levels(kind, c):
    require_gpu()
    import torch

    import paper_2608_22322_amd as al

    nb = 20000
    lmin, delta = _blocks(nb, 311 + kind)
    meta = np.stack([lmin, delta], axis=1).reshape(-1)
    md = torch.from_numpy(meta).cuda()
    out = torch.empty(nb * 255, dtype=torch.float64, device="cuda")
    al.diag_levels(kind, md, nb, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(nb, 255)

    # extended-precision reference (x87 long double: 64-bit significand)
    q1 = np.arange(255, dtype=np.longdouble)  # q - 1
    st = delta.astype(np.longdouble) / 254
    E = lmin.astype(np.longdouble)[:, None] + q1[None, :] * st[:, None]
    ref = np.exp2(E)
    rel = np.abs((got.astype(np.longdouble) - ref) / ref).astype(np.float64)
    bound = (math.log(2.0) * (np.abs(lmin.astype(np.float64))[:, None] + 3.0 * q1.astype(np.float64)[None, :] *
                              st.astype(np.float64)[:, None]) + c) * U
    worst = float((rel / bound).max())
    log(f"kind {kind}: max relative error {rel.max() / U:.1f} x 2^-53 "
        f"(largest fraction of the bound {worst:.3f}) over {nb * 255:,} levels")
    assert worst <= 1.0

    # fp32 levels against the oracle's fl32(exp2(E))
    # the oracle decodes blocks of 256 codes: code 0 (exact zero) then 1..255
    codes = np.tile(np.arange(256, dtype=np.uint8), nb)
    orc = oracle.al_dequantize(8, codes, meta, nb * 256, 256).reshape(nb, 256)[:, 1:]
    g32 = got.astype(np.float32)
    diff = g32 != orc
    n_diff = int(diff.sum())
    if n_diff:
        # each difference: fp32 neighbours, with 2^E within the bound of the midpoint between them
        a, b = g32[diff], orc[diff]
        assert np.array_equal(np.nextafter(a, b), b), "a level differs by more than one fp32 ulp"
        mid = (a.astype(np.longdouble) + b.astype(np.longdouble)) / 2
        dist = np.abs((ref[diff] - mid) / ref[diff]).astype(np.float64)
        assert np.all(dist <= 2 * bound[diff]), "a level differs away from an fp32 midpoint"
    log(f"kind {kind}: {n_diff} of {nb * 255:,} fp32 levels differ from the oracle's (each at an fp32 midpoint)")
    assert n_diff <= 10
