"""The streaming-rate diagnostic (al_diag_stream) touches every element exactly once, in both shapes.

Its outputs are fixed functions of its inputs (p.x += g0, p.w += g3 as bf16,
m ^= v, v += 1 per byte), so one call over ragged grids -- chunk counts that are
not multiples of 4 (a partly idle last workgroup) or of 32 (workgroups beyond
the XCD-ordered multiple of 8) -- shows that the workgroup -> chunk order is a
bijection: a skipped or repeated chunk leaves a byte unchanged or changed twice.
"""
import numpy as np
import pytest

from .gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("chunks", [1, 3, 8 * 4, 8 * 4 * 13 + 5, 8 * 4 * 97 + 4 * 3 + 2])
@pytest.mark.parametrize("nt", [False, True])
def test_diag_stream_covers_every_element_once(chunks, nt):
    require_gpu()
    import torch

    import paper_2608_22322_amd as al

    n = 2048 * chunks
    rng = np.random.default_rng(chunks)
    p0 = rng.standard_normal(n).astype(np.float32)
    g0 = (rng.standard_normal(n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    m0 = rng.integers(0, 256, n, dtype=np.uint8)
    v0 = rng.integers(0, 255, n, dtype=np.uint8)  # below 0xFF: the 4-byte add never carries
    p = torch.from_numpy(p0.copy()).cuda()
    g = torch.from_numpy(g0.view(np.int16).copy()).cuda()
    m = torch.from_numpy(m0.copy()).cuda()
    v = torch.from_numpy(v0.copy()).cuda()
    al.diag_stream(nt, p, g, m, v)
    torch.cuda.synchronize()
    pe = p0.copy()
    gf = (g0.astype(np.uint32) << 16).view(np.float32)
    pe[0::4] += gf[0::4]
    pe[3::4] += gf[3::4]
    log(f"diag_stream chunks={chunks} nt={nt}")
    assert np.array_equal(p.cpu().numpy().view(np.uint32), pe.view(np.uint32))
    assert np.array_equal(m.cpu().numpy(), m0 ^ v0)
    assert np.array_equal(v.cpu().numpy(), v0 + 1)


@pytest.mark.parametrize("chunks", [1, 3, 8 * 4 * 7 + 5])
def test_diag_stream_wide_shape_covers_every_element_once(chunks):
    require_gpu()
    import torch

    import paper_2608_22322_amd as al

    n = 4096 * chunks
    rng = np.random.default_rng(chunks + 1)
    p0 = rng.standard_normal(n).astype(np.float32)
    m0 = rng.integers(0, 256, n, dtype=np.uint8)
    v0 = rng.integers(0, 255, n, dtype=np.uint8)
    p = torch.from_numpy(p0.copy()).cuda()
    g = torch.zeros(n, dtype=torch.int16, device="cuda")
    m = torch.from_numpy(m0.copy()).cuda()
    v = torch.from_numpy(v0.copy()).cuda()
    al.diag_stream(True, p, g, m, v, wide=True)
    torch.cuda.synchronize()
    log(f"diag_stream wide chunks={chunks}")
    assert np.array_equal(p.cpu().numpy(), p0 + np.float32(1.0))
    assert np.array_equal(m.cpu().numpy(), m0 ^ v0)
    assert np.array_equal(v.cpu().numpy(), v0 + 1)
