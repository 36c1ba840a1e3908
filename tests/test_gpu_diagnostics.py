"""GPU checks of the update-error diagnostic (section 3.2, Eq. update_error) and of
al_diff_norms: E_upd from the library's kernels against E_upd computed by the oracle's
steps on the same states and gradient; invariants (FP32 codes give 0; states that are
already code levels give ~0)."""
import math

import numpy as np
import pytest

import oracle
from paper_2608_22322_amd import synth

from .gpu_util import log, require_gpu

pytestmark = pytest.mark.gpu

V_FLOOR = float(np.float32(2 * math.log2(1e-8)))


@pytest.fixture(scope="module")
def dev():
    require_gpu()
    import torch

    return torch.device("cuda:0")


def test_diff_norms_matches_fsum(dev):
    import torch

    import paper_2608_22322_amd as al

    for n in (0, 1, 1000, 300_001, 5_000_000):
        a = synth.normal_f32(synth.grad_key(1, n % 97), n, 1e-2) if n else np.zeros(0, np.float32)
        b = synth.normal_f32(synth.grad_key(2, n % 89), n, 1e-2) if n else np.zeros(0, np.float32)
        ad = torch.from_numpy(np.concatenate([a, np.zeros(4, np.float32)])).to(dev)
        bd = torch.from_numpy(np.concatenate([b, np.zeros(4, np.float32)])).to(dev)
        out = torch.zeros(al.DIFF_NORMS_OUT, dtype=torch.float64, device=dev)
        al.diff_norms(ad[:n], bd[:n], out)
        got = out[:2].cpu().numpy()
        d = a.astype(np.float64) - b.astype(np.float64)
        want = (math.fsum((d * d).tolist()), math.fsum((b.astype(np.float64) ** 2).tolist()))
        for k in range(2):
            assert got[k] == want[k] or abs(got[k] - want[k]) <= 2 ** -52 * abs(want[k]), (n, k, got[k], want[k])


def _adamw_states(dev, n, seed):
    import torch

    import paper_2608_22322_amd as al

    m = synth.normal_f32(synth.grad_key(seed, 1), n, 1e-4)
    v = np.abs(synth.normal_f32(synth.grad_key(seed, 2), n, 1e-6)).astype(np.float32)
    v[synth.normal_f32(synth.grad_key(seed, 3), n, 1.0) > 2.0] = 0.0  # some dormant entries
    m[v == 0] = 0.0
    g = synth.normal_f32(synth.grad_key(seed, 4), n, 1e-3)
    pad = lambda x: torch.from_numpy(np.concatenate([x, np.zeros(8, np.float32)])).to(dev)
    st = al.ParamState(None, pad(g), 1, n, m=pad(m), v=pad(v))
    return st, m, v, g


def _oracle_adamw_error(m, v, g, mspec, vspec, t):
    n = m.shape[0]
    pr, pq = np.zeros(n, np.float32), np.zeros(n, np.float32)
    mr, vr = oracle.State(oracle.FP32, n), oracle.State(oracle.FP32, n)
    mr.codes[:], vr.codes[:] = m, v
    oracle.adamw_step(pr, g, mr, vr, t)
    mq = oracle.State(mspec.codec, n, mspec.block)
    vq = oracle.State(vspec.codec, n, vspec.block, vspec.log_floor)
    mq.codes[:], mq.meta[:], _ = oracle.uf8_quantize(m, mspec.block)
    vq.codes[:], vq.meta[:], _ = oracle.al_quantize(8, v, vspec.block, vspec.log_floor)
    oracle.adamw_step(pq, g, mq, vq, t)
    d = pq.astype(np.float64) - pr.astype(np.float64)
    return math.sqrt(math.fsum((d * d).tolist())) / math.sqrt(math.fsum((pr.astype(np.float64) ** 2).tolist()))


@pytest.mark.parametrize("block", [256, 2048])
def test_adamw_update_error_matches_oracle(dev, block):
    import paper_2608_22322_amd as al
    from paper_2608_22322_amd.diagnostics import update_error

    n = 8 * 2048 + 300
    st, m, v, g = _adamw_states(dev, n, 11)
    mspec, vspec = al.Spec(al.UF8, 256), al.Spec(al.AL8, block, V_FLOOR)
    cfg = al.adamw_cfg(grad_bf16=False, m=mspec, v=vspec, weight_decay=0.0)
    e = update_error("adamw", [st], cfg, t=10)
    e_orc = _oracle_adamw_error(m, v, g, mspec, vspec, 10)
    log(f"AdamW B_V {block}: E_upd GPU {e:.6e} oracle {e_orc:.6e}")
    assert 1e-6 < e < 0.2
    assert abs(e - e_orc) <= 1e-3 * e_orc + 1e-7
    # FP32 codes reproduce the reference exactly
    cfg32 = al.adamw_cfg(grad_bf16=False, m=al.Spec(al.FP32), v=al.Spec(al.FP32), weight_decay=0.0)
    assert update_error("adamw", [st], cfg32, t=10) == 0.0


def test_update_error_of_code_levels_is_negligible(dev):
    """States that already sit on code levels re-encode to the same codes: E_upd ~ 0."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd.diagnostics import update_error

    n = 4 * 2048
    st, m, v, g = _adamw_states(dev, n, 13)
    mspec, vspec = al.Spec(al.UF8, 256), al.Spec(al.AL8, 256, V_FLOOR)
    for buf, spec in ((st.m, mspec), (st.v, vspec)):
        codes, meta = al.alloc_state(n, spec, dev)
        al.quantize(spec.codec, buf[:n], spec.block, spec.log_floor, codes, meta)
        al.dequantize(spec.codec, codes, meta, n, spec.block, buf)
    torch.cuda.synchronize()
    cfg = al.adamw_cfg(grad_bf16=False, m=mspec, v=vspec, weight_decay=0.0)
    e = update_error("adamw", [st], cfg, t=10)
    log(f"E_upd of code levels: {e:.3e}")
    assert e < 1e-5


def test_factored_update_error_ordering(dev):
    """Adafactor with AL16 factors has a far smaller update error than with AL8 (section 5 reports
    AL16 as near lossless); qualitative, parity unpinned."""
    import torch

    import paper_2608_22322_amd as al
    from paper_2608_22322_amd.diagnostics import update_error

    rows, cols = 96, 512
    g = synth.normal_f32(synth.grad_key(21, 1), rows * cols, 1e-3)
    R = np.abs(synth.normal_f32(synth.grad_key(21, 2), rows, 1e-6)).astype(np.float32) + np.float32(1e-7)
    C = np.abs(synth.normal_f32(synth.grad_key(21, 3), cols, 1e-6)).astype(np.float32) + np.float32(1e-7)
    pad = lambda x: torch.from_numpy(np.concatenate([x, np.zeros(8, np.float32)])).to(dev)
    st = al.ParamState(None, pad(g), rows, cols, vr=pad(R), vc=pad(C))
    floor = float(np.float32(math.log2(1e-30)))
    errs = {}
    for codec in (al.AL8, al.AL16):
        cfg = al.adafactor_cfg(grad_bf16=False, v=al.Spec(codec, 128, floor))
        errs[codec] = update_error("adafactor", [st], cfg, t=5)
    log(f"Adafactor E_upd: AL8 {errs[al.AL8]:.3e} AL16 {errs[al.AL16]:.3e}")
    assert 0 < errs[al.AL16] < errs[al.AL8] / 50
