"""CPU tests of the C ABI (no GPU needed): the library loads, exports every
declared symbol, rejects bad arguments with the documented status before any
HIP call, and its storage accounting reproduces the paper's numbers.
"""
import ctypes
import math
import os
import re

import pytest

import paper_2608_22322_amd as al
from paper_2608_22322_amd.workloads import tinyllama_shapes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MiB = 2.0**20
A = 1 << 20  # a 16-byte aligned fake device address (never dereferenced: validation fails first)


def _declared_symbols():
    names = set()
    for h in ("al.h", "al_synth.h"):
        txt = open(os.path.join(ROOT, "include", h)).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        names |= set(re.findall(r"\b(al_[a-z0-9_]+)\s*\(", txt))
    return names


def test_library_exports_every_declared_symbol():
    L = al.lib()
    declared = _declared_symbols()
    assert declared == set(al.EXPORTS), declared ^ set(al.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name
    assert al.version().endswith("gfx950")


# ----------------------------------------------------------------- storage (section 4.4)
def test_al8_bits_per_element():
    """Eq. al_memory: c_AL8 = 1 + 8/B bytes; 8.25 bits at B=256 and 8.031 at B=2048 (section 5)."""
    n = 2048 * 1000
    assert al.state_bytes(al.AL8, n, 256) * 8 / n == pytest.approx(8.25, abs=0)
    assert al.state_bytes(al.AL8, n, 2048) * 8 / n == pytest.approx(8.03125, abs=0)
    assert al.state_bytes(al.AL16, n, 2048) == 2 * n + 8 * (n // 2048)


def test_block_size_memory_estimates():
    """Section 5 (topology and block scale): a 1.1B-element AL8 state takes 1081.8 MiB at B=256 and
    1053.1 MiB at B=2048."""
    assert round(al.state_bytes(al.AL8, 1_100_000_000, 256) / MiB, 1) == 1081.8
    assert round(al.state_bytes(al.AL8, 1_100_000_000, 2048) / MiB, 1) == 1053.1


def test_table4_state_memory_reproduced():
    """Table 4 optimizer-state MiB on TinyLlama-1.1B, reproduced from per-tensor padded storage: 2-D tensors
    quantized, 1-D tensors' states kept FP32 (the paper's default grouping), factored vectors padded per
    vector."""
    sh = tinyllama_shapes()
    n_all = sum(s.n for s in sh)
    assert n_all == 1_100_048_384 and len(sh) == 201
    assert round(8 * n_all / MiB, 1) == 8392.7  # AdamW FP32
    ours = sum(al.state_bytes(al.UF8, s.n, 256) + al.state_bytes(al.AL8, s.n, 2048) if s.is_2d else 8 * s.n
               for s in sh)
    assert round(ours / MiB, 1) == 2119.2  # AdamW UF8 + AL8, B_V 2048
    for B, want in ((256, 1.2), (2048, 1.3)):
        af = sum(al.state_bytes(al.AL8, s.rows, B) + al.state_bytes(al.AL8, s.cols, B) if s.is_2d else 4 * s.n
                 for s in sh)
        assert round(af / MiB, 1) == want  # Adafactor AL8 factored
    assert round(sum(4 * (s.rows + s.cols) if s.is_2d else 4 * s.n for s in sh) / MiB, 1) == 3.6  # HF

    def came(vc, cc):
        tot = 0
        for s in sh:
            if s.is_2d:
                tot += al.state_bytes(al.UF8, s.n, 256)
                for L in (s.rows, s.cols):
                    tot += al.state_bytes(vc, L, 2048) + al.state_bytes(cc, L, 2048)
            else:
                tot += 8 * s.n
        return round(tot / MiB, 1)

    assert came(al.AL8, al.AL8) == 1068.0
    assert came(al.AL8, al.FP32) == 1070.3
    assert came(al.AL16, al.AL16) == 1069.8
    cf = sum(4 * s.n + 8 * (s.rows + s.cols) if s.is_2d else 8 * s.n for s in sh)
    assert round(cf / MiB, 1) == 4203.2  # CAME FP32


def test_storage_queries_reject_bad_arguments():
    assert al.code_bytes(al.AL8, -1, 256) == -1
    assert al.code_bytes(al.AL8, 10, 100) == -1
    assert al.code_bytes(9, 10, 256) == -1
    assert al.code_bytes(al.FP32, 10, 0) == 40
    assert al.meta_floats(al.UF8, 257, 256) == 2
    assert al.code_bytes(al.AL16, 257, 256) == 1024


# ----------------------------------------------------------------- validation before any HIP call
def _status(fn):
    with pytest.raises(al.ALError) as ei:
        fn()
    return ei.value.status


def _q(codec=al.AL8, x=A, n=1000, block=256, lf=-53.0, codes=A, meta=A):
    al.check(al.lib().al_quantize(codec, x, n, block, lf, codes, meta, None))


def test_quantize_validation():
    assert _status(lambda: _q(codec=al.FP32)) == 1
    assert _status(lambda: _q(codec=7)) == 1
    assert _status(lambda: _q(n=-1)) == 1
    assert _status(lambda: _q(block=100)) == 1
    assert _status(lambda: _q(block=32)) == 1
    assert _status(lambda: _q(lf=math.inf)) == 1
    assert _status(lambda: _q(x=None)) == 1
    assert _status(lambda: _q(x=A + 4)) == 2
    assert _status(lambda: _q(meta=A + 8)) == 2
    _q(n=0)  # empty input is a no-op, no HIP call
    assert "block" in al.lib().al_last_error().decode() or al.lib().al_last_error().decode() == ""


def test_dequantize_validation():
    L = al.lib()
    assert _status(lambda: al.check(L.al_dequantize(al.FP32, A, A, 10, 256, A, None))) == 1
    assert _status(lambda: al.check(L.al_dequantize(al.AL8, A, A, 10, 48, A, None))) == 1
    assert _status(lambda: al.check(L.al_dequantize(al.AL8, None, A, 10, 256, A, None))) == 1
    assert _status(lambda: al.check(L.al_dequantize(al.AL8, A, A, 10, 256, A + 2, None))) == 2
    al.check(L.al_dequantize(al.AL8, None, None, 0, 256, None, None))


def _adamw_ws(ts, cfg=None):
    arr = (al.Tensor * max(len(ts), 1))(*ts)
    cfg = cfg or al.adamw_cfg()
    out = ctypes.c_size_t(0)
    al.check(al.lib().al_adamw_workspace_bytes(arr, len(ts), ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def _adamw(ts, cfg=None, step=1, nt=None, ws=A, ws_bytes=1 << 20):
    arr = (al.Tensor * max(len(ts), 1))(*ts)
    cfg = cfg or al.adamw_cfg()
    al.check(al.lib().al_adamw_step(arr, len(ts) if nt is None else nt, ctypes.byref(cfg), step, ws, ws_bytes,
                                    None))


def _t(**kw):
    base = dict(param=A, grad=A, rows=4, cols=256, m=A, m_meta=A, v=A, v_meta=A)
    base.update(kw)
    return al.Tensor(**base)


def test_adamw_validation():
    assert _status(lambda: _adamw([_t()], step=0)) == 1
    assert _status(lambda: _adamw([_t()], nt=-1)) == 1
    assert _status(lambda: _adamw([_t(rows=-1)])) == 1
    assert _status(lambda: _adamw([_t(param=None)])) == 1
    assert _status(lambda: _adamw([_t(v_meta=None)])) == 1
    assert _status(lambda: _adamw([_t(m=A + 1)])) == 2
    assert _status(lambda: _adamw([_t(vr=A)])) == 1  # factored slot on the dense path
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(beta1=1.0))) == 1
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(lr=math.nan))) == 1
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(m=al.Spec(al.AL8, 256)))) == 1
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(v=al.Spec(al.UF8, 256)))) == 1
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(v=al.Spec(al.AL8, 96)))) == 1
    assert _status(lambda: _adamw([_t()], cfg=al.adamw_cfg(m=al.Spec(al.UF8, 128)))) == 4
    cfg = al.adamw_cfg()
    cfg.grad_dtype = 5
    assert _status(lambda: _adamw([_t()], cfg=cfg)) == 1
    # FP32 states need no metadata; empty tensors and empty lists enqueue nothing
    _adamw([_t(rows=0, param=None, grad=None, m=None, v=None, m_meta=None, v_meta=None)], ws=None, ws_bytes=0)
    _adamw([], ws=None, ws_bytes=0)
    assert "NULL" not in al.lib().al_last_error().decode()


def test_adamw_noalloc_validation():
    """The allocation-free AdamW variant validates like al_adamw_step and rejects lists beyond its fixed table of
    4096 non-empty tensors before any HIP call; empty tensors do not count."""
    L = al.lib()

    def call(ts, nt=None, cfg=None, step=1):
        arr = (al.Tensor * max(len(ts), 1))(*ts)
        cfg = cfg or al.adamw_cfg()
        al.check(L.al_adamw_step_noalloc(arr, len(ts) if nt is None else nt, ctypes.byref(cfg), step, None))

    assert _status(lambda: call([_t()], step=0)) == 1
    assert _status(lambda: call([_t(m=A + 1)])) == 2
    assert _status(lambda: call([_t()] * 4097)) == 4
    assert "4096" in L.al_last_error().decode()
    empty = _t(rows=0, param=None, grad=None, m=None, v=None, m_meta=None, v_meta=None)
    call([empty] * 5000)
    call([])


def test_adamw_workspace():
    """The workspace holds the descriptor table: 64 + 8 bytes per non-empty tensor in two 256-byte aligned
    parts; a call without it (or with too little, or misaligned) is rejected before any HIP call."""
    ts = [_t(), _t(rows=0, param=None, grad=None, m=None, v=None, m_meta=None, v_meta=None), _t(cols=512)]
    assert _adamw_ws(ts) == 256 + 256
    assert _adamw_ws([_t()] * 5) == 512 + 256
    assert _adamw_ws([_t()] * 33) == 2304 + 512  # 64 x 33 = 2112 and 8 x 33 = 264, each rounded up to 256
    assert _adamw_ws([]) == 0
    need = _adamw_ws(ts)
    assert _status(lambda: _adamw(ts, ws=None, ws_bytes=need)) == 3
    assert _status(lambda: _adamw(ts, ws=A, ws_bytes=need - 1)) == 3
    assert _status(lambda: _adamw(ts, ws=A + 16, ws_bytes=need)) == 2
    assert _status(lambda: _adamw_ws([_t(rows=-1)])) == 1


# ----------------------------------------------------------------- factored paths (Adafactor, CAME)
def _ft(rows=8, cols=256, came=False, **kw):
    """A fake 2-D (rows > 1) or 1-D tensor with the slots the factored paths expect."""
    base = dict(param=A, grad=A, rows=rows, cols=cols)
    if rows > 1:
        base.update(vr=A, vr_meta=A, vc=A, vc_meta=A)
        if came:
            base.update(cr=A, cr_meta=A, cc=A, cc_meta=A)
    else:
        base.update(v=A, v_meta=A)
    if came:
        base.update(m=A, m_meta=A)
    base.update(kw)
    return al.Tensor(**base)


def _fac_ws(ts, came, cfg=None):
    arr = (al.Tensor * max(len(ts), 1))(*ts)
    out = ctypes.c_size_t(0)
    if came:
        cfg = cfg or al.came_cfg()
        al.check(al.lib().al_came_workspace_bytes(arr, len(ts), ctypes.byref(cfg), ctypes.byref(out)))
    else:
        cfg = cfg or al.adafactor_cfg()
        al.check(al.lib().al_adafactor_workspace_bytes(arr, len(ts), ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def _fac_step(ts, came, cfg=None, step=1, ws=A, ws_bytes=None, nt=None):
    arr = (al.Tensor * max(len(ts), 1))(*ts)
    if ws_bytes is None:
        ws_bytes = _fac_ws(ts, came, cfg) if ts else 0
    n = len(ts) if nt is None else nt
    if came:
        cfg = cfg or al.came_cfg()
        al.check(al.lib().al_came_step(arr, n, ctypes.byref(cfg), step, ws, ws_bytes, None))
    else:
        cfg = cfg or al.adafactor_cfg()
        al.check(al.lib().al_adafactor_step(arr, n, ctypes.byref(cfg), step, ws, ws_bytes, None))


@pytest.mark.parametrize("came", [False, True])
def test_factored_validation_shapes_and_slots(came):
    good = [_ft(came=came), _ft(rows=1, cols=512, came=came)]
    assert _status(lambda: _fac_step(good, came, step=0)) == 1
    assert _status(lambda: _fac_step(good, came, nt=-1)) == 1
    assert _status(lambda: _fac_step([_ft(rows=-2, came=came)], came, ws_bytes=1 << 20)) == 1
    assert _status(lambda: _fac_step([_ft(came=came, param=None)], came, ws_bytes=1 << 20)) == 1
    assert _status(lambda: _fac_step([_ft(came=came, grad=A + 2)], came, ws_bytes=1 << 20)) == 2
    # a 2-D tensor needs its row and column factors and must not carry an unfactored v
    assert _status(lambda: _fac_step([_ft(came=came, vr=None)], came, ws_bytes=1 << 20)) == 1
    assert _status(lambda: _fac_step([_ft(came=came, vc_meta=None)], came, ws_bytes=1 << 20)) == 1
    assert _status(lambda: _fac_step([_ft(came=came, vc=A + 8)], came, ws_bytes=1 << 20)) == 2
    assert _status(lambda: _fac_step([_ft(came=came, v=A, v_meta=A)], came, ws_bytes=1 << 20)) == 1
    # a 1-D tensor keeps an unfactored v and no factors
    assert _status(lambda: _fac_step([_ft(rows=1, came=came, v=None)], came, ws_bytes=1 << 20)) == 1
    assert _status(lambda: _fac_step([_ft(rows=1, came=came, vr=A, vr_meta=A)], came, ws_bytes=1 << 20)) == 1
    if came:
        assert _status(lambda: _fac_step([_ft(came=True, cr=None)], True, ws_bytes=1 << 20)) == 1
        assert _status(lambda: _fac_step([_ft(came=True, m=None)], True, ws_bytes=1 << 20)) == 1
        assert _status(lambda: _fac_step([_ft(rows=1, came=True, cc=A, cc_meta=A)], True, ws_bytes=1 << 20)) == 1
    else:
        # Adafactor keeps no momentum and no confidence factors
        assert _status(lambda: _fac_step([_ft(m=A, m_meta=A)], False, ws_bytes=1 << 20)) == 1
        assert _status(lambda: _fac_step([_ft(cr=A, cr_meta=A)], False, ws_bytes=1 << 20)) == 1
    # empty tensors and empty lists enqueue nothing and need no workspace
    _fac_step([_ft(rows=0, cols=0, came=came, param=None, grad=None)], came, ws=None, ws_bytes=0)
    _fac_step([], came, ws=None, ws_bytes=0)


@pytest.mark.parametrize("came", [False, True])
def test_factored_validation_workspace(came):
    ts = [_ft(rows=300, cols=66, came=came), _ft(rows=1, cols=777, came=came), _ft(rows=5, cols=7, came=came)]
    need = _fac_ws(ts, came)
    assert need > 0 and need % 256 == 0
    assert _status(lambda: _fac_step(ts, came, ws=None, ws_bytes=need)) == 3
    assert _status(lambda: _fac_step(ts, came, ws_bytes=need - 1)) == 3
    assert _status(lambda: _fac_step(ts, came, ws=A + 16, ws_bytes=need)) == 2
    assert "workspace" in al.lib().al_last_error().decode()
    # the column and row partials are double-double pairs: at least n/8 bytes per factored tensor
    assert need >= (300 * 66 + 5 * 7) // 8
    assert _fac_ws(ts + [_ft(rows=64, cols=4096, came=came)], came) > need
    arr = (al.Tensor * 1)()
    cfg = al.came_cfg() if came else al.adafactor_cfg()
    fn = al.lib().al_came_workspace_bytes if came else al.lib().al_adafactor_workspace_bytes
    assert _status(lambda: al.check(fn(arr, 0, ctypes.byref(cfg), None))) == 1


def test_adafactor_cfg_validation():
    t = [_ft()]
    bad = [dict(lr=-1.0), dict(eps1=math.nan), dict(clip_threshold=0.0), dict(decay_rate=0.5),
           dict(weight_decay=-0.1)]
    for kw in bad:
        assert _status(lambda: _fac_step(t, False, cfg=al.adafactor_cfg(**kw), ws_bytes=1 << 20)) == 1, kw
    for spec in (al.Spec(al.UF8, 256), al.Spec(al.AL8, 96), al.Spec(al.AL8, 256, math.inf)):
        assert _status(lambda: _fac_step(t, False, cfg=al.adafactor_cfg(v=spec), ws_bytes=1 << 20)) == 1, spec
    cfg = al.adafactor_cfg()
    cfg.grad_dtype = 9
    assert _status(lambda: _fac_step(t, False, cfg=cfg, ws_bytes=1 << 20)) == 1
    cfg = al.adafactor_cfg()
    cfg.flags = 2  # only AL_FLAG_EXACT_SUMS (1) is defined
    assert _status(lambda: _fac_step(t, False, cfg=cfg, ws_bytes=1 << 20)) == 1
    assert al.adafactor_cfg(exact_sums=True).flags == al.FLAG_EXACT_SUMS == 1


def test_came_cfg_validation():
    t = [_ft(came=True)]
    bad = [dict(beta1=1.0), dict(beta2=-0.1), dict(beta3=1.5), dict(eps2=-1.0, conf=al.Spec(al.AL16, 128, -53.0)), dict(clip_threshold=-1.0),
           dict(lr=math.inf)]
    for kw in bad:
        assert _status(lambda: _fac_step(t, True, cfg=al.came_cfg(**kw), ws_bytes=1 << 20)) == 1, kw
    for kw in (dict(m=al.Spec(al.AL8, 256)), dict(v=al.Spec(al.UF8, 256)), dict(conf=al.Spec(al.UF8, 256)),
               dict(conf=al.Spec(al.AL16, 4096))):
        assert _status(lambda: _fac_step(t, True, cfg=al.came_cfg(**kw), ws_bytes=1 << 20)) == 1, kw
    assert _status(lambda: _fac_step(t, True, cfg=al.came_cfg(m=al.Spec(al.UF8, 128)), ws_bytes=1 << 20)) == 4
    cfg = al.came_cfg()
    cfg.flags = 3
    assert _status(lambda: _fac_step(t, True, cfg=cfg, ws_bytes=1 << 20)) == 1
    assert al.came_cfg(exact_sums=True).flags == 1


def test_tinyllama_workspace_sizes():
    """Workspace for the full TinyLlama list: descriptor table, RMS partials and per-tensor partials."""
    shapes = tinyllama_shapes()
    for came in (False, True):
        ts = [_ft(rows=s.rows, cols=s.cols, came=came) for s in shapes]
        need = _fac_ws(ts, came)
        two_d = sum(s.n for s in shapes if s.rows > 1)
        assert two_d / 8 <= need <= two_d / 8 * 1.2, (came, need)


def test_g1_grouping_reproduces_table4_adafactor_memory():
    """Section 6: G1 keeps 1-D, norm, embedding and LM-head states FP32; Table 4 lists 1.4 / 1.5 MiB of
    Adafactor state under G1 at B = 256 / 2048 (against 1.2 / 1.3 under G0)."""
    from paper_2608_22322_amd import grouping

    sh = tinyllama_shapes()
    prot = grouping.protected_flags(sh, "G1")
    names = {s.name for s, p in zip(sh, prot) if p and s.is_2d}
    assert names == {"embed", "lm_head"}
    assert all(p for s, p in zip(sh, prot) if not s.is_2d)
    for B, g0, g1 in ((256, 1.2, 1.4), (2048, 1.3, 1.5)):
        specs = {"v": al.Spec(al.AL8, B)}
        assert round(grouping.grouped_state_bytes(sh, "adafactor", specs, "G0") / MiB, 1) == g0
        assert round(grouping.grouped_state_bytes(sh, "adafactor", specs, "G1") / MiB, 1) == g1
    # the G0 AdamW and CAME rows of Table 4 through the same accounting
    assert round(grouping.grouped_state_bytes(sh, "adamw", {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL8, 2048)},
                                              "G0") / MiB, 1) == 2119.2
    assert round(grouping.grouped_state_bytes(sh, "came", {"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL16, 2048),
                                                           "conf": al.Spec(al.AL16, 2048)}, "G0") / MiB, 1) == 1069.8
    assert not any(grouping.protected_flags(sh, "G0"))
    with pytest.raises(ValueError):
        grouping.protected_flags(sh, "G2")


def test_diff_norms_validation():
    L = al.lib()
    assert _status(lambda: al.check(L.al_diff_norms(A, A, -1, A, None))) == 1
    assert _status(lambda: al.check(L.al_diff_norms(A, A, 10, None, None))) == 1
    assert _status(lambda: al.check(L.al_diff_norms(None, A, 10, A, None))) == 1
    assert _status(lambda: al.check(L.al_diff_norms(A + 4, A, 10, A, None))) == 2
    assert _status(lambda: al.check(L.al_diff_norms(A, A, 10, A + 8, None))) == 2


def test_diag_stream_validation():
    L = al.lib()
    assert _status(lambda: al.check(L.al_diag_stream(4, A, A, A, A, 4096, None))) == 1
    assert _status(lambda: al.check(L.al_diag_stream(-1, A, A, A, A, 4096, None))) == 1
    assert _status(lambda: al.check(L.al_diag_stream(0, A, A, A, A, 2047, None))) == 1
    assert _status(lambda: al.check(L.al_diag_stream(3, A, A, A, A, 2048, None))) == 1  # wide: multiple of 4096
    assert _status(lambda: al.check(L.al_diag_stream(1, None, A, A, A, 2048, None))) == 1
    assert _status(lambda: al.check(L.al_diag_stream(1, A, A, A + 4, A, 2048, None))) == 2
    assert al.lib().al_diag_stream(2, A, A, A, A, 0, None) == 0  # empty: no HIP call


# ----------------------------------------------------------------- APOLLO
def _at(rows=40, cols=96, **kw):
    base = dict(param=A, grad=A, rows=rows, cols=cols, proj=A, m=A, m_meta=A, v=A, v_meta=A, norm_state=A)
    base.update(kw)
    return al.ApolloTensor(**base)


def _ap_ws(ts, cfg=None):
    arr = (al.ApolloTensor * max(len(ts), 1))(*ts)
    return al.apollo_workspace_bytes(arr, len(ts), cfg or al.apollo_cfg(rank=64))


def _ap_step(ts, cfg=None, step=1, ws=A, ws_bytes=None, nt=None):
    cfg = cfg or al.apollo_cfg(rank=64)
    arr = (al.ApolloTensor * max(len(ts), 1))(*ts)
    if ws_bytes is None:
        ws_bytes = _ap_ws(ts, cfg) if ts else 0
    al.check(al.lib().al_apollo_step(arr, len(ts) if nt is None else nt, ctypes.byref(cfg), step, ws, ws_bytes,
                                     None))


def test_apollo_workspace_layout():
    # descriptors, then per tensor R and Rt (C x rank fp32), three C-double vectors and a 16-byte slot,
    # then the AdamW launch's descriptor table (64 + 8 bytes per tensor), each region 256-byte aligned
    def al256(x):
        return (x + 255) // 256 * 256

    C, r = 96, 64  # 40 x 96: the rows are projected, 96 channels
    per = 2 * al256(C * r * 4) + 3 * al256(C * 8) + al256(16)
    one = _ap_ws([_at()])
    assert one - per - 512 in (256, 512)  # the descriptor tables of one tensor
    two = _ap_ws([_at(), _at(rows=96, cols=40)])  # the transposed shape has the same 96 channels
    assert two - one - per in (0, 256)  # a second descriptor may spill into one more 256-byte line
    big = _ap_ws([_at(rows=5632, cols=2048)])  # 5632 channels (rows >= cols), same one-descriptor table
    assert big - one == 2 * (al256(5632 * r * 4) - al256(C * r * 4)) + 3 * (al256(5632 * 8) - al256(C * 8))
    assert _ap_ws([_at(rows=0)]) == 0 and _ap_ws([]) == 0


def test_apollo_validation():
    assert _status(lambda: _ap_step([_at()], step=0)) == 1
    assert _status(lambda: _ap_step([_at()], nt=-1)) == 1
    assert _status(lambda: _ap_step([_at(rows=-1)])) == 1
    assert _status(lambda: _ap_step([_at(proj=None)])) == 1
    assert _status(lambda: _ap_step([_at(param=A + 4)])) == 2
    assert _status(lambda: _ap_step([_at(proj=A + 8)])) == 2
    assert _status(lambda: _ap_step([_at(v_meta=None)])) == 1
    assert _status(lambda: _ap_step([_at(norm_state=None)])) == 1  # the limiter is on by default
    assert _status(lambda: _ap_step([_at()], cfg=al.apollo_cfg(rank=96))) == 1
    assert _status(lambda: _ap_step([_at()], cfg=al.apollo_cfg(rank=64, beta2=1.0))) == 1
    assert _status(lambda: _ap_step([_at()], cfg=al.apollo_cfg(rank=64, m=al.Spec(al.AL8, 256)))) == 1
    assert _status(lambda: _ap_step([_at()], cfg=al.apollo_cfg(rank=64, v=al.Spec(al.UF8, 256)))) == 1
    assert _status(lambda: _ap_step([_at()], cfg=al.apollo_cfg(rank=64, m=al.Spec(al.UF8, 512)))) == 4
    need = _ap_ws([_at()])
    assert _status(lambda: _ap_step([_at()], ws=None)) == 3
    assert _status(lambda: _ap_step([_at()], ws_bytes=need - 1)) == 3
    assert _status(lambda: _ap_step([_at()], ws=A + 16)) == 2
    cfg = al.apollo_cfg(rank=64)
    cfg.grad_dtype = 7
    assert _status(lambda: _ap_step([_at()], cfg=cfg)) == 1
    # empty tensors and empty lists enqueue nothing
    _ap_step([_at(rows=0, param=None, grad=None, proj=None, m=None, v=None, m_meta=None, v_meta=None)])
    _ap_step([])


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus 2 exits with status 2 and says why, before touching a GPU."""
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
