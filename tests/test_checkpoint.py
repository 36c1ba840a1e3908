"""Checkpoint format and migration bookkeeping on the CPU (section 7.1: checkpoints keep the
code type and metadata and round-trip exactly). The GPU resume and migration checks are in
test_gpu_checkpoint.py."""
import os

import numpy as np
import pytest
import torch

import paper_2608_22322_amd as al
from paper_2608_22322_amd import checkpoint


def _states():
    g = torch.Generator().manual_seed(3)
    a = al.ParamState(torch.zeros(8), torch.zeros(8), 4, 2,
                      m=torch.randint(-127, 128, (256,), generator=g, dtype=torch.int8), m_meta=torch.rand(4),
                      v=torch.randint(0, 256, (2048,), generator=g, dtype=torch.uint8), v_meta=torch.rand(4))
    b = al.ParamState(torch.zeros(300), torch.zeros(300), 20, 15,
                      m=torch.randint(-127, 128, (512,), generator=g, dtype=torch.int8), m_meta=torch.rand(4),
                      vr=torch.randint(-32768, 32767, (128,), generator=g, dtype=torch.int16), vr_meta=torch.rand(4),
                      vc=torch.rand(15), vc_meta=None)
    specs = [{"m": al.Spec(al.UF8, 256), "v": al.Spec(al.AL8, 2048, -53.15)},
             {"m": al.Spec(al.UF8, 256), "vr": al.Spec(al.AL16, 128, -99.66), "vc": al.Spec(al.FP32)}]
    return [a, b], specs


def _fresh(states):
    """The same tensors with zeroed state buffers of the same layout."""
    out = []
    for s in states:
        f = al.ParamState(None, None, s.rows, s.cols)
        for role in checkpoint.ROLES:
            for attr in (role, role + "_meta"):
                buf = getattr(s, attr)
                if buf is not None:
                    setattr(f, attr, torch.zeros_like(buf))
        out.append(f)
    return out


def test_round_trip_exact(tmp_path):
    states, specs = _states()
    path = os.path.join(tmp_path, "opt.safetensors")
    checkpoint.save(path, states, specs, ["w0", "w1"], "came", 17)
    fresh = _fresh(states)
    before = {(i, a): getattr(f, a) for i, f in enumerate(fresh) for a in ("m", "m_meta", "v", "vr", "vc")}
    assert checkpoint.load(path, fresh, specs, kind="came") == ("came", 17)
    for (i, a), buf in before.items():
        assert getattr(fresh[i], a) is buf  # loaded in place: arrays built over the buffers stay valid
    for s, f, sp in zip(states, fresh, specs):
        for role in sp:
            a, b = getattr(s, role), getattr(f, role)
            assert a.dtype == b.dtype and torch.equal(a, b)
            ma, mb = getattr(s, role + "_meta"), getattr(f, role + "_meta")
            assert (ma is None) == (mb is None)
            if ma is not None:
                assert torch.equal(ma, mb)


def test_load_rejects_other_shapes(tmp_path):
    states, specs = _states()
    path = os.path.join(tmp_path, "opt.safetensors")
    checkpoint.save(path, states, specs, ["w0", "w1"], "adamw", 1)
    with pytest.raises(ValueError):
        checkpoint.load(path, _fresh(states)[:1], specs[:1])
    swapped = [al.ParamState(None, None, 4, 2), al.ParamState(None, None, 15, 20)]
    with pytest.raises(ValueError):
        checkpoint.load(path, swapped, specs)


def test_load_rejects_other_codes_and_layouts(tmp_path):
    """A checkpoint is loaded only into states of the same codes: another block size (whose code and metadata
    arrays the kernels would index differently), codec or floor, a missing or differently sized buffer, a
    different dtype or optimizer kind are rejected before anything is overwritten."""
    states, specs = _states()
    path = os.path.join(tmp_path, "opt.safetensors")
    checkpoint.save(path, states, specs, ["w0", "w1"], "came", 3)

    def rejects(fresh, sp, kind=None):
        snap = [{a: getattr(f, a).clone() for a in ("m", "m_meta") if getattr(f, a) is not None} for f in fresh]
        with pytest.raises(ValueError):
            checkpoint.load(path, fresh, sp, kind=kind)
        for f, sn in zip(fresh, snap):  # nothing overwritten
            for a, v in sn.items():
                assert torch.equal(getattr(f, a), v)

    other_block = [dict(specs[0], v=al.Spec(al.AL8, 256, -53.15)), specs[1]]
    rejects(_fresh(states), other_block)
    rejects(_fresh(states), [dict(specs[0], v=al.Spec(al.AL16, 2048, -53.15)), specs[1]])
    rejects(_fresh(states), [dict(specs[0], v=al.Spec(al.AL8, 2048, -50.0)), specs[1]])
    rejects(_fresh(states), [{"m": specs[0]["m"]}, specs[1]])  # a role missing from the expected set
    rejects(_fresh(states), specs, kind="adamw")
    f = _fresh(states)
    f[1].vc = None
    rejects(f, specs)
    f = _fresh(states)
    f[0].v = torch.zeros(1024, dtype=torch.uint8)  # too short for B_V 2048 codes
    rejects(f, specs)
    f = _fresh(states)
    f[0].m = torch.zeros(256, dtype=torch.uint8)  # UF8 codes are int8
    rejects(f, specs)
    assert checkpoint.load(path, _fresh(states), specs) == ("came", 3)
