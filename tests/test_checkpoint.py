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


def test_round_trip_exact(tmp_path):
    states, specs = _states()
    path = os.path.join(tmp_path, "opt.safetensors")
    checkpoint.save(path, states, specs, ["w0", "w1"], "came", 17)
    fresh = [al.ParamState(None, None, s.rows, s.cols) for s in states]
    kind, step, got_specs = checkpoint.load(path, fresh, device="cpu")
    assert (kind, step) == ("came", 17)
    for s, f, sp, gsp in zip(states, fresh, specs, got_specs):
        assert set(gsp) == set(sp)
        for role, spec in sp.items():
            assert (gsp[role].codec, gsp[role].block) == (spec.codec, spec.block)
            assert np.float32(gsp[role].log_floor) == np.float32(spec.log_floor)
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
        checkpoint.load(path, [al.ParamState(None, None, 4, 2)], device="cpu")
    with pytest.raises(ValueError):
        checkpoint.load(path, [al.ParamState(None, None, 4, 2), al.ParamState(None, None, 15, 20)], device="cpu")
