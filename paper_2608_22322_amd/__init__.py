"""Python binding of libal.so, the gfx950 quantized optimizer-step library.

Argument marshalling only: every step of the optimizer and the codecs runs in
the HIP kernels behind the C ABI declared in include/al.h. PyTorch is used
for device memory and streams. There is no CPU fallback: if the library is
missing, :func:`lib` raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libal.so")

FP32, AL8, AL16, UF8 = 0, 1, 2, 3
FLAG_EXACT_SUMS = 1  # factored steps: recompute every row / column mean exactly (a check of the fast path)
DTYPE_F32, DTYPE_BF16 = 0, 1
STATUS = {0: "AL_OK", 1: "AL_EINVAL", 2: "AL_EALIGN", 3: "AL_EWORKSPACE", 4: "AL_EUNSUPPORTED", 5: "AL_EHIP"}


class ALError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class StateSpec(ctypes.Structure):
    _fields_ = [("codec", ctypes.c_int32), ("block", ctypes.c_int32), ("log_floor", ctypes.c_float)]


class Tensor(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64),
                ("m", ctypes.c_void_p), ("m_meta", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("v_meta", ctypes.c_void_p),
                ("vr", ctypes.c_void_p), ("vr_meta", ctypes.c_void_p),
                ("vc", ctypes.c_void_p), ("vc_meta", ctypes.c_void_p),
                ("cr", ctypes.c_void_p), ("cr_meta", ctypes.c_void_p),
                ("cc", ctypes.c_void_p), ("cc_meta", ctypes.c_void_p)]


class AdamWCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("grad_dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("m", StateSpec), ("v", StateSpec)]


class AdafactorCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("eps1", ctypes.c_double), ("clip_threshold", ctypes.c_double),
                ("decay_rate", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("grad_dtype", ctypes.c_int32), ("flags", ctypes.c_int32), ("v", StateSpec)]


class CAMECfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("beta3", ctypes.c_double), ("eps1", ctypes.c_double), ("eps2", ctypes.c_double),
                ("clip_threshold", ctypes.c_double), ("weight_decay", ctypes.c_double),
                ("grad_dtype", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("m", StateSpec), ("v", StateSpec), ("conf", StateSpec)]


class ApolloTensor(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64), ("proj", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("m_meta", ctypes.c_void_p), ("v", ctypes.c_void_p), ("v_meta", ctypes.c_void_p),
                ("norm_state", ctypes.c_void_p)]


class ApolloCfg(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double), ("gamma", ctypes.c_double),
                ("rank", ctypes.c_int32), ("grad_dtype", ctypes.c_int32), ("m", StateSpec), ("v", StateSpec)]


_lib = None

# every symbol include/al.h and include/al_synth.h declare
EXPORTS = ("al_version", "al_last_error", "al_code_bytes", "al_meta_floats", "al_state_bytes", "al_quantize",
           "al_dequantize", "al_adamw_workspace_bytes", "al_adamw_step", "al_adamw_step_noalloc",
           "al_adafactor_workspace_bytes", "al_came_workspace_bytes",
           "al_adafactor_step", "al_came_step", "al_apollo_workspace_bytes", "al_apollo_step", "al_diag_math",
           "al_diag_levels", "al_diag_stream", "al_diff_norms", "al_synth_normal")


def lib():
    """Load libal.so (built in-tree by build.py). Raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2608_22322_amd/build.py "
                               "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, f, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
        u64 = ctypes.c_uint64
        L.al_version.restype = ctypes.c_char_p
        L.al_last_error.restype = ctypes.c_char_p
        for name in ("al_code_bytes", "al_meta_floats", "al_state_bytes"):
            getattr(L, name).argtypes = [i32, i64, i32]
            getattr(L, name).restype = i64
        L.al_quantize.argtypes = [i32, vp, i64, i32, f, vp, vp, vp]
        L.al_dequantize.argtypes = [i32, vp, vp, i64, i32, vp, vp]
        L.al_adamw_workspace_bytes.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(AdamWCfg),
                                               ctypes.POINTER(sz)]
        L.al_adamw_step.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(AdamWCfg), i64, vp, sz, vp]
        L.al_adamw_step_noalloc.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(AdamWCfg), i64, vp]
        L.al_adafactor_workspace_bytes.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(AdafactorCfg),
                                                   ctypes.POINTER(sz)]
        L.al_came_workspace_bytes.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(CAMECfg),
                                              ctypes.POINTER(sz)]
        L.al_adafactor_step.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(AdafactorCfg), i64, vp, sz, vp]
        L.al_came_step.argtypes = [ctypes.POINTER(Tensor), i32, ctypes.POINTER(CAMECfg), i64, vp, sz, vp]
        L.al_apollo_workspace_bytes.argtypes = [ctypes.POINTER(ApolloTensor), i32, ctypes.POINTER(ApolloCfg),
                                                ctypes.POINTER(sz)]
        L.al_apollo_step.argtypes = [ctypes.POINTER(ApolloTensor), i32, ctypes.POINTER(ApolloCfg), i64, vp, sz, vp]
        L.al_synth_normal.argtypes = [vp, i32, i64, u64, f, u64, u64, vp]
        L.al_diag_math.argtypes = [i32, vp, i64, vp, vp]
        L.al_diag_levels.argtypes = [i32, vp, i64, vp, vp]
        L.al_diag_stream.argtypes = [i32, vp, vp, vp, vp, i64, vp]
        L.al_diff_norms.argtypes = [vp, vp, i64, vp, vp]
        for name in ("al_quantize", "al_dequantize", "al_adamw_workspace_bytes", "al_adamw_step", "al_adamw_step_noalloc",
                     "al_adafactor_workspace_bytes",
                     "al_came_workspace_bytes", "al_adafactor_step", "al_came_step", "al_apollo_workspace_bytes",
                     "al_apollo_step", "al_diag_math", "al_diag_levels", "al_diag_stream",
                     "al_diff_norms", "al_synth_normal"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != 0:
        raise ALError(status, lib().al_last_error().decode())


def version() -> str:
    return lib().al_version().decode()


def code_bytes(codec: int, n: int, block: int) -> int:
    return lib().al_code_bytes(codec, n, block)


def meta_floats(codec: int, n: int, block: int) -> int:
    return lib().al_meta_floats(codec, n, block)


def state_bytes(codec: int, n: int, block: int) -> int:
    return lib().al_state_bytes(codec, n, block)


# --------------------------------------------------------------------- torch plumbing
def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def log2_floor_of(eps_squared: float) -> float:
    """l_floor as binary32: log2 of an optimizer's squared numerical floor."""
    import numpy as np

    return float(np.float32(math.log2(eps_squared)))


@dataclass
class Spec:
    codec: int
    block: int = 256
    log_floor: float = 0.0

    def c(self) -> StateSpec:
        return StateSpec(self.codec, self.block, self.log_floor)


def alloc_state(n: int, spec: Spec, device="cuda"):
    """Zeroed (codes, meta) device buffers for an n-element state (fresh state = all zero)."""
    import torch

    if spec.codec == FP32:
        return torch.zeros(max(n, 1), dtype=torch.float32, device=device), None
    dt = {AL8: torch.uint8, AL16: torch.int16, UF8: torch.int8}[spec.codec]
    nc = code_bytes(spec.codec, n, spec.block) // (2 if spec.codec == AL16 else 1)
    codes = torch.zeros(max(nc, 1), dtype=dt, device=device)
    meta = torch.zeros(max(meta_floats(spec.codec, n, spec.block), 4), dtype=torch.float32, device=device)
    return codes, meta


def quantize(codec: int, x, block: int, log_floor: float, codes, meta, stream=None) -> None:
    check(lib().al_quantize(codec, _ptr(x), x.numel(), block, log_floor, _ptr(codes), _ptr(meta), _stream(stream)))


def dequantize(codec: int, codes, meta, n: int, block: int, out, stream=None) -> None:
    check(lib().al_dequantize(codec, _ptr(codes), _ptr(meta), n, block, _ptr(out), _stream(stream)))


def diag_math(fn: int, x, out, stream=None) -> None:
    check(lib().al_diag_math(fn, _ptr(x), x.numel(), _ptr(out), _stream(stream)))


def diag_levels(kind: int, meta, nblocks: int, out, stream=None) -> None:
    """Binary64 AL8 levels of codes 1..255 per block through the step's split tables (kind 0: two factors,
    1: three factors), before the fp32 rounding."""
    check(lib().al_diag_levels(kind, _ptr(meta), nblocks, _ptr(out), _stream(stream)))


def diag_stream(nontemporal: bool, p, g, m, v, stream=None, wide: bool = False) -> None:
    """Streaming rate probe of the AdamW byte mix (al_diag_stream): the step's access shape, or with wide=True
    the fastest shape found for the mix (4096-element chunks, 16 bytes per lane from every stream)."""
    mode = (2 | 1) if wide else int(bool(nontemporal))
    check(lib().al_diag_stream(mode, _ptr(p), _ptr(g), _ptr(m), _ptr(v), p.numel(), _stream(stream)))


DIFF_NORMS_OUT = 4098  # doubles of the al_diff_norms output / scratch buffer


def diff_norms(a, b, out, stream=None) -> None:
    """out[0] = sum (a - b)^2, out[1] = sum b^2 (float32 device tensors of equal size; out: float64
    device tensor of at least DIFF_NORMS_OUT elements)."""
    if a.numel() != b.numel() or out.numel() < DIFF_NORMS_OUT:
        raise ValueError("diff_norms: sizes")
    check(lib().al_diff_norms(_ptr(a), _ptr(b), a.numel(), _ptr(out), _stream(stream)))


def synth_normal(out, key: int, sigma: float, mask_key: int = 0, mask_frac: float = 0.0, stream=None) -> None:
    """Fill a float32 or bfloat16 device tensor with the seeded generator of synth.py."""
    import torch

    from . import synth

    dt = DTYPE_BF16 if out.dtype == torch.bfloat16 else DTYPE_F32
    check(lib().al_synth_normal(_ptr(out), dt, out.numel(), key, float(synth.normal_scale(sigma)), mask_key,
                                synth.mask_threshold(mask_frac), _stream(stream)))


@dataclass
class ParamState:
    """Device buffers of one parameter tensor and its optimizer state."""
    param: object
    grad: object
    rows: int
    cols: int
    m: object = None
    m_meta: object = None
    v: object = None
    v_meta: object = None
    vr: object = None
    vr_meta: object = None
    vc: object = None
    vc_meta: object = None
    cr: object = None
    cr_meta: object = None
    cc: object = None
    cc_meta: object = None

    def c(self) -> Tensor:
        return Tensor(_ptr(self.param), _ptr(self.grad), self.rows, self.cols,
                      _ptr(self.m), _ptr(self.m_meta), _ptr(self.v), _ptr(self.v_meta),
                      _ptr(self.vr), _ptr(self.vr_meta), _ptr(self.vc), _ptr(self.vc_meta),
                      _ptr(self.cr), _ptr(self.cr_meta), _ptr(self.cc), _ptr(self.cc_meta))


def tensor_array(states) -> ctypes.Array:
    arr = (Tensor * max(len(states), 1))()
    for i, s in enumerate(states):
        arr[i] = s.c()
    return arr


def adamw_cfg(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_bf16=True,
              m: Spec | None = None, v: Spec | None = None) -> AdamWCfg:
    m = m or Spec(UF8, 256)
    v = v or Spec(AL8, 256, log2_floor_of(eps * eps))
    return AdamWCfg(lr, beta1, beta2, eps, weight_decay, DTYPE_BF16 if grad_bf16 else DTYPE_F32, 0, m.c(), v.c())


def adafactor_cfg(lr=1e-3, eps1=1e-30, clip_threshold=1.0, decay_rate=-0.8, weight_decay=0.0, grad_bf16=True,
                  v: Spec | None = None, exact_sums: bool = False) -> AdafactorCfg:
    v = v or Spec(AL8, 256, log2_floor_of(eps1))
    return AdafactorCfg(lr, eps1, clip_threshold, decay_rate, weight_decay,
                        DTYPE_BF16 if grad_bf16 else DTYPE_F32, FLAG_EXACT_SUMS if exact_sums else 0, v.c())


def came_cfg(lr=1e-4, beta1=0.9, beta2=0.999, beta3=0.9999, eps1=1e-30, eps2=1e-16, clip_threshold=1.0,
             weight_decay=0.0, grad_bf16=True, m: Spec | None = None, v: Spec | None = None,
             conf: Spec | None = None, exact_sums: bool = False) -> CAMECfg:
    m = m or Spec(UF8, 256)
    v = v or Spec(AL16, 128, log2_floor_of(eps1))
    conf = conf or Spec(AL16, 128, log2_floor_of(eps2))
    return CAMECfg(lr, beta1, beta2, beta3, eps1, eps2, clip_threshold, weight_decay,
                   DTYPE_BF16 if grad_bf16 else DTYPE_F32, FLAG_EXACT_SUMS if exact_sums else 0, m.c(), v.c(),
                   conf.c())


def adamw_workspace_bytes(states, cfg: AdamWCfg, arr=None) -> int:
    arr = arr if arr is not None else tensor_array(states)
    out = ctypes.c_size_t(0)
    check(lib().al_adamw_workspace_bytes(arr, len(states), ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def workspace(nbytes: int, device="cuda"):
    """A device workspace of nbytes (at least 256 so the pointer is never NULL; torch's allocator aligns it to
    at least 256 bytes)."""
    import torch

    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _ws_args(ws):
    return (None, 0) if ws is None else (_ptr(ws), ws.numel() * ws.element_size())


def adamw_step(states, cfg: AdamWCfg, step: int, ws, stream=None, arr=None) -> None:
    """One fused AdamW step over a list of ParamState (or a prebuilt tensor_array); ws: a device workspace of
    at least adamw_workspace_bytes (the step's descriptor table)."""
    arr = arr if arr is not None else tensor_array(states)
    check(lib().al_adamw_step(arr, len(states), ctypes.byref(cfg), step, *_ws_args(ws), _stream(stream)))


def adamw_step_noalloc(states, cfg: AdamWCfg, step: int, stream=None, arr=None) -> None:
    """al_adamw_step without a workspace (the library's fixed per-GPU table, at most 4096 tensors); for callers
    that cannot allocate. Calls that may overlap on one GPU race."""
    arr = arr if arr is not None else tensor_array(states)
    check(lib().al_adamw_step_noalloc(arr, len(states), ctypes.byref(cfg), step, _stream(stream)))


def adafactor_workspace_bytes(states, cfg: AdafactorCfg, arr=None) -> int:
    arr = arr if arr is not None else tensor_array(states)
    out = ctypes.c_size_t(0)
    check(lib().al_adafactor_workspace_bytes(arr, len(states), ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def came_workspace_bytes(states, cfg: CAMECfg, arr=None) -> int:
    arr = arr if arr is not None else tensor_array(states)
    out = ctypes.c_size_t(0)
    check(lib().al_came_workspace_bytes(arr, len(states), ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def adafactor_step(states, cfg: AdafactorCfg, step: int, ws, stream=None, arr=None) -> None:
    arr = arr if arr is not None else tensor_array(states)
    check(lib().al_adafactor_step(arr, len(states), ctypes.byref(cfg), step, *_ws_args(ws), _stream(stream)))


def came_step(states, cfg: CAMECfg, step: int, ws, stream=None, arr=None) -> None:
    arr = arr if arr is not None else tensor_array(states)
    check(lib().al_came_step(arr, len(states), ctypes.byref(cfg), step, *_ws_args(ws), _stream(stream)))


# ------------------------------------------------------------------ APOLLO (projected states)
def apollo_cfg(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, gamma=1.01, rank=256, grad_bf16=True,
               m: Spec = None, v: Spec = None) -> ApolloCfg:
    m = m or Spec(UF8, 256)
    v = v or Spec(AL8, 2048, log2_floor_of(eps * eps))
    return ApolloCfg(lr, beta1, beta2, eps, weight_decay, gamma, rank, 1 if grad_bf16 else 0, m.c(), v.c())


def apollo_tensor_array(items) -> ctypes.Array:
    """items: (param, grad, rows, cols, proj, m, m_meta, v, v_meta, norm_state) tuples of device tensors."""
    arr = (ApolloTensor * max(len(items), 1))()
    for i, (p, g, rows, cols, proj, m, mm, v, vm, ns) in enumerate(items):
        arr[i] = ApolloTensor(_ptr(p), _ptr(g), rows, cols, _ptr(proj), _ptr(m), _ptr(mm), _ptr(v), _ptr(vm),
                              _ptr(ns))
    return arr


def apollo_workspace_bytes(arr, nt: int, cfg: ApolloCfg) -> int:
    out = ctypes.c_size_t(0)
    check(lib().al_apollo_workspace_bytes(arr, nt, ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def apollo_step(arr, nt: int, cfg: ApolloCfg, step: int, ws, stream=None) -> None:
    check(lib().al_apollo_step(arr, nt, ctypes.byref(cfg), step, *_ws_args(ws), _stream(stream)))
