"""TEST INFRASTRUCTURE -- the CPU oracle. Not part of the product path.

A ctypes wrapper over ``liboracle.so`` (plain binary64 C in ``al_oracle.c``).
Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package. It shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "al_oracle.c")

FP32, AL8, AL16, UF8 = 0, 1, 2, 3
BITS = {AL8: 8, AL16: 16}
CODE_DTYPE = {FP32: np.float32, AL8: np.uint8, AL16: np.uint16, UF8: np.int8}


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc: binary64, no contraction, no fast-math."""
    if force or not os.path.exists(_LIB_PATH):
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


class Spec(ctypes.Structure):
    _fields_ = [("codec", ctypes.c_int32), ("block", ctypes.c_int32), ("log_floor", ctypes.c_float)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32, d, f = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_float
        L.orc_exact_sum.argtypes = [vp, i64]
        L.orc_exact_sum.restype = d
        L.orc_al_quantize.argtypes = [i32, vp, i64, i32, f, vp, vp, vp]
        L.orc_al_dequantize.argtypes = [i32, vp, vp, i64, i32, vp]
        L.orc_uf8_quantize.argtypes = [vp, i64, i32, vp, vp, vp]
        L.orc_uf8_dequantize.argtypes = [vp, vp, i64, i32, vp]
        L.orc_state_decode.argtypes = [Spec, vp, vp, i64, vp]
        L.orc_state_encode.argtypes = [Spec, vp, i64, vp, vp, vp]
        L.orc_adamw_step.argtypes = [i64, vp, vp, i32, d, d, d, d, d, i64, Spec, vp, vp, Spec, vp, vp, vp, vp]
        L.orc_adafactor_step.argtypes = [i64, i64, vp, vp, i32, d, d, d, d, d, i64, Spec,
                                         vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_came_step.argtypes = [i64, i64, vp, vp, i32, d, d, d, d, d, d, d, d, i64,
                                    Spec, Spec, Spec, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                    vp, vp, vp, vp, vp, vp]
        for name in ("orc_al_quantize", "orc_al_dequantize", "orc_uf8_quantize", "orc_uf8_dequantize",
                     "orc_state_decode", "orc_state_encode", "orc_adamw_step", "orc_adafactor_step",
                     "orc_came_step"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def nblocks(n: int, block: int) -> int:
    return (n + block - 1) // block


def meta_len(codec: int, n: int, block: int) -> int:
    if codec == FP32:
        return 0
    return nblocks(n, block) * (1 if codec == UF8 else 2)


def code_len(codec: int, n: int, block: int) -> int:
    return n if codec == FP32 else nblocks(n, block) * block


class State:
    """One optimizer state (codes + metadata) in host memory under a spec."""

    def __init__(self, codec: int, n: int, block: int = 256, log_floor: float = 0.0):
        self.codec, self.n, self.block = codec, n, block
        self.log_floor = float(np.float32(log_floor))
        self.codes = np.zeros(code_len(codec, n, block), dtype=CODE_DTYPE[codec])
        self.meta = np.zeros(max(meta_len(codec, n, block), 1), dtype=np.float32)
        self.y = np.full(n, np.nan)

    @property
    def spec(self) -> Spec:
        return Spec(self.codec, self.block, self.log_floor)

    def copy(self) -> "State":
        s = State.__new__(State)
        s.codec, s.n, s.block, s.log_floor = self.codec, self.n, self.block, self.log_floor
        s.codes, s.meta, s.y = self.codes.copy(), self.meta.copy(), self.y.copy()
        return s

    def decode(self) -> np.ndarray:
        out = np.empty(self.n, dtype=np.float32)
        _check(lib().orc_state_decode(self.spec, _p(self.codes), _p(self.meta), self.n, _p(out)), "decode")
        return out

    def encode(self, x: np.ndarray) -> None:
        x = np.ascontiguousarray(x, dtype=np.float32)
        _check(lib().orc_state_encode(self.spec, _p(x), self.n, _p(self.codes), _p(self.meta), _p(self.y)),
               "encode")


def exact_sum(x) -> float:
    x = np.ascontiguousarray(x, dtype=np.float64)
    return lib().orc_exact_sum(_p(x), x.shape[0])


def al_quantize(bits: int, x, block: int, log_floor: float):
    x = np.ascontiguousarray(x, dtype=np.float32)
    n = x.shape[0]
    codes = np.zeros(nblocks(n, block) * block, dtype=np.uint8 if bits == 8 else np.uint16)
    meta = np.zeros(max(2 * nblocks(n, block), 1), dtype=np.float32)
    y = np.full(n, np.nan)
    _check(lib().orc_al_quantize(bits, _p(x), n, block, float(log_floor), _p(codes), _p(meta), _p(y)),
           "al_quantize")
    return codes, meta[:2 * nblocks(n, block)], y


def al_dequantize(bits: int, codes, meta, n: int, block: int):
    codes = np.ascontiguousarray(codes, dtype=np.uint8 if bits == 8 else np.uint16)
    meta = np.ascontiguousarray(meta, dtype=np.float32)
    out = np.empty(n, dtype=np.float32)
    _check(lib().orc_al_dequantize(bits, _p(codes), _p(meta), n, block, _p(out)), "al_dequantize")
    return out


def uf8_quantize(x, block: int = 256):
    x = np.ascontiguousarray(x, dtype=np.float32)
    n = x.shape[0]
    codes = np.zeros(nblocks(n, block) * block, dtype=np.int8)
    meta = np.zeros(max(nblocks(n, block), 1), dtype=np.float32)
    y = np.full(n, np.nan)
    _check(lib().orc_uf8_quantize(_p(x), n, block, _p(codes), _p(meta), _p(y)), "uf8_quantize")
    return codes, meta[:nblocks(n, block)], y


def uf8_dequantize(codes, meta, n: int, block: int = 256):
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    meta = np.ascontiguousarray(meta, dtype=np.float32)
    out = np.empty(n, dtype=np.float32)
    _check(lib().orc_uf8_dequantize(_p(codes), _p(meta), n, block, _p(out)), "uf8_dequantize")
    return out


def _grad(g):
    g = np.ascontiguousarray(g)
    if g.dtype == np.uint16:
        return g, 1
    return np.ascontiguousarray(g, dtype=np.float32), 0


def adamw_step(p, g, m: State, v: State, t: int, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01):
    """One AdamW step on one tensor, in place. g: float32 array or uint16 bf16 bits."""
    assert p.dtype == np.float32 and p.flags.c_contiguous
    g, gb = _grad(g)
    _check(lib().orc_adamw_step(p.shape[0], _p(p), _p(g), gb, lr, beta1, beta2, eps, wd, t,
                                m.spec, _p(m.codes), _p(m.meta), v.spec, _p(v.codes), _p(v.meta),
                                _p(m.y), _p(v.y)), "adamw_step")


def adafactor_step(p, g, rows: int, cols: int, vr: State, vc: State, v: State, t: int, lr=1e-3,
                   eps1=1e-30, clip_d=1.0, decay_rate=-0.8, wd=0.0):
    """One Adafactor step on one tensor, in place. Factored (vr, vc) when rows > 1, else v."""
    g, gb = _grad(g)
    spec = (vr if rows > 1 else v).spec
    nul = None
    _check(lib().orc_adafactor_step(
        rows, cols, _p(p), _p(g), gb, lr, eps1, clip_d, decay_rate, wd, t, spec,
        _p(vr.codes) if vr else nul, _p(vr.meta) if vr else nul,
        _p(vc.codes) if vc else nul, _p(vc.meta) if vc else nul,
        _p(v.codes) if v else nul, _p(v.meta) if v else nul,
        _p(vr.y) if vr else nul, _p(vc.y) if vc else nul, _p(v.y) if v else nul), "adafactor_step")


def came_step(p, g, rows: int, cols: int, m: State, vr: State, vc: State, v: State, cr: State, cc: State,
              t: int, lr=1e-4, beta1=0.9, beta2=0.999, beta3=0.9999, eps1=1e-30, eps2=1e-16, clip_d=1.0,
              wd=0.0):
    """One CAME step on one tensor, in place. Factored states when rows > 1, else v only."""
    g, gb = _grad(g)
    fac = rows > 1
    vspec = (vr if fac else v).spec
    cspec = cr.spec if fac else Spec(0, 256, 0.0)

    def c(s):
        return (_p(s.codes), _p(s.meta), _p(s.y)) if s is not None else (None, None, None)

    mc, vrc, vcc, vvc, crc, ccc = c(m), c(vr), c(vc), c(v), c(cr), c(cc)
    _check(lib().orc_came_step(
        rows, cols, _p(p), _p(g), gb, lr, beta1, beta2, beta3, eps1, eps2, clip_d, wd, t,
        m.spec, vspec, cspec, mc[0], mc[1], vrc[0], vrc[1], vcc[0], vcc[1], vvc[0], vvc[1],
        crc[0], crc[1], ccc[0], ccc[1], mc[2], vrc[2], vcc[2], vvc[2], crc[2], ccc[2]), "came_step")
