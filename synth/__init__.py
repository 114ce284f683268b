"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This package holds no arithmetic of the decoding method.  It turns
(seed, tensor name, element index) into numbers with a counter-based
generator (Philox-4x32-10, Salmon et al., SC'11) implemented in
``philox.c``, so that the oracle and the GPU consume identical bits:

* ``normal_bf16`` -- N(0, std) as bfloat16 bit patterns (uint16),
* ``uniform_int`` -- integers uniform in [lo, hi],
* ``normal_f64``  -- the underlying standard normals (for tests).

Each tensor draws from its own stream, keyed by the 32-bit FNV-1a hash of
its name, so tensors are independent of generation order and can be
produced piecewise (``offset``) for large shapes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "philox.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile libsynth.so next to its source (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"],
                       check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        u32, u64, i32 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
        vp = ctypes.c_void_p
        lib.synth_philox4x32_10.argtypes = [vp, vp, vp]
        lib.synth_normal_f64.argtypes = [u32, u32, u64, u64, vp]
        lib.synth_normal_bf16.argtypes = [u32, u32, u64, u64, ctypes.c_double, vp]
        lib.synth_uniform_int.argtypes = [u32, u32, u64, u64, i32, i32, vp]
        lib.synth_f32_to_bf16.argtypes = [ctypes.c_float]
        lib.synth_f32_to_bf16.restype = ctypes.c_uint16
        _lib = lib
    return _lib


def stream_id(name: str) -> int:
    """32-bit FNV-1a hash of a tensor name: the Philox key's second word."""
    h = 0x811C9DC5
    for b in name.encode("utf-8"):
        h ^= b
        h = (h * 0x01000193) & 0xFFFFFFFF
    return h


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    _load().synth_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def normal_f64(seed: int, name: str, shape, offset: int = 0) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float64)
    _load().synth_normal_f64(seed & 0xFFFFFFFF, stream_id(name), offset, n, out.ctypes.data)
    return out.reshape(shape)


def normal_bf16(seed: int, name: str, shape, std: float, offset: int = 0, out=None) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of N(0, std) draws, row-major ``shape``."""
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(shape, dtype=np.uint16)
    assert out.dtype == np.uint16 and out.flags.c_contiguous and out.size == n
    _load().synth_normal_bf16(seed & 0xFFFFFFFF, stream_id(name), offset, n, float(std), out.ctypes.data)
    return out


def uniform_int(seed: int, name: str, shape, lo: int, hi: int, offset: int = 0) -> np.ndarray:
    """int32 values uniform in the closed range [lo, hi]."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.int32)
    _load().synth_uniform_int(seed & 0xFFFFFFFF, stream_id(name), offset, n, int(lo), int(hi), out.ctypes.data)
    return out.reshape(shape)


def f32_to_bf16(x: float) -> int:
    return int(_load().synth_f32_to_bf16(float(x)))


def bf16_ones(n: int) -> np.ndarray:
    """bfloat16 bit patterns of 1.0 (0x3F80)."""
    return np.full(n, 0x3F80, dtype=np.uint16)


def f32_array_to_bf16(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def gain_bf16(seed: int, name: str, n: int, std: float) -> np.ndarray:
    """bfloat16 bit patterns of 1 + std * z (z standard normal, its own stream): a seeded vector of
    scale factors near one.  std = 0 gives exact ones."""
    if std == 0.0:
        return bf16_ones(n)
    return f32_array_to_bf16((1.0 + std * normal_f64(seed, name, (n,))).astype(np.float32))
