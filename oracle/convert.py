"""Oracle of the 32 <-> 16-bit conversion nodes of section 5.5 (test
infrastructure only; the product package never imports it).

The converter itself is written in C (``oracle/convert.c``), compiled with gcc
on first use into ``oracle/_convert.so``: a plain loop over the arithmetic
definition, fast enough to walk all 2**32 fp32 inputs in a test.

  ``truncate_bf16_bits(f32)``  16-bit patterns of float32 values after the
                               converter (low 16 fraction bits dropped).
  ``truncate_bf16(x)``         values: x is first rounded to fp32 (the value a
                               32-bit producer hands the converter), then
                               converted; returned as exact float64.
  ``truncate_bf16_range(first, count)``  the converter applied to the fp32
                               bit patterns first .. first + count - 1.
  ``widen_bf16(bits)``         16 -> 32 bits: the low half filled with zeros
                               (the exact value of the pattern, as float64).
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "convert.c")
LIB = os.path.join(_HERE, "_convert.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile convert.c (when missing or older than its source)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = f"{LIB}.tmp{os.getpid():x}"
        subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
                        SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        lib.oracle_trunc16_one.argtypes = [ctypes.c_float]
        lib.oracle_trunc16_one.restype = ctypes.c_uint16
        lib.oracle_trunc16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        lib.oracle_trunc16.restype = None
        lib.oracle_trunc16_range.argtypes = [ctypes.c_uint32, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_trunc16_range.restype = None
        _lib = lib
    return _lib


def truncate_bf16_bits(f32) -> np.ndarray:
    """16-bit patterns of the converter applied to float32 values."""
    f = np.ascontiguousarray(f32, dtype=np.float32)
    out = np.empty(f.shape, dtype=np.uint16)
    _load().oracle_trunc16(f.ctypes.data, out.ctypes.data, f.size)
    return out


def truncate_bf16_range(first: int, count: int) -> np.ndarray:
    """The converter on the fp32 bit patterns first, first + 1, ..., first + count - 1."""
    if first < 0 or count < 0 or first + count > 1 << 32:
        raise ValueError("range outside the 32-bit patterns")
    out = np.empty(count, dtype=np.uint16)
    _load().oracle_trunc16_range(first, count, out.ctypes.data)
    return out


def widen_bf16(bits) -> np.ndarray:
    """16 -> 32 bits with the low half zero: the exact value, as float64."""
    u = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def truncate_bf16(x) -> np.ndarray:
    """Values after a 32-bit producer (one rounding to fp32, nearest even)
    and the converter: float64 values that the 16-bit format holds exactly."""
    x = np.asarray(x, dtype=np.float64)
    return widen_bf16(truncate_bf16_bits(x.astype(np.float32)))
