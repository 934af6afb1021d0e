"""Seeded synthetic inputs shared by both sides of every parity test.

This package is the only code that the oracle and the GPU path have in
common.  It turns (seed, stream, index) into numbers and lays the numbers out
as model tensors; it contains none of the MoE method's arithmetic (no routing,
no prediction, no cache policy, no expert math).

* ``normal()``: Philox4x32-10 + Box-Muller normals from ``synth.c`` (a small C
  library built with gcc), fp32 or bf16 (round-to-nearest-even).
* ``configs``: the five workload shapes.
* ``model``: seeded weight and input recipes for those shapes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsynth.so")
_SRC = os.path.join(_HERE, "synth.c")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile synth.c into libsynth.so (gcc, OpenMP)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-march=x86-64-v3", "-fno-math-errno", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _SO)
    return _SO


def lib() -> ctypes.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_SO):
                build(force=False)
            l = ctypes.CDLL(_SO)
            u64, sz, f32 = ctypes.c_uint64, ctypes.c_size_t, ctypes.c_float
            for name in ("synth_normal_f32", "synth_normal_bf16"):
                fn = getattr(l, name)
                fn.argtypes = [u64, u64, u64, sz, f32, f32, ctypes.c_void_p]
                fn.restype = None
            l.synth_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
            l.synth_philox4x32_10.restype = None
            i64 = ctypes.c_int64
            l.synth_quant_int4.argtypes = [ctypes.c_void_p, i64, i64, i64, ctypes.c_void_p, ctypes.c_void_p]
            l.synth_quant_int4.restype = None
            _lib = l
    return _lib


def philox4x32_10(ctr, key):
    """Raw Philox4x32-10 block (for known-answer tests)."""
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    lib().synth_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def normal(seed: int, stream: int, n: int, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32", offset: int = 0, out=None):
    """n normals (mean + std * N(0,1)) of stream ``stream`` starting at ``offset``.

    dtype 'f32' returns float32; 'bf16' returns the raw bf16 bits as uint16.
    ``out`` may be a numpy array or an integer address of n elements.
    """
    if dtype == "f32":
        fn, npdt = lib().synth_normal_f32, np.float32
    elif dtype == "bf16":
        fn, npdt = lib().synth_normal_bf16, np.uint16
    else:
        raise ValueError(dtype)
    if out is None:
        arr = np.empty(n, dtype=npdt)
        addr = arr.ctypes.data
    elif isinstance(out, int):
        arr, addr = None, out
    else:
        arr = out
        assert arr.dtype == npdt and arr.size >= n and arr.flags["C_CONTIGUOUS"]
        addr = arr.ctypes.data
    if n:
        fn(ctypes.c_uint64(seed & (2**64 - 1)), ctypes.c_uint64(stream & (2**64 - 1)),
           ctypes.c_uint64(offset), ctypes.c_size_t(n), ctypes.c_float(mean), ctypes.c_float(std),
           ctypes.c_void_p(addr))
    return arr


def quant_int4(w_bf16, rows: int, K: int, group: int, codes_addr: int, scales_addr: int) -> None:
    """4-bit storage of a bf16 matrix [rows, K] (raw uint16 bits, C-contiguous
    numpy array): codes (rows x K/2 bytes) to codes_addr, bf16 scales (rows x
    K/group) to scales_addr; see synth_quant_int4 in synth.c."""
    w = np.ascontiguousarray(w_bf16, dtype=np.uint16)
    assert w.size == rows * K and K % group == 0 and group % 2 == 0
    lib().synth_quant_int4(ctypes.c_void_p(w.ctypes.data), rows, K, group, ctypes.c_void_p(codes_addr),
                           ctypes.c_void_p(scales_addr))
