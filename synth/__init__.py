"""Seeded synthetic inputs (counter-based splitmix64 + Box-Muller).

This module is shared by the tests, the benchmark and the oracle checks; it holds
none of the method's arithmetic.  Values depend only on (seed, tensor id, index).
Element type codes: 0 = fp16, 1 = bf16, 2 = fp32 (the same codes the library uses).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsynth.so")
F16, BF16, F32 = 0, 1, 2
_lib = None


def build():
    """Compile libsynth.so with gcc (plain C, OpenMP)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           os.path.join(_HERE, "gen.c"), "-o", _SO + ".tmp", "-lm"]
    subprocess.check_call(cmd)
    os.replace(_SO + ".tmp", _SO)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        i64, u64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
        L.synth_fill_normal.argtypes = [vp, i64, ctypes.c_int, u64, u64, ctypes.c_double, ctypes.c_double]
        L.synth_fill_int.argtypes = [vp, i64, ctypes.c_int, u64, u64, ctypes.c_int, ctypes.c_int]
        L.synth_encode.argtypes = [vp, vp, i64, ctypes.c_int]
        for f in (L.synth_fill_normal, L.synth_fill_int, L.synth_encode):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc):
    if rc != 0:
        raise ValueError("synth: invalid arguments")


def fill_normal_ptr(ptr, n, dtype, seed, tensor_id, mean=0.0, std=1.0):
    """Fill n elements at host address ptr with mean + std * N(0, 1)."""
    _check(lib().synth_fill_normal(ctypes.c_void_p(ptr), n, dtype, seed, tensor_id, mean, std))


def fill_int_ptr(ptr, n, dtype, seed, tensor_id, lo, hi):
    """Fill n elements at host address ptr with uniform integers in [lo, hi]."""
    _check(lib().synth_fill_int(ctypes.c_void_p(ptr), n, dtype, seed, tensor_id, lo, hi))


def _np_dtype(dtype):
    return np.float32 if dtype == F32 else np.uint16


def normal(shape, dtype, seed, tensor_id, mean=0.0, std=1.0):
    """numpy array (uint16 bit patterns for fp16/bf16, float32 otherwise)."""
    a = np.empty(shape, dtype=_np_dtype(dtype))
    fill_normal_ptr(a.ctypes.data, a.size, dtype, seed, tensor_id, mean, std)
    return a


def integers(shape, dtype, seed, tensor_id, lo, hi):
    a = np.empty(shape, dtype=_np_dtype(dtype))
    fill_int_ptr(a.ctypes.data, a.size, dtype, seed, tensor_id, lo, hi)
    return a


def encode(values, dtype):
    """Encode float values (exactly representable ones stay exact) into dtype bits."""
    src = np.ascontiguousarray(values, dtype=np.float32)
    a = np.empty(src.shape, dtype=_np_dtype(dtype))
    _check(lib().synth_encode(ctypes.c_void_p(src.ctypes.data), ctypes.c_void_p(a.ctypes.data),
                              src.size, dtype))
    return a


# Tensor ids used by the OPT-shaped workloads: one id per (layer, linear, part).
LINEAR_NAMES = ("qkv", "out", "fc1", "fc2")


def weight_id(layer, which):
    return 1000 + 8 * layer + 2 * LINEAR_NAMES.index(which)


def bias_id(layer, which):
    return weight_id(layer, which) + 1


def act_id(step):
    return 10 + step
