"""ORACLE - test infrastructure only.

Plain, slow, obviously correct CPU implementations of what the heterogeneous
Linear path computes.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package; the library never
does.  It shares no code with the library (its C file has its own fp16/bf16
decoders and its own loops).

- ``linear`` / ``linear_sample``: y = x W^T + b in binary32, sequential order
  (HeteGen Sec. 3.1, Fig. 3a, Eq. 2; Sec. 4.2, Fig. 5a: the partitioned module
  computes the same output as the unpartitioned one).
- ``planner``: the computation-distribution law (Sec. 3.2, Eq. 4-7; Eq. 8-9).
- ``attention``: decode attention over a KV cache and the decode step with it
  (Sec. 2.1, Eq. 1).
- ``alpha_bench``, ``scheduler``: the alpha benchmark's fit and solve (Sec. 4.4)
  and the module scheduler (Sec. 4.5, Eq. 13).
- ``decode_step``: the stack of decoder-layer linears with the GPU-side glue
  (Sec. 4.2 keeps non-linear modules on the GPU; glue defined in the design
  notes: pre-LayerNorm, V slice of a one-position attention, ReLU, residual).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
F16, BF16, F32 = 0, 1, 2
_lib = None


def build():
    """Compile liboracle.so (plain C, no fused multiply-add contraction)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", os.path.join(_HERE, "oracle.c"), "-o", _SO + ".tmp"]
    subprocess.check_call(cmd)
    os.replace(_SO + ".tmp", _SO)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        L.oracle_decode_f16.argtypes = [ctypes.c_uint16]
        L.oracle_decode_f16.restype = ctypes.c_float
        L.oracle_decode_bf16.argtypes = [ctypes.c_uint16]
        L.oracle_decode_bf16.restype = ctypes.c_float
        L.oracle_decode.argtypes = [vp, i32, i64, vp]
        L.oracle_linear_f32.argtypes = [vp, i32, i32, i32, vp, i32, i32, vp, vp, i32]
        L.oracle_linear_sample.argtypes = [vp, i32, i32, i32, vp, i32, i32, vp, vp, vp, i64, vp]
        for f in (L.oracle_decode, L.oracle_linear_f32, L.oracle_linear_sample):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def decode(a, dtype):
    """Decode an array of dtype bit patterns (uint16) or float32 into float32."""
    a = np.ascontiguousarray(a)
    out = np.empty(a.shape, dtype=np.float32)
    if lib().oracle_decode(_ptr(a), dtype, a.size, _ptr(out)) != 0:
        raise ValueError("oracle.decode: bad arguments")
    return out


def linear(x, W, bias, dtype):
    """y[B, N] (float32) = x[B, K] W[N, K]^T + bias[N], sequential binary32.

    x, W, bias: uint16 bit patterns for fp16/bf16, float32 for fp32; bias may be None.
    """
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    if x.ndim == 1:
        x = x[None, :]
    B, K = x.shape
    N = W.shape[0]
    assert W.shape[1] == K
    b = None if bias is None else np.ascontiguousarray(bias)
    y = np.empty((B, N), dtype=np.float32)
    rc = lib().oracle_linear_f32(_ptr(x), K, B, K, _ptr(W), N, dtype, _ptr(b), _ptr(y), N)
    if rc != 0:
        raise ValueError("oracle.linear: bad arguments")
    return y


def linear_sample(x, W, bias, dtype, rows_b, rows_j):
    """y[rows_b[i], rows_j[i]] for each i, computed one by one (same arithmetic as linear)."""
    x = np.ascontiguousarray(x)
    if x.ndim == 1:
        x = x[None, :]
    W = np.ascontiguousarray(W)
    B, K = x.shape
    N = W.shape[0]
    rb = np.ascontiguousarray(rows_b, dtype=np.int32)
    rj = np.ascontiguousarray(rows_j, dtype=np.int64)
    out = np.empty(rb.shape, dtype=np.float32)
    b = None if bias is None else np.ascontiguousarray(bias)
    rc = lib().oracle_linear_sample(_ptr(x), K, B, K, _ptr(W), N, dtype, _ptr(b), _ptr(rb), _ptr(rj),
                                    rb.size, _ptr(out))
    if rc != 0:
        raise ValueError("oracle.linear_sample: bad arguments")
    return out


def linear_ptr(x_ptr, ldx, B, K, W_ptr, N, dtype, bias_ptr, y):
    """Same as linear() on raw host addresses (pinned buffers); y is a float32 [B, N] array."""
    rc = lib().oracle_linear_f32(ctypes.c_void_p(x_ptr), ldx, B, K, ctypes.c_void_p(W_ptr), N, dtype,
                                 ctypes.c_void_p(bias_ptr) if bias_ptr else None, _ptr(y), N)
    if rc != 0:
        raise ValueError("oracle.linear_ptr: bad arguments")
    return y


def split_rows(N, alpha_cpu):
    """Output-feature split of one linear: GPU rows [0, n_gpu), CPU rows [n_gpu, N).

    The paper partitions the module's weight (Sec. 3.1, Eq. 2) with a fraction alpha
    on the GPU (Sec. 3.2).  The library's alpha is the CPU fraction (1 - alpha of the
    paper); n_cpu = min(N, floor(alpha_cpu * N + 1/2)).
    """
    import math
    n_cpu = min(N, int(math.floor(alpha_cpu * N + 0.5)))
    return N - n_cpu, n_cpu
