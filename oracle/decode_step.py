"""ORACLE - test infrastructure only: one decode step over a stack of decoder-layer linears.

HeteGen applies heterogeneous parallelism to the linear modules only and keeps the
other modules on the GPU (Sec. 4.2); decoding feeds one token per step through
every layer (Sec. 2.1, Eq. 1).  The glue between the linears is a reading (the
paper leaves it to the model): a pre-LayerNorm OPT-style layer with an
empty KV cache, where one-position attention returns the value projection exactly.

Per layer, with act() = round-to-nearest-even to the activation type:

    h = act(LN(x))                      LN: gamma = 1, beta = 0, eps = 1e-5, biased variance
    q = act(h Wqkv^T + bqkv)            columns ordered [query | key | value], each H wide
    a = q[:, 2H:3H]                     value part
    x = act(x + (a Wout^T + bout))
    h = act(LN(x))
    f = act(ReLU(h Wfc1^T + bfc1))
    x = act(x + (f Wfc2^T + bfc2))

The linears are the oracle's binary32 linear; LN, ReLU and the residual sum are
done in float64 on the decoded values.
"""
import numpy as np

from . import F16, BF16, F32, decode, linear

LN_EPS = 1e-5


def layer_norm(x):
    """Row-wise LayerNorm without affine terms, float64."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS)


BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127  # largest finite bfloat16


def _bf16_round(v):
    """Round float64 values once to bfloat16, nearest with ties to even; bit patterns.

    bfloat16 has binary32's sign and 8-bit exponent and 8 significand bits (7 stored).
    A value of magnitude 2^e <= |v| < 2^(e+1) is rounded to a multiple of its spacing
    2^(e-7); below the smallest normal 2^-126 the spacing stays 2^-133 (subnormals).
    |v| / spacing is exact in float64 and np.rint rounds its halves to even, which is
    the even last significand bit.  Results beyond the largest finite value are
    infinities; NaN becomes the quiet NaN 0x7FC0.
    """
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    _, e = np.frexp(a)                      # a = m 2^e, 0.5 <= m < 1: exponent e - 1
    spacing = np.ldexp(1.0, np.maximum(e - 1, -126) - 7)
    with np.errstate(over="ignore", invalid="ignore"):
        r = np.rint(a / spacing) * spacing
        mag = np.where(r > BF16_MAX, np.inf, r).astype(np.float32)  # exact: r has 8 bits
    bits = (mag.view(np.uint32) >> 16).astype(np.uint16)
    bits = np.where(np.signbit(v), bits | np.uint16(0x8000), bits)
    return np.where(np.isnan(v), np.uint16(0x7FC0), bits).astype(np.uint16)


def to_bits(v, dtype):
    """Round float values once to dtype (nearest, ties to even); bit patterns (binary32
    values for F32)."""
    v = np.asarray(v, dtype=np.float64)
    if dtype == F16:
        # float64 -> float16 directly (one rounding); beyond the range: infinities
        with np.errstate(over="ignore"):
            return v.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        return _bf16_round(v)
    return v.astype(np.float32)


def decode_step(x_bits, layers, H, dtype):
    """Run all layers on x [B, H] (dtype bits).

    layers: list of dicts with keys 'qkv', 'out', 'fc1', 'fc2', each a (W_bits, b_bits) pair.
    Returns (x_out_bits, trace) where trace is a list, in execution order, of
    (name, layer, input_bits, output_bits) for every linear.
    """
    x = decode(x_bits, dtype).astype(np.float64)
    trace = []
    for l, lw in enumerate(layers):
        h = to_bits(layer_norm(x), dtype)
        q = linear(h, lw["qkv"][0], lw["qkv"][1], dtype)
        q_bits = to_bits(q, dtype)
        trace.append(("qkv", l, h, q_bits))
        a = np.ascontiguousarray(q_bits[:, 2 * H:3 * H])
        o = linear(a, lw["out"][0], lw["out"][1], dtype).astype(np.float64)
        x_bits_mid = to_bits(x + o, dtype)
        trace.append(("out", l, a, x_bits_mid))
        x = decode(x_bits_mid, dtype).astype(np.float64)
        h2 = to_bits(layer_norm(x), dtype)
        f = linear(h2, lw["fc1"][0], lw["fc1"][1], dtype).astype(np.float64)
        f_bits = to_bits(np.maximum(f, 0.0), dtype)
        trace.append(("fc1", l, h2, f_bits))
        o2 = linear(f_bits, lw["fc2"][0], lw["fc2"][1], dtype).astype(np.float64)
        x_bits_out = to_bits(x + o2, dtype)
        trace.append(("fc2", l, f_bits, x_bits_out))
        x = decode(x_bits_out, dtype).astype(np.float64)
    return to_bits(x, dtype), trace
