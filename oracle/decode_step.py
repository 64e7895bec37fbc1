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
import torch

from . import F16, BF16, F32, decode, linear

LN_EPS = 1e-5


def layer_norm(x):
    """Row-wise LayerNorm without affine terms, float64."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS)


def to_bits(v, dtype):
    """Round float values to dtype (nearest even) and return the bit patterns."""
    v = np.asarray(v, dtype=np.float64)
    if dtype == F16:
        # float64 -> float16 directly (one rounding)
        return v.astype(np.float16).view(np.uint16)
    if dtype == BF16:
        t = torch.from_numpy(np.ascontiguousarray(v)).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16)
    return v.astype(np.float32)


def act(v, dtype):
    return decode(to_bits(v, dtype), dtype).astype(np.float64)


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
