"""ORACLE - test infrastructure only: decode attention over a KV cache.

HeteGen Sec. 2.1, Eq. 1: at a decode step the new token's key and value are
concatenated to the cached keys and values of the earlier positions, and the new
token's query attends to all of them.  Multi-head scaled dot-product attention,
head h of width D (H / D heads), positions j = 0..pos:

    s_j = q_h . K_{j,h} / sqrt(D),     a_h = sum_j softmax(s)_j V_{j,h}

in float64 on the decoded activation-type values; callers round the result to the
activation type.  The full decode step with a cache is the stack of decoder
layers of `decode_step` with this attention in place of the empty-cache value
slice.
"""
import numpy as np

from . import decode, linear
from .decode_step import layer_norm, to_bits


def append(cache, new):
    """Eq. 1: the cache of one layer [B, pos, H] with the new token's row [B, H] appended."""
    new = np.asarray(new)[:, None, :]
    return new if cache is None or cache.shape[1] == 0 else np.concatenate([cache, new], axis=1)


def attend(q, K, V, head_dim):
    """q [B, H], K and V [B, n, H] (float values); returns [B, H] float64."""
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    B, H = q.shape
    out = np.empty((B, H), np.float64)
    for b in range(B):
        for h in range(H // head_dim):
            cols = slice(h * head_dim, (h + 1) * head_dim)
            s = K[b, :, cols] @ q[b, cols] / np.sqrt(head_dim)
            p = np.exp(s - s.max())
            out[b, cols] = (p / p.sum()) @ V[b, :, cols]
    return out


def decode_step_kv(x_bits, layers, H, dtype, k_cache, v_cache, head_dim):
    """One decode step of x [B, H] (dtype bits) with per-layer caches of the earlier
    positions (lists of [B, pos, H] dtype bits, or None when empty).

    Returns (x_out_bits, trace, k_cache', v_cache'): the trace lists, per linear,
    (name, layer, input_bits, output_bits); the caches have the new token appended.
    """
    x = decode(x_bits, dtype).astype(np.float64)
    trace, kc_out, vc_out = [], [], []
    for l, lw in enumerate(layers):
        h = to_bits(layer_norm(x), dtype)
        qkv = to_bits(linear(h, lw["qkv"][0], lw["qkv"][1], dtype), dtype)
        trace.append(("qkv", l, h, qkv))
        Kl = append(k_cache[l], qkv[:, H:2 * H])
        Vl = append(v_cache[l], qkv[:, 2 * H:3 * H])
        kc_out.append(Kl)
        vc_out.append(Vl)
        a = to_bits(attend(decode(qkv[:, :H], dtype), decode(Kl, dtype), decode(Vl, dtype), head_dim), dtype)
        o = linear(a, lw["out"][0], lw["out"][1], dtype).astype(np.float64)
        x_mid = to_bits(x + o, dtype)
        trace.append(("out", l, a, x_mid))
        x = decode(x_mid, dtype).astype(np.float64)
        h2 = to_bits(layer_norm(x), dtype)
        f = to_bits(np.maximum(linear(h2, lw["fc1"][0], lw["fc1"][1], dtype).astype(np.float64), 0.0), dtype)
        trace.append(("fc1", l, h2, f))
        o2 = linear(f, lw["fc2"][0], lw["fc2"][1], dtype).astype(np.float64)
        x_out = to_bits(x + o2, dtype)
        trace.append(("fc2", l, f, x_out))
        x = decode(x_out, dtype).astype(np.float64)
    return to_bits(x, dtype), trace, kc_out, vc_out
