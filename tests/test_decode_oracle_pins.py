"""Pins of the decode-step oracle (glue around the linears) on the CPU."""
import numpy as np
import pytest
import torch

import oracle
from oracle import decode_step as ds
import synth


def test_layer_norm_matches_torch_and_invariants():
    x = synth.normal((4, 96), oracle.F32, 2, 1, 0.3, 2.0).astype(np.float64)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), eps=ds.LN_EPS).numpy()
    ours = ds.layer_norm(x)
    assert np.allclose(ours, ref, rtol=0, atol=1e-12)
    assert np.allclose(ours.mean(-1), 0, atol=1e-12)
    assert np.allclose((ours ** 2).mean(-1), 1 / (1 + ds.LN_EPS / x.var(-1)), rtol=1e-12)


def _f32(bits):
    return np.array([bits], np.uint32).view(np.float32)[0]


# Hand-worked rounding cases: (float64 value, expected 16-bit pattern).
# bfloat16 keeps 7 significand bits after the point, so 1 + 2^-8 is the tie between
# 0x3F80 (1) and 0x3F81 (1 + 2^-7); ties go to the even last bit.
BF16_CASES = [
    (float(_f32(0x3F808000)), 0x3F80),            # 1 + 2^-8: tie, down to even
    (float(_f32(0x3F818000)), 0x3F82),            # 1 + 3 * 2^-8: tie, up to even
    (float(_f32(0x3F808001)), 0x3F81),            # just above the tie
    (float(_f32(0x3F807FFF)), 0x3F80),            # just below the tie
    (-float(_f32(0x3F818000)), 0xBF82),           # sign kept
    (1.0 + 2.0 ** -8 + 2.0 ** -30, 0x3F81),       # one rounding from float64 (through
                                                  # binary32 it would round twice, to 0x3F80)
    (float(_f32(0x3FFF8000)), 0x4000),            # 2 - 2^-8: tie, carries into the next binade
    ((2.0 - 2.0 ** -7) * 2.0 ** 127, 0x7F7F),     # largest finite
    ((2.0 - 2.0 ** -8) * 2.0 ** 127, 0x7F80),     # its tie with 2^128 rounds to infinity
    (2.0 ** 200, 0x7F80),
    (float("-inf"), 0xFF80),
    (2.0 ** -133, 0x0001),                        # smallest subnormal
    (2.0 ** -134, 0x0000),                        # half of it: tie, down to zero
    (3 * 2.0 ** -134, 0x0002),                    # tie between 1 and 2 subnormal units
    (2.0 ** -126, 0x0080),                        # smallest normal
    (-0.0, 0x8000),
    (0.0, 0x0000),
]

# binary16: 10 stored significand bits, so 1 + 2^-11 is the tie after 1.
F16_CASES = [
    (1.0 + 2.0 ** -11, 0x3C00),
    (1.0 + 3 * 2.0 ** -11, 0x3C02),
    (1.0 + 2.0 ** -11 + 2.0 ** -40, 0x3C01),     # above the tie by less than binary32 resolves
    (65504.0, 0x7BFF),                           # largest finite
    (65520.0, 0x7C00),                           # tie with 2^16: infinity
    (2.0 ** -24, 0x0001),
    (2.0 ** -25, 0x0000),
    (3 * 2.0 ** -25, 0x0002),
    (-2.5, 0xC100),
]


@pytest.mark.parametrize("dtype,cases", [(oracle.BF16, BF16_CASES), (oracle.F16, F16_CASES)])
def test_to_bits_hand_worked_rounding(dtype, cases):
    v = np.array([c[0] for c in cases], np.float64)
    want = np.array([c[1] for c in cases], np.uint16)
    got = ds.to_bits(v, dtype)
    bad = [(c[0], hex(c[1]), hex(int(g))) for c, g in zip(cases, got) if int(g) != c[1]]
    assert not bad, bad


def test_to_bits_bf16_nan_stays_nan():
    got = ds.to_bits(np.array([np.nan, -np.nan]), oracle.BF16)
    assert np.all((got & 0x7F80) == 0x7F80) and np.all((got & 0x007F) != 0)


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_to_bits_on_binary32_values_matches_independent_encoder(dtype):
    # binary32 inputs (normals over the whole range, subnormals, values near the types'
    # limits) are rounded once by either route: the oracle's float64 path must give the
    # bits of the generator's integer round-to-nearest-even from binary32
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]          # finite only
    v = bits.view(np.float32)
    extra = synth.normal((4096,), oracle.F32, 3, 1, 0, 3)
    v = np.concatenate([v, extra]).astype(np.float32)
    assert np.array_equal(ds.to_bits(v.astype(np.float64), dtype), synth.encode(v, dtype))


def _layer(H, F, dtype, tid, zero=False):
    shapes = {"qkv": (3 * H, H), "out": (H, H), "fc1": (F, H), "fc2": (H, F)}
    lw = {}
    for i, (name, (n, k)) in enumerate(shapes.items()):
        if zero:
            W = synth.encode(np.zeros((n, k), np.float32), dtype)
            b = synth.encode(np.zeros((n,), np.float32), dtype)
        else:
            W = synth.normal((n, k), dtype, 0, tid + 2 * i, 0, 0.02)
            b = synth.normal((n,), dtype, 0, tid + 2 * i + 1, 0, 0.02)
        lw[name] = (W, b)
    return lw


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_zero_weights_leave_residual_stream_unchanged(dtype):
    H, F = 16, 64
    x = synth.normal((2, H), dtype, 0, 1)
    out, trace = ds.decode_step(x, [_layer(H, F, dtype, 0, zero=True)] * 3, H, dtype)
    assert np.array_equal(out, x)
    assert [t[0] for t in trace] == ["qkv", "out", "fc1", "fc2"] * 3


def test_value_slice_and_residual_by_hand():
    # Wqkv selects the value block as the identity, Wout = I, everything else 0:
    # x1 = act(x + act(LN(x))) after attention; the MLP adds nothing.
    dtype, H, F = oracle.F16, 8, 16
    lw = _layer(H, F, dtype, 0, zero=True)
    Wq = np.zeros((3 * H, H), np.float32)
    Wq[2 * H:3 * H] = np.eye(H)
    lw["qkv"] = (synth.encode(Wq, dtype), lw["qkv"][1])
    lw["out"] = (synth.encode(np.eye(H, dtype=np.float32), dtype), lw["out"][1])
    x = synth.normal((1, H), dtype, 0, 9)
    xd = oracle.decode(x, dtype).astype(np.float64)
    h = oracle.decode(ds.to_bits(ds.layer_norm(xd), dtype), dtype).astype(np.float64)
    want = ds.to_bits(xd + h, dtype)
    out, trace = ds.decode_step(x, [lw], H, dtype)
    assert np.array_equal(out, want)
    q = oracle.decode(trace[0][3], dtype)
    assert np.all(q[:, :2 * H] == 0) and np.array_equal(q[:, 2 * H:], h.astype(np.float32))


def test_relu_applied_to_fc1_output():
    dtype, H, F = oracle.F16, 8, 16
    lw = _layer(H, F, dtype, 40)
    x = synth.normal((3, H), dtype, 0, 2)
    _, trace = ds.decode_step(x, [lw], H, dtype)
    name, _, h2, f_bits = trace[2]
    assert name == "fc1"
    f = oracle.decode(f_bits, dtype)
    pre = oracle.linear(h2, lw["fc1"][0], lw["fc1"][1], dtype)
    assert np.all(f >= 0) and np.all((pre > 0) == (f > 0) | (np.abs(pre) < 1e-7))
