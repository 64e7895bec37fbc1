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


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_to_bits_matches_library_rounding(dtype):
    v = synth.normal((4096,), oracle.F32, 3, 1, 0, 3).astype(np.float64)
    bits = ds.to_bits(v, dtype)
    if dtype == oracle.F16:
        ref = torch.from_numpy(v).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    else:
        ref = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)


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
