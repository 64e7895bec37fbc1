"""Pins of the oracle against facts fixed outside it (CPU only).

Each test checks the oracle against something other than its own formula: a
library routine, exact integer arithmetic, a float64 brute force with the
binary32 error bound, or a closed form.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth

U32 = 2.0 ** -24  # unit roundoff of binary32


def _gamma(n):
    return n * U32 / (1.0 - n * U32)


def test_decode_f16_exhaustive_matches_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.decode(bits, oracle.F16)
    ref = bits.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_decode_bf16_exhaustive_matches_torch():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.decode(bits, oracle.BF16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16, oracle.F32])
@pytest.mark.parametrize("B,K,N", [(1, 8, 1), (1, 1024, 37), (4, 520, 64), (8, 2040, 17)])
def test_linear_integer_inputs_exact(dtype, B, K, N):
    # x, W in {-1, 0, 1}, bias in {-4..4}: every partial sum is an integer below 2^24,
    # so the binary32 result equals the exact integer result.
    x = synth.integers((B, K), dtype, 0, 1, -1, 1)
    W = synth.integers((N, K), dtype, 0, 2, -1, 1)
    b = synth.integers((N,), dtype, 0, 3, -4, 4)
    xi = oracle.decode(x, dtype).astype(np.int64)
    Wi = oracle.decode(W, dtype).astype(np.int64)
    bi = oracle.decode(b, dtype).astype(np.int64)
    exact = xi @ Wi.T + bi
    y = oracle.linear(x, W, b, dtype)
    assert np.array_equal(y.astype(np.int64), exact)
    assert np.array_equal(y, exact.astype(np.float32))


def _brute_force_f64(x, W, b):
    B, K = x.shape
    N = W.shape[0]
    out = np.zeros((B, N))
    absd = np.zeros((B, N))
    for bb in range(B):
        for j in range(N):
            s = 0.0
            a = 0.0
            for k in range(K):
                p = float(x[bb, k]) * float(W[j, k])
                s += p
                a += abs(p)
            if b is not None:
                s += float(b[j])
                a += abs(float(b[j]))
            out[bb, j] = s
            absd[bb, j] = a
    return out, absd


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
@pytest.mark.parametrize("B,K,N", [(1, 64, 5), (3, 40, 7), (8, 16, 3)])
def test_linear_random_within_binary32_bound_of_float64(dtype, B, K, N):
    x = synth.normal((B, K), dtype, 7, 11, 0.0, 1.0)
    W = synth.normal((N, K), dtype, 7, 12, 0.0, 0.02)
    b = synth.normal((N,), dtype, 7, 13, 0.0, 0.02)
    xd, Wd, bd = (oracle.decode(a, dtype).astype(np.float64) for a in (x, W, b))
    ref, absd = _brute_force_f64(xd, Wd, bd)
    y = oracle.linear(x, W, b, dtype).astype(np.float64)
    # Sequential summation of K products and a bias: |err| <= gamma_{K+1} * sum|terms|
    # (Higham, Accuracy and Stability of Numerical Algorithms, eq. 3.5).
    bound = _gamma(K + 1) * absd
    assert np.all(np.abs(y - ref) <= bound + 1e-30)
    # a dropped term or a wrong row would be far outside that bound
    assert np.max(bound) < 1e-3 * np.max(np.abs(Wd))


def test_linear_bias_none_and_fp32_inputs():
    x = synth.normal((2, 24), oracle.F32, 1, 1)
    W = synth.normal((5, 24), oracle.F32, 1, 2, 0.0, 0.5)
    y = oracle.linear(x, W, None, oracle.F32).astype(np.float64)
    ref, absd = _brute_force_f64(x.astype(np.float64), W.astype(np.float64), None)
    assert np.all(np.abs(y - ref) <= _gamma(25) * absd)


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_linear_matches_torch_linear_fp32(dtype):
    B, K, N = 4, 1024, 96
    x = synth.normal((B, K), dtype, 3, 1)
    W = synth.normal((N, K), dtype, 3, 2, 0.0, 0.02)
    b = synth.normal((N,), dtype, 3, 3, 0.0, 0.02)
    xd, Wd, bd = (torch.from_numpy(oracle.decode(a, dtype)) for a in (x, W, b))
    ref = torch.nn.functional.linear(xd.double(), Wd.double(), bd.double()).numpy()
    absd = (xd.double().abs() @ Wd.double().abs().T + bd.double().abs()).numpy()
    y = oracle.linear(x, W, b, dtype).astype(np.float64)
    assert np.all(np.abs(y - ref) <= _gamma(K + 1) * absd)


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_linear_order_is_sequential_with_bias_last(dtype):
    # products 2^24, 1, -2^24 (all exact in binary32).  In the order k = 0, 1, 2:
    # 2^24 + 1 rounds (tie to even) to 2^24, minus 2^24 gives 0; the exact sum is 1.
    x = synth.encode(np.array([[4096.0, 1.0, -4096.0]], np.float32), dtype)
    W = synth.encode(np.array([[4096.0, 1.0, 4096.0]], np.float32), dtype)
    zero = synth.encode(np.array([0.0], np.float32), dtype)
    one = synth.encode(np.array([1.0], np.float32), dtype)
    assert oracle.linear(x, W, zero, dtype)[0, 0] == 0.0
    # bias added after the last product: 0 + 1 = 1.  (Exact: 2; bias first: 1 + 2^24 -> 2^24,
    # + 1 -> 2^24, - 2^24 -> 0.)
    assert oracle.linear(x, W, one, dtype)[0, 0] == 1.0


def test_linear_sample_equals_full():
    dtype = oracle.F16
    x = synth.normal((3, 256), dtype, 5, 1)
    W = synth.normal((77, 256), dtype, 5, 2, 0.0, 0.02)
    b = synth.normal((77,), dtype, 5, 3, 0.0, 0.02)
    full = oracle.linear(x, W, b, dtype)
    rb = np.array([0, 2, 1, 2, 0])
    rj = np.array([0, 76, 33, 5, 76])
    s = oracle.linear_sample(x, W, b, dtype, rb, rj)
    assert np.array_equal(s, full[rb, rj])


def test_linear_rejects_bad_arguments():
    x = synth.normal((1, 8), oracle.F16, 0, 1)
    W = synth.normal((4, 8), oracle.F16, 0, 2)
    with pytest.raises(ValueError):
        oracle.linear_sample(x, W, None, oracle.F16, [0], [4])


def test_split_rows_reading():
    # alpha is the CPU fraction; GPU rows lead.  Half-way cases round up.
    assert oracle.split_rows(4096, 0.0) == (4096, 0)
    assert oracle.split_rows(4096, 1.0) == (0, 4096)
    assert oracle.split_rows(4096, 0.25) == (3072, 1024)
    assert oracle.split_rows(4096, 0.5) == (2048, 2048)
    assert oracle.split_rows(3, 0.5) == (1, 2)      # 1.5 -> 2 CPU rows
    assert oracle.split_rows(7, 1.0 / 7) == (6, 1)
    prev = 0
    for a in np.linspace(0, 1, 101):
        g, c = oracle.split_rows(1001, float(a))
        assert g + c == 1001 and c >= prev
        prev = c


def test_linear_ptr_equals_array_form_with_row_stride():
    # the raw-address form (pinned buffers in the benchmark's baseline) reads x with a row
    # stride and writes the same bits as the array form
    B, K, N, dt = 3, 72, 40, oracle.F16
    xs = synth.normal((B, K + 8), dt, 4, 1)
    W = synth.normal((N, K), dt, 4, 2, 0, 0.02)
    b = synth.normal((N,), dt, 4, 3, 0, 0.02)
    y = np.empty((B, N), np.float32)
    oracle.linear_ptr(xs.ctypes.data, K + 8, B, K, W.ctypes.data, N, dt, b.ctypes.data, y)
    ref = oracle.linear(np.ascontiguousarray(xs[:, :K]), W, b, dt)
    assert np.array_equal(y.view(np.uint32), ref.view(np.uint32))
