"""The CPU share of the heterogeneous linear (host cores only, no device) against
the oracle: random inputs within the tolerance, integer inputs bit for bit, and the
same bits for every thread count and row range."""
import numpy as np
import pytest

import oracle
import synth
from common import TOL, rel_err

hg = pytest.importorskip("paper_2403_01164_amd")


def _problem(B, K, N, dtype, kind, seed):
    if kind == "int":
        x = synth.integers((B, K), dtype, seed, 1, -1, 1)
        W = synth.integers((N, K), dtype, seed, 2, -1, 1)
        b = synth.integers((N,), dtype, seed, 3, -4, 4)
    else:
        x = synth.normal((B, K), dtype, seed, 1, 0.0, 1.0)
        W = synth.normal((N, K), dtype, seed, 2, 0.0, 0.02)
        b = synth.normal((N,), dtype, seed, 3, 0.0, 0.02)
    return x, W, b


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 8])
@pytest.mark.parametrize("K", [8, 24, 48, 520, 1032, 4096])
def test_random_inputs_match_oracle(dtype, B, K):
    # K covers a tail of 8, 16 or 24 elements after whole 32-element chunks, no tail, and
    # shares shorter than one chunk (the bf16 dot-product path works in 32-element chunks)
    N = 77
    x, W, b = _problem(B, K, N, dtype, "normal", seed=K + B)
    ref = oracle.linear(x, W, b, dtype)
    for r0, r1 in ((0, N), (13, 70), (5, 6)):
        y = hg.hetegen_cpu_linear(oracle.decode(x, dtype), W.ctypes.data, b.ctypes.data, dtype, r0, r1)
        assert rel_err(y, ref[:, r0:r1]) <= TOL, (r0, r1)


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B", [1, 4, 8])
def test_integer_inputs_bit_exact(dtype, B):
    K, N = 240, 131
    x, W, b = _problem(B, K, N, dtype, "int", seed=9)
    ref = oracle.linear(x, W, b, dtype)
    y = hg.hetegen_cpu_linear(oracle.decode(x, dtype), W.ctypes.data, b.ctypes.data, dtype, 0, N)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("B", [1, 3, 8])
def test_same_bits_for_any_thread_count_and_row_range(B):
    dtype, K, N = synth.F16, 4096, 203
    x, W, b = _problem(B, K, N, dtype, "normal", seed=4)
    xf = oracle.decode(x, dtype)
    full = hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, 0, N, threads=1)
    for t in (2, 5, 8):
        assert np.array_equal(hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, 0, N, threads=t), full)
    # a row's value does not depend on which other rows share its call
    part = hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, 37, 151, threads=3)
    assert np.array_equal(part, full[:, 37:151])


@pytest.mark.parametrize("K", [8, 40, 1032])
def test_bf16_weights_keep_binary32_x(K):
    # x values that bf16 cannot hold (1 + 2^-10) with bf16 weights of 1 (and of 2 in one
    # row): the exact binary32 sums, not those of x rounded to bf16; and bf16 x values on
    # the same weights still give exact sums (the dot-product path where the host has it)
    B, N = 2, 9
    one, two = 0x3F80, 0x4000  # bf16 bit patterns of 1 and 2
    W = np.full((N, K), one, np.uint16)
    W[3] = two
    xf = np.full((B, K), 1.0 + 2.0 ** -10, np.float32)
    xf[1, ::2] = 1.0  # a second row mixing bf16 values in
    y = hg.hetegen_cpu_linear(xf, W.ctypes.data, 0, synth.BF16, 0, N)
    ref = xf.astype(np.float64).sum(axis=1)[:, None] * np.where(np.arange(N) == 3, 2.0, 1.0)[None, :]
    assert np.array_equal(y.astype(np.float64), ref)
    xb = np.full((B, K), 1.5, np.float32)
    y = hg.hetegen_cpu_linear(xb, W.ctypes.data, 0, synth.BF16, 0, N)
    assert np.array_equal(y.astype(np.float64), 1.5 * K * np.where(np.arange(N) == 3, 2.0, 1.0)[None, :].repeat(B, 0))


def test_no_bias_and_empty_range():
    dtype, B, K, N = synth.BF16, 2, 64, 10
    x, W, b = _problem(B, K, N, dtype, "normal", seed=5)
    ref = oracle.linear(x, W, None, dtype)
    assert rel_err(hg.hetegen_cpu_linear(oracle.decode(x, dtype), W.ctypes.data, 0, dtype, 0, N), ref) <= TOL
    assert hg.hetegen_cpu_linear(oracle.decode(x, dtype), W.ctypes.data, 0, dtype, 4, 4).shape == (B, 0)


def test_bad_arguments():
    x = np.zeros((1, 12), np.float32)
    W = np.zeros((4, 12), np.uint16)
    with pytest.raises(hg.HetegenError):  # K % 8
        hg.hetegen_cpu_linear(x, W.ctypes.data, 0, synth.F16, 0, 4)
    with pytest.raises(hg.HetegenError):  # rows reversed
        hg.hetegen_cpu_linear(np.zeros((1, 8), np.float32), W.ctypes.data, 0, synth.F16, 3, 2)


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("K", [48, 264, 520, 4104])
def test_batch_rows_independent(dtype, K):
    # every batch row gets the bits it gets alone (batches of 5-8 run in two groups over
    # L1-resident chunks; the order of each row's products does not change)
    B, N = 8, 37
    x, W, b = _problem(B, K, N, dtype, "normal", seed=K)
    xf = oracle.decode(x, dtype)
    full = hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, 0, N)
    for nb in (5, 6, 7):
        part = hg.hetegen_cpu_linear(np.ascontiguousarray(xf[:nb]), W.ctypes.data, b.ctypes.data, dtype, 0, N)
        assert np.array_equal(part, full[:nb]), nb
    for bb in range(B):
        one = hg.hetegen_cpu_linear(np.ascontiguousarray(xf[bb:bb + 1]), W.ctypes.data, b.ctypes.data, dtype, 0, N)
        assert np.array_equal(one[0], full[bb]), bb


def test_calls_from_several_threads():
    # the worker team runs one job at a time; concurrent callers get their own results
    import threading
    dtype, B, K, N = synth.BF16, 5, 520, 2051
    x, W, b = _problem(B, K, N, dtype, "normal", seed=11)
    xf = oracle.decode(x, dtype)
    ref = hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, 0, N)
    bad = []

    def worker(k):
        for it in range(60):
            r0, r1 = (k * 13 + it) % 40, N - (it * 7) % 50
            y = hg.hetegen_cpu_linear(xf, W.ctypes.data, b.ctypes.data, dtype, r0, r1, threads=1 + (it + k) % 8)
            if not np.array_equal(y, ref[:, r0:r1]):
                bad.append((k, it))

    ts = [threading.Thread(target=worker, args=(k,)) for k in range(4)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not bad
