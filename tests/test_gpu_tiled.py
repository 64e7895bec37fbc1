"""GPU parity of the matrix-core GEMV on tile-ordered weights (hetegen_tile_weights,
hetegen_linear_tiled) through the C ABI, against the oracle linear.

The tile layout is checked element by element against its definition in the header;
integer inputs (every partial sum an exact integer in binary32) must give the oracle's
bits, including when the sum over K is split across workgroups; random inputs must be
within the tolerance; each batch row's result must not depend on the others.
"""
import numpy as np
import pytest

import oracle
import synth
from common import TOL, U_ACT, np_from_dev, rel_err, torch_dev_from_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")


@pytest.fixture(scope="module")
def ctx():
    c = hg.hetegen_create(0)
    yield c
    hg.hetegen_destroy(c)


def _tiled(ctx, W_bits):
    """Device copy of W [N, K] (bit patterns) in tile order."""
    N, K = W_bits.shape
    Wd = torch_dev_from_np(W_bits)
    nb = hg.hetegen_tiled_bytes(N, K)
    Wt = torch.full((nb // 2,), -1, dtype=torch.int16, device="cuda")
    hg.hetegen_tile_weights(ctx, Wd.data_ptr(), N, K, Wt.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return Wt


def _run(ctx, x_bits, Wt, N, dtype, bias_bits=None, y_f32=True):
    B, K = x_bits.shape
    xd = torch_dev_from_np(x_bits)
    bd = torch_dev_from_np(bias_bits) if bias_bits is not None else None
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda") if y_f32 else \
        torch.full((B, N), -1, dtype=torch.int16, device="cuda")
    hg.hetegen_linear_tiled(ctx, xd.data_ptr(), B, K, Wt.data_ptr(), N, dtype, bd.data_ptr() if bd is not None else 0,
                            y.data_ptr(), hg.F32 if y_f32 else dtype, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return np_from_dev(y, np.float32) if y_f32 else np_from_dev(y, np.uint16)


@pytest.mark.parametrize("N,K", [(37, 72), (16, 32), (50, 4104)])
def test_tile_layout_matches_definition(ctx, N, K):
    W = synth.integers((N, K), synth.F16, 0, 7, -1000, 1000)
    Wt = np_from_dev(_tiled(ctx, W), np.uint16)
    RT, KT = -(-N // 16), -(-K // 32)
    assert Wt.size * 2 == hg.hetegen_tiled_bytes(N, K) == RT * KT * 1024
    tiles = Wt.reshape(RT, KT, 64, 8)  # [row tile][k tile][lane][element]
    want = np.zeros((RT * 16, KT * 32), np.uint16)
    want[:N, :K] = W
    for lane in range(64):
        r, g = lane % 16, lane // 16
        for e in range(8):
            got = tiles[:, :, lane, e]                      # [RT, KT]
            ref = want[r::16, :][:, g * 8 + e::32]          # rows 16 t + r, columns 32 k + 8 g + e
            assert np.array_equal(got, ref), (lane, e)


# on a 256-CU device the last four split K (into 4, 8, 8 and 8); the first two cannot (K < 2048)
SHAPES = [(37, 72), (256, 1024), (1000, 4104), (130, 8192), (48, 16384), (16, 36864)]


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("N,K", SHAPES)
@pytest.mark.parametrize("B", [1, 3, 8])
def test_linear_tiled_parity(ctx, dtype, N, K, B):
    W = synth.normal((N, K), dtype, 0, 11, 0, 0.02)
    b = synth.normal((N,), dtype, 0, 12, 0, 0.02)
    x = synth.normal((B, K), dtype, 0, 13)
    Wt = _tiled(ctx, W)
    ref = oracle.linear(x, W, b, dtype).astype(np.float64)
    y = _run(ctx, x, Wt, N, dtype, b)
    assert rel_err(y, ref) <= TOL
    y16 = _run(ctx, x, Wt, N, dtype, b, y_f32=False)
    assert rel_err(oracle.decode(y16, dtype), ref) <= TOL + U_ACT[dtype]


@pytest.mark.parametrize("N,K,dtype", [
    (4096, 16384, synth.F16),   # OPT-6.7B fc2: 256 row tiles, unsplit on a 256-CU device
    (5120, 5120, synth.F16),    # OPT-13B out: 320 row tiles, 4 K-splits
    (5120, 20480, synth.F16),   # OPT-13B fc2: 4 K-splits
    (7168, 28672, synth.F16),   # OPT-30B fc2: 448 row tiles, unsplit
    (9216, 9216, synth.BF16),   # OPT-66B out: 576 row tiles, 2 K-splits
    (9216, 36864, synth.BF16),  # OPT-66B fc2: 2 K-splits
    (27648, 9216, synth.BF16),  # OPT-66B qkv: 1728 row tiles, unsplit
])
@pytest.mark.parametrize("B", [1, 8])
def test_linear_tiled_full_size_opt_shapes(ctx, N, K, dtype, B):
    # the matrix-core GEMV at full OPT out / fc2 / qkv sizes, where the split rule keeps or
    # drops the split over K: 288 output rows (the first and last 16, 256 more at random)
    # against the oracle, and the bits do not change from call to call
    W = synth.normal((N, K), dtype, 0, 71, 0, 0.02)
    b = synth.normal((N,), dtype, 0, 72, 0, 0.02)
    x = synth.normal((B, K), dtype, 0, 73)
    Wt = _tiled(ctx, W)
    y = _run(ctx, x, Wt, N, dtype, b)
    rows = np.unique(np.concatenate([np.arange(16), np.arange(N - 16, N),
                                     np.random.default_rng(N + K).choice(N, 256, replace=False)]))
    ref = oracle.linear(x, np.ascontiguousarray(W[rows]), np.ascontiguousarray(b[rows]), dtype).astype(np.float64)
    assert rel_err(y[:, rows], ref) <= TOL
    assert np.array_equal(_run(ctx, x, Wt, N, dtype, b).view(np.uint32), y.view(np.uint32))


@pytest.mark.parametrize("dtype,N,K", [(synth.F16, 100, 2040), (synth.BF16, 40, 248), (synth.F16, 64, 16384),
                                       (synth.BF16, 33, 36864)])
@pytest.mark.parametrize("B", [1, 2, 5, 8])  # lanes of product columns past B read no x
def test_linear_tiled_integer_inputs_bit_exact(ctx, dtype, N, K, B):
    # x, W in {-1, 0, 1}, bias in {-4..4}: every partial sum is an integer below 2^24, so any
    # summation order (the matrix core's, the split over K) gives the oracle's bits
    W = synth.integers((N, K), dtype, 0, 21, -1, 1)
    b = synth.integers((N,), dtype, 0, 22, -4, 4)
    x = synth.integers((B, K), dtype, 0, 23, -1, 1)
    Wt = _tiled(ctx, W)
    ref = oracle.linear(x, W, b, dtype)
    y = _run(ctx, x, Wt, N, dtype, b)
    assert np.array_equal(y.view(np.uint32), ref.view(np.uint32))
    if (dtype == synth.F16 and K <= 2040) or (dtype == synth.BF16 and K <= 248):  # exact in the 16-bit type too
        y16 = _run(ctx, x, Wt, N, dtype, b, y_f32=False)
        assert np.array_equal(y16, synth.encode(ref, dtype))


@pytest.mark.parametrize("N,K", [(300, 4096), (64, 16384)])
def test_linear_tiled_batch_rows_independent(ctx, N, K):
    # the matrix core computes each column (batch row) on its own: a row's bits do not
    # depend on the batch size or on the other rows, with or without the split over K
    dtype = synth.F16
    W = synth.normal((N, K), dtype, 0, 31, 0, 0.02)
    b = synth.normal((N,), dtype, 0, 32, 0, 0.02)
    x = synth.normal((8, K), dtype, 0, 33)
    Wt = _tiled(ctx, W)
    y8 = _run(ctx, x, Wt, N, dtype, b)
    for B in (1, 2, 5):
        for r0 in range(0, 8 - B + 1, 3):
            y = _run(ctx, np.ascontiguousarray(x[r0:r0 + B]), Wt, N, dtype, b)
            assert np.array_equal(y.view(np.uint32), y8[r0:r0 + B].view(np.uint32)), (B, r0)


def test_linear_tiled_split_counters_reset_between_calls(ctx):
    # a split launch leaves its arrival counters at zero: repeated calls, with batch and
    # shape changes in between, keep giving the same bits
    dtype = synth.F16
    shapes = [(64, 16384), (130, 8192), (16, 36864)]
    data = []
    for i, (N, K) in enumerate(shapes):
        W = synth.normal((N, K), dtype, 0, 40 + i, 0, 0.02)
        x = synth.normal((8, K), dtype, 0, 50 + i)
        data.append((x, _tiled(ctx, W), N))
    first = [_run(ctx, x, Wt, N, dtype) for x, Wt, N in data]
    for rep in range(3):
        for (x, Wt, N), f in zip(data, first):
            y = _run(ctx, np.ascontiguousarray(x[:1 + rep]), Wt, N, dtype)
            assert np.array_equal(y.view(np.uint32), f[:1 + rep].view(np.uint32))


def test_linear_tiled_no_bias(ctx):
    dtype, N, K = synth.BF16, 200, 512
    W = synth.normal((N, K), dtype, 0, 61, 0, 0.02)
    x = synth.normal((2, K), dtype, 0, 62)
    y = _run(ctx, x, _tiled(ctx, W), N, dtype)
    assert rel_err(y, oracle.linear(x, W, None, dtype)) <= TOL


def test_linear_tiled_argument_errors(ctx):
    dtype, N, K = synth.F16, 32, 64
    W = synth.normal((N, K), dtype, 0, 71, 0, 0.02)
    Wt = _tiled(ctx, W)
    x = torch_dev_from_np(synth.normal((1, K), dtype, 0, 72))
    y = torch.empty((9, N), dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    call = lambda *a: hg.hetegen_linear_tiled_status(ctx, *a)
    assert call(x.data_ptr(), 0, K, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    assert call(x.data_ptr(), 9, K, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    assert call(x.data_ptr(), 1, 60, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    assert call(x.data_ptr(), 1, K, Wt.data_ptr(), 0, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_INVALID_ARG
    assert call(0, 1, K, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_INVALID_ARG
    assert call(x.data_ptr(), 1, K, Wt.data_ptr(), N, hg.F32, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    assert call(x.data_ptr(), 1, K, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.BF16, s) == hg.ERR_UNSUPPORTED
    assert call(x.data_ptr() + 2, 1, K, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    # x of 2^30 elements or more: refused before anything is read (x is read through a
    # buffer descriptor with 32-bit offsets)
    for c in (call, lambda *a: hg.hetegen_linear_tiled_noalloc_status(ctx, *a)):
        assert c(x.data_ptr(), 8, 1 << 27, Wt.data_ptr(), N, dtype, 0, y.data_ptr(), hg.F32, s) == hg.ERR_UNSUPPORTED
    assert hg.hetegen_tiled_bytes(0, K) == 0 and hg.hetegen_tiled_bytes(N, 60) == 0
    with pytest.raises(hg.HetegenError):
        hg.hetegen_tile_weights(ctx, Wt.data_ptr(), N, 60, Wt.data_ptr(), s)
