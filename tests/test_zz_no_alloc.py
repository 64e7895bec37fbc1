"""GPU test of hetegen_linear_tiled_noalloc: the allocation-free variant of
hetegen_linear_tiled (split-K partials and counters in the library's fixed scratch)
must give the bits of hetegen_linear_tiled, call after call, including a smaller
call after a larger one, and refuse shapes beyond its scratch without launching."""
import numpy as np
import pytest

import oracle
import synth
from common import TOL, np_from_dev, rel_err, torch_dev_from_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")


@pytest.fixture(scope="module")
def ctx():
    c = hg.hetegen_create(0)
    yield c
    hg.hetegen_destroy(c)


def _case(ctx, N, K, B, dtype, tid):
    W = synth.normal((N, K), dtype, 0, tid, 0, 0.02)
    b = synth.normal((N,), dtype, 0, tid + 1, 0, 0.02)
    x = synth.normal((B, K), dtype, 0, tid + 2)
    Wd = torch_dev_from_np(W)
    Wt = torch.empty((hg.hetegen_tiled_bytes(N, K) // 2,), dtype=torch.int16, device="cuda")
    hg.hetegen_tile_weights(ctx, Wd.data_ptr(), N, K, Wt.data_ptr(), torch.cuda.current_stream().cuda_stream)
    return dict(N=N, K=K, B=B, dtype=dtype, W=W, b=b, x=x, Wt=Wt, xd=torch_dev_from_np(x), bd=torch_dev_from_np(b))


def _call(ctx, c, fn):
    y = torch.full((c["B"], c["N"]), float("nan"), dtype=torch.float32, device="cuda")
    fn(ctx, c["xd"].data_ptr(), c["B"], c["K"], c["Wt"].data_ptr(), c["N"], c["dtype"], c["bd"].data_ptr(),
       y.data_ptr(), hg.F32, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return np_from_dev(y, np.float32)


def test_noalloc_matches_allocating_entry_point_call_after_call(ctx):
    # a large split call (fc2 of OPT-6.7B at batch 8, 4 splits), then a smaller one (2 splits,
    # batch 2), then an unsplit one, then the large one again: each gives the allocating
    # entry point's bits and stays within the tolerance of the oracle
    cases = [_case(ctx, 4096, 16384, 8, synth.F16, 100), _case(ctx, 130, 8192, 2, synth.BF16, 110),
             _case(ctx, 300, 1024, 3, synth.F16, 120)]
    for c in cases + cases[:1]:
        ref_lib = _call(ctx, c, hg.hetegen_linear_tiled)
        got = _call(ctx, c, hg.hetegen_linear_tiled_noalloc)
        assert np.array_equal(got.view(np.uint32), ref_lib.view(np.uint32)), (c["N"], c["K"], c["B"])
        ref = oracle.linear(c["x"], c["W"], c["b"], c["dtype"]).astype(np.float64)
        assert rel_err(got, ref) <= TOL


def test_noalloc_refuses_shapes_beyond_its_scratch(ctx):
    # 16400 rows at K = 36864 and batch 8 need 1025 * 8 * 16 * 8 = 1049600 partial floats,
    # above the 1048576 of the fixed scratch; 16384 rows fit exactly.  The buffers are
    # full-sized, so the refusal is the entry point's check, not a lucky launch.
    K, B, dt = 36864, 8, synth.F16
    x = torch.zeros((B, K), dtype=torch.int16, device="cuda")
    Wt = torch.zeros((hg.hetegen_tiled_bytes(16400, K) // 2,), dtype=torch.int16, device="cuda")
    y = torch.zeros((B, 16400), dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    rc = hg.hetegen_linear_tiled_noalloc_status(ctx, x.data_ptr(), B, K, Wt.data_ptr(), 16400, dt, 0, y.data_ptr(),
                                                hg.F32, s)
    assert rc == hg.ERR_UNSUPPORTED
    assert "scratch" in hg.hetegen_last_error(ctx)
    rc = hg.hetegen_linear_tiled_noalloc_status(ctx, x.data_ptr(), B, K, Wt.data_ptr(), 16384, dt, 0, y.data_ptr(),
                                                hg.F32, s)
    assert rc == hg.OK
    torch.cuda.synchronize()
    assert np.all(np_from_dev(y[:, :16384], np.float32) == 0.0)
