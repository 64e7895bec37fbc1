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
    # a large split call (fc2 of OPT-13B at batch 8, 4 splits), then a smaller one (8 splits,
    # batch 2), then an unsplit one, then the large one again: each gives the allocating
    # entry point's bits and stays within the tolerance of the oracle
    cases = [_case(ctx, 5120, 20480, 8, synth.F16, 100), _case(ctx, 130, 8192, 2, synth.BF16, 110),
             _case(ctx, 300, 1024, 3, synth.F16, 120)]
    for c in cases + cases[:1]:
        ref_lib = _call(ctx, c, hg.hetegen_linear_tiled)
        got = _call(ctx, c, hg.hetegen_linear_tiled_noalloc)
        assert np.array_equal(got.view(np.uint32), ref_lib.view(np.uint32)), (c["N"], c["K"], c["B"])
        ref = oracle.linear(c["x"], c["W"], c["b"], c["dtype"]).astype(np.float64)
        assert rel_err(got, ref) <= TOL


def _status(ctx, N, K, B, dt=synth.F16):
    # full-sized zero buffers, so that an accepted call is a valid launch and a refusal is
    # the entry point's check, not a lucky launch
    x = torch.zeros((B, K), dtype=torch.int16, device="cuda")
    Wt = torch.zeros((hg.hetegen_tiled_bytes(N, K) // 2,), dtype=torch.int16, device="cuda")
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    rc = hg.hetegen_linear_tiled_noalloc_status(ctx, x.data_ptr(), B, K, Wt.data_ptr(), N, dt, 0, y.data_ptr(),
                                                hg.F32, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return rc, y


def test_noalloc_refuses_shapes_beyond_its_scratch(ctx):
    # The split over K (one workgroup per 16-row tile unless that loads the compute units
    # more than 1.15x unevenly) on a 256-CU device: [16400, 36864] is 1025 row tiles in 2
    # splits, 1025 * 2 * 16 * 8 = 262400 partial floats at batch 8, and [4112, 36864] 257 row
    # tiles in 8 splits, 263168, both above the 262144 of the fixed scratch; [14240, 36864],
    # 890 row tiles in 2 splits, needs 227840 and runs.
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the shapes are chosen for a 256-CU device")
    for N in (16400, 4112):
        rc, _ = _status(ctx, N, 36864, 8)
        assert rc == hg.ERR_UNSUPPORTED, N
        assert "scratch" in hg.hetegen_last_error(ctx)
    rc, y = _status(ctx, 14240, 36864, 8)
    assert rc == hg.OK
    assert np.all(np_from_dev(y, np.float32) == 0.0)
    # at batch 4 the 1025-tile shape needs half as much and runs
    rc, y = _status(ctx, 16400, 36864, 4)
    assert rc == hg.OK
    assert np.all(np_from_dev(y, np.float32) == 0.0)
