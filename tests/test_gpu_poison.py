"""GPU race checks with poisoned staging (HETEGEN_POISON): every device staging slot,
pinned staging buffer and host hand-off buffer is filled with all-ones bits (NaN in
fp16, bf16 and binary32) before each reuse.  A stale or early read would then give NaN
instead of an old value that might happen to be right, so integer-input results must
still equal the oracle bit for bit, and decode steps must give the bits of an
unpoisoned context."""
import os

import numpy as np
import pytest

import oracle
import synth
from common import Pageable, Pinned, torch_dev_from_np
from gpu_model import Model

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")


def _create(**kw):
    old = os.environ.get("HETEGEN_POISON")
    os.environ["HETEGEN_POISON"] = "1"
    try:
        return hg.hetegen_create(0, **kw)
    finally:
        if old is None:
            del os.environ["HETEGEN_POISON"]
        else:
            os.environ["HETEGEN_POISON"] = old


@pytest.fixture(scope="module")
def pctx():
    # 4 KiB chunks, two device slots and two pinned staging buffers: every buffer is reused
    # as often as possible; chunks above 1 MiB would split over the pin team, so a second
    # context uses 3 MiB chunks for that
    cs = {"tiny": _create(chunk_bytes=4096, ring_depth=2, pin_threads=3, pin_ring=2),
          "team": _create(chunk_bytes=3 << 20, ring_depth=2, pin_threads=4, pin_ring=2)}
    yield cs
    for c in cs.values():
        hg.hetegen_destroy(c)


def _linear(ctx, x, W_ptr, N, K, dtype, bias_ptr, bias_np, alpha, W_dev=0):
    B = x.shape[0]
    xd = torch_dev_from_np(x)
    bd = torch_dev_from_np(bias_np)
    y = torch.full((B, N), float("nan"), dtype=torch.float32, device="cuda")
    hg.hetegen_linear(ctx, xd.data_ptr(), B, K, W_ptr, W_dev, N, dtype, bias_ptr, bd.data_ptr(), alpha, y.data_ptr(),
                      hg.F32, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("which", ["tiny", "team"])
@pytest.mark.parametrize("pageable", [False, True])
@pytest.mark.parametrize("B", [1, 8])
def test_integer_inputs_bit_exact_with_poisoned_staging(pctx, which, pageable, B):
    ctx = pctx[which]
    dtype, K, N = synth.F16, 1024 if which == "team" else 256, 3001
    Wp = Pinned(hg, ctx, (N, K), np.uint16)
    bias = Pinned(hg, ctx, (N,), np.uint16)
    try:
        synth.fill_int_ptr(Wp.ptr, N * K, dtype, 5, 2, -1, 1)
        synth.fill_int_ptr(bias.ptr, N, dtype, 5, 3, -4, 4)
        x = synth.integers((B, K), dtype, 5, 1, -1, 1)
        W_ptr = Wp.ptr
        if pageable:
            Wq = Pageable((N, K), np.uint16)
            Wq.a[:] = Wp.a
            W_ptr = Wq.ptr
        ref = oracle.linear(x, Wp.a, bias.a, dtype)
        for alpha in (0.0, 0.3, 0.77, 1.0, 0.0):
            y = _linear(ctx, x, W_ptr, N, K, dtype, bias.ptr, bias.a, alpha)
            assert not np.isnan(y).any(), alpha
            assert np.array_equal(y, ref), alpha
    finally:
        Wp.free()
        bias.free()


@pytest.mark.parametrize("mode", ["streamed", "hetero"])
def test_decode_steps_same_bits_with_poisoned_staging(pctx, mode):
    # the same 3-layer stack on an unpoisoned and a poisoned context: identical outputs
    dtype, L, H, F = synth.F16, 3, 256, 1024
    alpha = 0.0 if mode == "streamed" else [0.0, 0.3, 1.0, 0.5, 0.0, 0.0, 0.7, 0.25, 0.1, 1.0, 0.0, 0.6]
    plain = hg.hetegen_create(0, chunk_bytes=4096, ring_depth=2)
    try:
        ref_m = Model(plain, L, H, F, dtype, alpha, 0, max_batch=4)
        m = Model(pctx["tiny"], L, H, F, dtype, alpha, 0, max_batch=4, weights=(ref_m.W, ref_m.b))
        try:
            for B in (1, 4):
                x = synth.normal((B, H), dtype, 0, synth.act_id(B))
                want = ref_m.step(x)
                for _ in range(2):
                    assert np.array_equal(m.step(x), want), B
        finally:
            m.free()
            ref_m.free()
    finally:
        hg.hetegen_destroy(plain)
