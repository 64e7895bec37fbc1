"""GPU parity of decode steps at the OPT hidden sizes, through the C ABI.

The LayerNorm in front of qkv and fc1 has four implementations, chosen by batch size,
placement and hidden size H: fused into the batch-1 GEMV with the row in registers
(H = 512 * NC, NC in {1, 2, 4, 5, 8, 10, 14}), fused into the workgroup GEMV's LDS
prologue (the row-major copy at batch 1, other H), and materialised by the LayerNorm
kernel with the row in registers, NI = ceil(H / 2048) 16-byte chunks per thread (the
matrix-core tiles of models for batches of 2 or more, and every linear with CPU rows or
streamed rows).  All of them
form the same sums in the same order, so on the same input rows they must give the
same bits; each step is also checked teacher-forced against the oracle.  The hidden
sizes span every NC and NI instantiation (OPT-1.3B 2048 ... OPT-175B 12288 and the
largest supported, 16384), in fp16 and bf16.

The OPT-30B and OPT-66B layer tests run one decoder layer at the full shapes of the
heterogeneous workloads (hidden 7168 / FFN 28672 fp16, hidden 9216 / FFN 36864 bf16)
with CPU rows and streamed rows, at their batch sizes.
"""
import numpy as np
import pytest

import synth
from gpu_model import Model

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")


@pytest.fixture(scope="module")
def ctx():
    c = hg.hetegen_create(0, chunk_bytes=8 << 20, ring_depth=8)
    yield c
    hg.hetegen_destroy(c)


def _qkv_input(m, tr, B):
    """The traced input of layer 0's qkv (the LayerNorm of the step input)."""
    return m.split_trace(tr, B)[0][2]


# hidden size: NC of the register-LayerNorm GEMV at batch 1 (0: not a multiple of 512 or
# not instantiated), NI of the LayerNorm kernel
HIDDEN = [(1024, 2, 1), (2048, 4, 1), (2560, 5, 2), (4096, 8, 2), (5120, 10, 3), (7168, 14, 4), (9216, 0, 5),
          (12288, 0, 8), (16384, 0, 8)]


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("H,nc,ni", HIDDEN)
def test_layernorm_paths_agree_at_hidden_size(ctx, dtype, H, nc, ni):
    F = H  # one layer, F = H keeps the weights at 12 H^2 bytes
    sample = None if H <= 5120 else 256
    x = synth.normal((8, H), dtype, 0, synth.act_id(0))
    ln_in = {}
    # row-major model: batch 1 (register or LDS LayerNorm fused in the GEMV), resident
    m = Model(ctx, 1, H, F, dtype, 0.0, 1, max_batch=1)
    weights = (m.W, m.b)
    try:
        for B in (1,):
            xb = np.ascontiguousarray(x[:B])
            out, tr = m.step(xb, trace=True)
            last, _ = m.check_teacher_forced(xb, tr, sample=sample)
            assert np.array_equal(out, last)
            ln_in[("fused", B)] = _qkv_input(m, tr, B)
        # models for batches of 2 or more, batches 2 and 8: LayerNorm kernel (NI), matrix-core GEMV
        t = Model(ctx, 1, H, F, dtype, 0.0, 1, max_batch=8, weights=weights)
        try:
            for B in (8, 2):
                xb = np.ascontiguousarray(x[:B])
                out, tr = t.step(xb, trace=True)
                last, _ = t.check_teacher_forced(xb, tr, sample=sample)
                assert np.array_equal(out, last)
                ln_in[("kernel", B)] = _qkv_input(t, tr, B)
        finally:
            t.free()
        # CPU rows and streamed rows: LayerNorm kernel with the host hand-off
        h = Model(ctx, 1, H, F, dtype, 0.4, 0, max_batch=2, weights=weights)
        try:
            xb = np.ascontiguousarray(x[:2])
            out, tr = h.step(xb, trace=True)
            last, _ = h.check_teacher_forced(xb, tr, sample=sample)
            assert np.array_equal(out, last)
            ln_in[("split", 2)] = _qkv_input(h, tr, 2)
        finally:
            h.free()
    finally:
        m.free()
    # the same input rows give the same normalised bits on every path
    ref = ln_in[("kernel", 8)]
    for (path, B), v in ln_in.items():
        assert np.array_equal(v, ref[:B]), (path, B)


@pytest.mark.parametrize("B", [1, 4])
@pytest.mark.parametrize("mode", ["split", "streamed"])
def test_opt30b_layer_teacher_forced(ctx, B, mode):
    # one OPT-30B-shaped layer (hidden 7168, FFN 28672, fp16) in pinned host memory:
    # CPU rows plus streamed rows at fractions near the planner's, or every row streamed
    dtype, H, F = synth.F16, 7168, 28672
    alpha = [0.85, 0.8, 0.86, 0.84] if mode == "split" else 0.0
    m = Model(ctx, 1, H, F, dtype, alpha, 0, max_batch=4)
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        last, worst = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
        assert np.array_equal(m.step(x), out)
        print("OPT-30B layer %s B=%d: worst relative error %.3g" % (mode, B, worst))
    finally:
        m.free()


@pytest.mark.parametrize("B", [1, 8])
def test_opt66b_layer_bf16_teacher_forced(ctx, B):
    # one OPT-66B-shaped layer (hidden 9216, FFN 36864, bf16) in host memory, half of the
    # rows on the CPU and half streamed
    dtype, H, F = synth.BF16, 9216, 36864
    m = Model(ctx, 1, H, F, dtype, 0.5, 0, max_batch=8)
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        last, worst = m.check_teacher_forced(x, tr, sample=None if B == 1 else 512)
        assert np.array_equal(out, last)
        print("OPT-66B layer B=%d: worst relative error %.3g" % (B, worst))
    finally:
        m.free()


@pytest.mark.parametrize("H,dtype", [(7168, synth.F16), (9216, synth.BF16)])
@pytest.mark.parametrize("partials", ["default", "1"])
def test_large_hidden_layernorm_partials_choice(ctx, H, dtype, partials):
    # two resident layers (F = H) in tile order at batch 8: above H = 6144 the library
    # normalises qkv and fc1 after LayerNorm launches; HETEGEN_LN_PARTIALS=1 makes it combine
    # the partials of out / fc2 (H / 16 of them per batch row) instead.  Both pass the
    # teacher-forced check, and agree within the tolerance per layer.
    import os
    from common import TOL, U_ACT, rel_err
    import oracle
    L, F, B = 2, H, 8
    old = os.environ.get("HETEGEN_LN_PARTIALS")
    if partials != "default":
        os.environ["HETEGEN_LN_PARTIALS"] = partials
    try:
        m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=8)
    finally:
        if old is None:
            os.environ.pop("HETEGEN_LN_PARTIALS", None)
        else:
            os.environ["HETEGEN_LN_PARTIALS"] = old
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(7))
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr, sample=256)
        assert np.array_equal(out, last)
        for b in (3, 2):
            assert np.array_equal(m.step(np.ascontiguousarray(x[:b])), out[:b]), b
        ref = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1, weights=(m.W, m.b))
        try:
            want = ref.step(x[:1])
        finally:
            ref.free()
        assert rel_err(oracle.decode(out[:1], dtype), oracle.decode(want, dtype), floor=1.0) <= L * (TOL + U_ACT[dtype])
    finally:
        m.free()


def test_hidden_size_above_limit_rejected(ctx):
    W = [0] * 4
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_model_create(ctx, 1, 16392, 64, synth.F16, W, None, [0.0] * 4, [0] * 4, 1)
    assert e.value.status in (hg.ERR_UNSUPPORTED, hg.ERR_INVALID_ARG)
