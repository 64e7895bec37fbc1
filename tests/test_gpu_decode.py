"""GPU parity of hetegen_decode_step (teacher-forced per linear) through the C ABI.

Each linear's traced input is fed to the oracle linear; the oracle output, finished
with the same ReLU / residual sum in float64, must match the traced output within
2e-3 + the activation type's rounding.  Placement of the value slice and of the
ReLU output is checked bit for bit; the LayerNorm inputs are checked against the
oracle's LayerNorm.  The graph replay of an all-resident step must be bit-identical
to the eager step.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import attention as oat
from oracle import decode_step as ods
from common import TOL, U_ACT, Pinned, np_from_dev, rel_err, torch_dev_from_np
from gpu_model import NAMES, Model, shapes

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")

@pytest.fixture(scope="module")
def ctx():
    c = hg.hetegen_create(0, chunk_bytes=1 << 20, ring_depth=4)
    yield c
    hg.hetegen_destroy(c)


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B", [1, 3, 8])
@pytest.mark.parametrize("mode", ["resident", "streamed", "hetero", "mixed"])
def test_small_stack_teacher_forced(ctx, dtype, B, mode):
    L, H, F = 3, 256, 1024
    if mode == "resident":
        alpha, res = 0.0, 1
    elif mode == "streamed":
        alpha, res = 0.0, 0
    elif mode == "hetero":
        alpha, res = 0.45, 0
    else:  # per-linear mix of resident, streamed, split and CPU-only linears
        alpha = [0.0, 0.3, 1.0, 0.5, 0.0, 0.0, 0.7, 0.25, 0.1, 1.0, 0.0, 0.6]
        res = [1, 0, 0, 0, 0, 1, 0, 1, 0, 0, 1, 0]
    m = Model(ctx, L, H, F, dtype, alpha, res)
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
        # the untraced step (graph replay when all-resident) gives the same bits
        assert np.array_equal(m.step(x), out)
        assert np.array_equal(m.step(x), out)
    finally:
        m.free()


def test_end_to_end_drift_is_small(ctx):
    # not teacher-forced: the oracle runs the whole stack from the same input
    dtype, L, H, F = synth.F16, 4, 256, 1024
    m = Model(ctx, L, H, F, dtype, 0.3, 0)
    try:
        x = synth.normal((2, H), dtype, 0, synth.act_id(1))
        out = m.step(x)
        layers = [{n: (m.W[4 * l + i].a, m.b[4 * l + i].a) for i, n in enumerate(NAMES)} for l in range(L)]
        ref, _ = ods.decode_step(x, layers, H, dtype)
        assert rel_err(oracle.decode(out, dtype), oracle.decode(ref, dtype)) <= 2e-2
    finally:
        m.free()


def test_graph_replays_match_eager(ctx):
    dtype, L, H, F = synth.F16, 2, 512, 2048
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        xs = [synth.normal((1, H), dtype, 0, synth.act_id(t)) for t in range(3)]
        eager = [m.step(x, trace=True)[0] for x in xs]   # tracing forces the eager path
        for _ in range(3):
            for x, e in zip(xs, eager):
                assert np.array_equal(m.step(x), e)
    finally:
        m.free()


def test_set_alpha_changes_split_not_result(ctx):
    dtype, L, H, F = synth.F16, 1, 256, 1024
    m = Model(ctx, L, H, F, dtype, 0.0, 0)
    try:
        x = synth.normal((2, H), dtype, 0, synth.act_id(2))
        outs = []
        for a in (0.0, 0.5, 1.0):
            hg.hetegen_model_set_alpha(m.m, [a] * 4)
            o, tr = m.step(x, trace=True)
            m.check_teacher_forced(x, tr)
            outs.append(oracle.decode(o, dtype))
        for o in outs[1:]:
            assert rel_err(o, outs[0]) <= 2 * (TOL + U_ACT[dtype])
    finally:
        m.free()


@pytest.mark.parametrize("B", [1, 4])
def test_opt67b_shape_two_layers_resident(ctx, B):
    # OPT-6.7B decoder-layer shapes at full size (two of the 32 layers)
    dtype, L, H, F = synth.F16, 2, 4096, 16384
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=4)
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
        assert np.array_equal(m.step(x), out)
    finally:
        m.free()


def test_opt67b_full_model_resident_as_benchmarked(ctx):
    # the benchmark's workload itself: all 32 OPT-6.7B-shaped layers resident, batch 1, the
    # default execution mode; every one of the 128 linears checked against the oracle on the
    # input it was given, and the untraced step gives the same bits
    dtype, L, H, F = synth.F16, 32, 4096, 16384
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        assert hg.hetegen_model_last_exec(m.m) == 3  # eager per-linear launches
        last, worst = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
        assert np.array_equal(m.step(x), out)
        print("32 layers: worst per-linear relative error %.3g" % worst)
    finally:
        m.free()


def test_opt67b_full_model_batched_as_benchmarked(ctx):
    # the batched workload as benchmarked: all 32 OPT-6.7B-shaped layers resident in a model
    # created for batch 8 (matrix-core tiles, k-major on a 256-CU device, no K split, LayerNorm
    # partials between the linears), at batches 8, 3 and 2; every linear checked against the
    # oracle on 256 sampled output rows of the input it was given, the untraced step gives the
    # same bits, and a batch row's bits do not depend on the batch size
    dtype, L, H, F = synth.F16, 32, 4096, 16384
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=8)
    try:
        layouts = hg.hetegen_model_layouts(m.m)
        assert layouts & hg.LAYOUT_TILED
        if torch.cuda.get_device_properties(0).multi_processor_count == 256:
            assert layouts & hg.LAYOUT_KMAJOR
        x = synth.normal((8, H), dtype, 0, synth.act_id(5))
        out8, tr = m.step(x, trace=True)
        assert hg.hetegen_model_last_exec(m.m) == 3  # eager per-linear launches
        last, worst = m.check_teacher_forced(x, tr, sample=256)
        assert np.array_equal(out8, last)
        assert np.array_equal(m.step(x), out8)
        for B in (3, 2):
            xb = np.ascontiguousarray(x[:B])
            out, tr = m.step(xb, trace=True)
            last, _ = m.check_teacher_forced(xb, tr, sample=256)
            assert np.array_equal(out, last)
            assert np.array_equal(out, out8[:B]), B
        print("32 layers at batch 8: worst per-linear relative error %.3g" % worst)
    finally:
        m.free()


def test_opt13b_shape_one_layer_hetero(ctx):
    dtype, L, H, F = synth.F16, 1, 5120, 20480
    m = Model(ctx, L, H, F, dtype, [0.62, 0.6, 0.63, 0.61], 0, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(0))
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
    finally:
        m.free()


def _model_with_env(ctx, env, *args, **kw):
    import os
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        return Model(ctx, *args, **kw)
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B,max_batch,dual", [(1, 1, True), (1, 2, True), (2, 2, True), (2, 4, True), (4, 4, True),
                                              (1, 8, True), (1, 8, False), (5, 8, True), (8, 8, False)])
def test_exec_modes_bit_identical(ctx, dtype, B, max_batch, dual):
    # persistent (one cooperative launch, grid barriers), graph replay and eager
    # per-linear launches compute every output row the same way; the persistent step runs
    # the row-major copy at batch 1 only (models for batches of 2 or more keep it beside
    # the tile order when memory allows, HETEGEN_DUAL_LAYOUT=0 keeps tiles only)
    L, H, F = 3, 512, 2048
    m = _model_with_env(ctx, {} if dual else {"HETEGEN_DUAL_LAYOUT": "0"}, L, H, F, dtype, 0.0, 1,
                        max_batch=max_batch)
    layouts = hg.hetegen_model_layouts(m.m) & ~(hg.LAYOUT_KMAJOR | hg.LAYOUT_SEGMAJOR)
    assert layouts == (hg.LAYOUT_ROWMAJOR if max_batch < 2 else
                       hg.LAYOUT_TILED | (hg.LAYOUT_ROWMAJOR if dual else 0))
    try:
        xs = [synth.normal((B, H), dtype, 0, synth.act_id(t)) for t in range(3)]
        outs = {}
        if not layouts & hg.LAYOUT_ROWMAJOR:
            with pytest.raises(hg.HetegenError) as e:
                hg.hetegen_model_set_exec(m.m, hg.EXEC_PERSISTENT)
            assert e.value.status == hg.ERR_UNSUPPORTED
        persistent = bool(layouts & hg.LAYOUT_ROWMAJOR) and B == 1
        modes = (hg.EXEC_EAGER, hg.EXEC_GRAPH, hg.EXEC_PERSISTENT, hg.EXEC_AUTO) if persistent else \
            (hg.EXEC_EAGER, hg.EXEC_GRAPH, hg.EXEC_AUTO)
        for mode in modes:
            hg.hetegen_model_set_exec(m.m, mode)
            outs[mode] = [m.step(x) for x in xs] + [m.step(xs[0])]
            want = {hg.EXEC_AUTO: hg.EXEC_EAGER}.get(mode, mode)
            assert hg.hetegen_model_last_exec(m.m) == want
        for mode, o in outs.items():
            for a, b in zip(o, outs[hg.EXEC_EAGER]):
                assert np.array_equal(a, b), mode
        # and the result is the teacher-forced-checked eager result
        _, tr = m.step(xs[1], trace=True)
        last, _ = m.check_teacher_forced(xs[1], tr)
        assert np.array_equal(outs[modes[-2]][1], last)
    finally:
        m.free()


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
def test_dual_layout_runs_each_batch_on_the_matching_copy(ctx, dtype):
    # a model for batches up to 8 with both copies gives, at batch 1, the bits of a
    # row-major model and, from batch 2, the bits of a tile-only model (same weights)
    L, H, F = 2, 1024, 8192
    rm = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        dual = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=8, weights=(rm.W, rm.b))
        tiles = _model_with_env(ctx, {"HETEGEN_DUAL_LAYOUT": "0"}, L, H, F, dtype, 0.0, 1, max_batch=8,
                                weights=(rm.W, rm.b))
        try:
            order = hg.LAYOUT_KMAJOR | hg.LAYOUT_SEGMAJOR  # tile and row orders
            assert hg.hetegen_model_layouts(rm.m) & ~order == hg.LAYOUT_ROWMAJOR
            assert hg.hetegen_model_layouts(dual.m) & ~order == hg.LAYOUT_ROWMAJOR | hg.LAYOUT_TILED
            assert hg.hetegen_model_layouts(tiles.m) & ~order == hg.LAYOUT_TILED
            for B in (1, 2, 3, 8):
                x = synth.normal((B, H), dtype, 0, synth.act_id(10 + B))
                want = (rm if B == 1 else tiles).step(x)
                out, tr = dual.step(x, trace=True)
                assert np.array_equal(out, want), B
                last, _ = dual.check_teacher_forced(x, tr)
                assert np.array_equal(out, last)
            # the tile-only model at batch 1 (matrix-core GEMV) passes teacher-forced too
            x = synth.normal((1, H), dtype, 0, synth.act_id(20))
            out, tr = tiles.step(x, trace=True)
            last, _ = tiles.check_teacher_forced(x, tr)
            assert np.array_equal(out, last)
        finally:
            tiles.free()
            dual.free()
    finally:
        rm.free()


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("H,F", [(1032, 2056), (512, 2048)])
def test_tiled_layernorm_from_partials(ctx, dtype, H, F):
    # on a model in tile order, qkv (after the first layer's) and fc1 take their LayerNorm
    # from the partials that the fc2 / out before them wrote (one pair per 16 outputs and
    # batch row; H = 1032 ends in a group of 8): teacher-forced against the oracle over
    # three layers, and each batch row's bits do not depend on the batch size
    L = 3
    m = _model_with_env(ctx, {"HETEGEN_DUAL_LAYOUT": "0"}, L, H, F, dtype, 0.0, 1, max_batch=8)
    try:
        assert hg.hetegen_model_layouts(m.m) == hg.LAYOUT_TILED
        x = synth.normal((8, H), dtype, 0, synth.act_id(3))
        out8, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out8, last)
        for B in (3, 5, 1):
            assert np.array_equal(m.step(np.ascontiguousarray(x[:B])), out8[:B]), B
        # the same model with LayerNorm launches instead passes too, and the two agree
        # within the tolerance per layer, relative to each row's largest output (their
        # LayerNorm roundings differ in places, and a one-unit difference in a large
        # value carries over to the small values after it)
        k = _model_with_env(ctx, {"HETEGEN_DUAL_LAYOUT": "0", "HETEGEN_LN_PARTIALS": "0"}, L, H, F, dtype, 0.0, 1,
                            max_batch=8, weights=(m.W, m.b))
        try:
            outk, trk = k.step(x, trace=True)
            lastk, _ = k.check_teacher_forced(x, trk)
            assert np.array_equal(outk, lastk)
            assert rel_err(oracle.decode(out8, dtype), oracle.decode(outk, dtype), floor=1.0) <= \
                L * (TOL + U_ACT[dtype])
        finally:
            k.free()
    finally:
        m.free()


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
def test_tile_order_does_not_change_bits(ctx, dtype):
    # tiles k-major (k-tile kt of row tile rt at kt * row tiles + rt) or in row-tile order:
    # every wavefront adds the same tiles in the same order, so the bits are the same at
    # every batch, and they pass the teacher-forced check.  On a 256-CU device the library
    # keeps fc1 [4096, 1024] (256 workgroups) and fc2 [1024, 4096] (64 row tiles in 4 K-splits)
    # k-major and qkv and out in row-tile order.
    L, H, F = 2, 1024, 4096
    env = {"HETEGEN_DUAL_LAYOUT": "0"}
    rule = _model_with_env(ctx, env, L, H, F, dtype, 0.0, 1, max_batch=8)
    try:
        rows = _model_with_env(ctx, dict(env, HETEGEN_TILE_KORDER="0"), L, H, F, dtype, 0.0, 1, max_batch=8,
                               weights=(rule.W, rule.b))
        kmaj = _model_with_env(ctx, dict(env, HETEGEN_TILE_KORDER="1"), L, H, F, dtype, 0.0, 1, max_batch=8,
                               weights=(rule.W, rule.b))
        try:
            assert hg.hetegen_model_layouts(rows.m) == hg.LAYOUT_TILED
            assert hg.hetegen_model_layouts(kmaj.m) == hg.LAYOUT_TILED | hg.LAYOUT_KMAJOR
            if torch.cuda.get_device_properties(0).multi_processor_count == 256:
                assert hg.hetegen_model_layouts(rule.m) == hg.LAYOUT_TILED | hg.LAYOUT_KMAJOR
            for B in (8, 3, 1):
                x = synth.normal((B, H), dtype, 0, synth.act_id(30 + B))
                want = rows.step(x)
                assert np.array_equal(kmaj.step(x), want), B
                out, tr = rule.step(x, trace=True)
                assert np.array_equal(out, want), B
                if B == 8:
                    last, _ = rule.check_teacher_forced(x, tr)
                    assert np.array_equal(out, last)
        finally:
            kmaj.free()
            rows.free()
    finally:
        rule.free()


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
def test_segment_major_rows_keep_bits(ctx, dtype):
    # fc2 [1024, 8192] (K >= 8192, a multiple of 2048) keeps its row-major copy segment-major
    # (2048-element segment s of row r at s * N + r); qkv, out and fc1 (K = 1024) stay
    # row-major.  Eager, graph and persistent steps at batch 1 give the bits of a model with
    # plain row-major copies, and pass the teacher-forced check; a model created for batch 8
    # (both copies, tiles made from the row-major staging) does at batches 1 and 8.
    L, H, F = 2, 1024, 8192
    plain = _model_with_env(ctx, {"HETEGEN_SEGMAJOR": "0"}, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        seg = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1, weights=(plain.W, plain.b))
        dual = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=8, weights=(plain.W, plain.b))
        try:
            assert hg.hetegen_model_layouts(plain.m) == hg.LAYOUT_ROWMAJOR
            assert hg.hetegen_model_layouts(seg.m) == hg.LAYOUT_ROWMAJOR | hg.LAYOUT_SEGMAJOR
            assert hg.hetegen_model_layouts(dual.m) & hg.LAYOUT_SEGMAJOR
            x = synth.normal((1, H), dtype, 0, synth.act_id(40))
            want = plain.step(x)
            for mode in (hg.EXEC_EAGER, hg.EXEC_GRAPH, hg.EXEC_PERSISTENT):
                hg.hetegen_model_set_exec(seg.m, mode)
                assert np.array_equal(seg.step(x), want), mode
                assert hg.hetegen_model_last_exec(seg.m) == mode
            hg.hetegen_model_set_exec(seg.m, hg.EXEC_AUTO)
            out, tr = seg.step(x, trace=True)
            last, _ = seg.check_teacher_forced(x, tr)
            assert np.array_equal(out, last) and np.array_equal(out, want)
            assert np.array_equal(dual.step(x), want)
            x8 = synth.normal((8, H), dtype, 0, synth.act_id(41))
            out8, tr8 = dual.step(x8, trace=True)
            last8, _ = dual.check_teacher_forced(x8, tr8)
            assert np.array_equal(out8, last8)
        finally:
            dual.free()
            seg.free()
    finally:
        plain.free()


@pytest.mark.parametrize("B", [3, 8])
def test_tiled_partials_only_between_matrix_core_linears(ctx, B):
    # a linear with CPU rows (layer 1's out) or host-resident rows (layer 2's fc2) writes no
    # partials, so the fc1 / qkv after it normalises after a LayerNorm launch, while the
    # other pairs keep the partials; stale partials would fail the teacher-forced check
    dtype, L, H, F = synth.F16, 3, 512, 2048
    alpha = [0.0] * (4 * L)
    alpha[4 * 1 + 1] = 0.3
    resident = [1] * (4 * L)
    resident[4 * 2 + 3] = 0
    m = _model_with_env(ctx, {"HETEGEN_DUAL_LAYOUT": "0"}, L, H, F, dtype, alpha, resident, max_batch=8)
    try:
        x = synth.normal((B, H), dtype, 0, synth.act_id(4))
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
        assert np.array_equal(m.step(x), out)
    finally:
        m.free()


def test_persistent_opt67b_shapes_two_layers(ctx):
    dtype, L, H, F = synth.F16, 2, 4096, 16384
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(0))
        hg.hetegen_model_set_exec(m.m, hg.EXEC_EAGER)
        eager = m.step(x)
        hg.hetegen_model_set_exec(m.m, hg.EXEC_PERSISTENT)
        for _ in range(3):
            assert np.array_equal(m.step(x), eager)
    finally:
        m.free()


@pytest.mark.parametrize("H", [2560, 5120, 7168])
def test_register_layernorm_hidden_sizes_bit_identical_to_persistent(ctx, H):
    # the register-LayerNorm GEMV at K = 512 * NC for NC = 5, 10, 14 (OPT-2.7B/13B/30B hidden
    # sizes) gives the workgroup kernel's bits, and matches the oracle teacher-forced
    dtype, L = synth.F16, 1
    m = Model(ctx, L, H, 4 * H, dtype, 0.0, 1, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(0))
        hg.hetegen_model_set_exec(m.m, hg.EXEC_EAGER)
        eager, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(eager, last)
        hg.hetegen_model_set_exec(m.m, hg.EXEC_PERSISTENT)
        assert np.array_equal(m.step(x), eager)
        assert hg.hetegen_model_last_exec(m.m) == hg.EXEC_PERSISTENT
    finally:
        m.free()


def test_barrier_wait_that_gives_up_is_reported(ctx):
    # a spin limit of one poll makes waits give up (outputs undefined, kernel still
    # drains); the next step on the model must report the failure
    dtype, L, H, F = synth.F16, 2, 256, 1024
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(0))
        hg.hetegen_model_set_exec(m.m, hg.EXEC_PERSISTENT, 1)
        for _ in range(4):
            m.step(x)
            try:
                m.step(x)
            except hg.HetegenError as e:
                assert e.status == hg.ERR_HIP and "barrier" in str(e)
                return
        pytest.skip("every barrier completed within one poll; the failure path was not reached")
    finally:
        m.free()


def test_forced_modes_rejected_for_split_models(ctx):
    m = Model(ctx, 1, 256, 1024, synth.F16, 0.5, 0, max_batch=1)
    try:
        with pytest.raises(hg.HetegenError) as e:
            hg.hetegen_model_set_exec(m.m, hg.EXEC_PERSISTENT)
        assert e.value.status == hg.ERR_UNSUPPORTED
        hg.hetegen_model_set_exec(m.m, hg.EXEC_EAGER)
    finally:
        m.free()


def test_step_alpha_benchmark_refines_and_keeps_parity(ctx):
    dtype, L, H, F = synth.F16, 2, 1024, 4096
    m = Model(ctx, L, H, F, dtype, [0.5] * 8, 0, max_batch=1)
    try:
        x = synth.normal((1, H), dtype, 0, synth.act_id(3))
        xd = torch_dev_from_np(x)
        od = torch.empty((1, H), dtype=torch.int16, device="cuda")
        for objective in (hg.BENCH_CROSSING, hg.BENCH_WALL):
            hg.hetegen_model_set_alpha(m.m, [0.5] * 8)
            d, crossed = hg.hetegen_model_alpha_benchmark(ctx, m.m, xd.data_ptr(), od.data_ptr(), 1, 0.1, 0.05, 2, 1,
                                                          objective, torch.cuda.current_stream().cuda_stream)
            assert -0.3 - 1e-9 <= d <= 0.3 + 1e-9  # up to three brackets of +-0.1
            a = hg.hetegen_model_get_alpha(m.m, 4 * L)
            assert all(abs(v - (0.5 + d)) < 1e-12 for v in a)
        out, tr = m.step(x, trace=True)
        last, _ = m.check_teacher_forced(x, tr)
        assert np.array_equal(out, last)
    finally:
        m.free()


def test_linear_times_reported_for_heterogeneous_steps(ctx):
    dtype, L, H, F = synth.F16, 2, 256, 1024
    m = Model(ctx, L, H, F, dtype, [0.5, 0.0, 0.4, 0.3] * L, [0, 1, 0, 0] * L)
    try:
        assert hg.hetegen_model_linear_ms(m.m, 4 * L) == [0.0] * (4 * L)
        m.step(synth.normal((1, H), dtype, 0, synth.act_id(0)))
        ms = hg.hetegen_model_linear_ms(m.m, 4 * L)
        assert all(np.isfinite(v) and v > 0 for v in ms)
    finally:
        m.free()


def test_read_floor_of_resident_rows(ctx):
    dtype, L, H, F = synth.F16, 2, 512, 2048
    m = Model(ctx, L, H, F, dtype, [0.0, 0.3, 0.0, 0.0] * L, [1, 1, 0, 1] * L)
    try:
        ms = hg.hetegen_model_read_ms(ctx, m.m, 3)
        assert np.isfinite(ms) and 0 < ms < 100
    finally:
        m.free()
    m = Model(ctx, 1, H, F, dtype, 0.5, 0)  # nothing resident
    try:
        with pytest.raises(hg.HetegenError):
            hg.hetegen_model_read_ms(ctx, m.m, 3)
        with pytest.raises(hg.HetegenError):
            hg.hetegen_model_read_ms(ctx, m.m, 0)
    finally:
        m.free()


# ---- full decode steps with a KV cache (Sec. 2.1, Eq. 1) ----
def _fill_cache(m, B, P, seed=0):
    """Synthetic keys and values of positions [0, P) for every layer (stands in for a
    prefill); returns the host copies per layer ([B, P, H] bits, or None)."""
    kc, vc, keep = [], [], []
    s = torch.cuda.current_stream().cuda_stream
    for l in range(m.L):
        if P == 0:
            kc.append(None)
            vc.append(None)
            continue
        k = synth.normal((B, P, m.H), m.dtype, seed, 5000 + 2 * l)
        v = synth.normal((B, P, m.H), m.dtype, seed, 5001 + 2 * l)
        kd, vd = torch_dev_from_np(k), torch_dev_from_np(v)
        keep += [kd, vd]
        hg.hetegen_model_kv_write(m.ctx, m.m, l, B, 0, P, kd.data_ptr(), vd.data_ptr(), s)
        kc.append(k)
        vc.append(v)
    torch.cuda.synchronize()
    return kc, vc


def _attn_ref(m, kc, vc, head_dim):
    H, dt = m.H, m.dtype

    def ref(l, qkv):
        K = oat.append(kc[l], qkv[:, H:2 * H])
        V = oat.append(vc[l], qkv[:, 2 * H:3 * H])
        return oat.attend(oracle.decode(qkv[:, :H], dt), oracle.decode(K, dt), oracle.decode(V, dt), head_dim)
    return ref


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B", [1, 3])
@pytest.mark.parametrize("P", [0, 1, 63, 64, 65, 150])
@pytest.mark.parametrize("head_dim", [64, 128])
def test_kv_step_teacher_forced(ctx, dtype, B, P, head_dim):
    L, H, F = 2, 256, 512
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, 160, head_dim)
        kc, vc = _fill_cache(m, B, P)
        x = synth.normal((B, H), dtype, 0, synth.act_id(P))
        out, tr = m.step_kv(x, P, trace=True)
        last, _ = m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, head_dim))
        assert np.array_equal(out, last)
    finally:
        m.free()


def test_kv_cache_appended_and_steps_chain(ctx):
    dtype, L, H, F, B, P, D = synth.F16, 2, 256, 512, 2, 70, 64
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, 80, D)
        kc, vc = _fill_cache(m, B, P)
        layers = [{n: (m.W[4 * l + i].a, m.b[4 * l + i].a) for i, n in enumerate(NAMES)} for l in range(L)]
        x = synth.normal((B, H), dtype, 0, synth.act_id(0))
        ref_k, ref_v = list(kc), list(vc)
        s = torch.cuda.current_stream().cuda_stream
        for t in range(3):
            pos = P + t
            out, tr = m.step_kv(x, pos, trace=True)
            m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, D))
            items = m.split_trace(tr, B)
            for l in range(L):
                qkv = items[4 * l][3]
                kd = torch.zeros((B, 1, H), dtype=torch.int16, device="cuda")
                vd = torch.zeros((B, 1, H), dtype=torch.int16, device="cuda")
                hg.hetegen_model_kv_read(ctx, m.m, l, B, pos, 1, kd.data_ptr(), vd.data_ptr(), s)
                torch.cuda.synchronize()
                assert np.array_equal(np_from_dev(kd, np.uint16)[:, 0], qkv[:, H:2 * H]), (t, l)
                assert np.array_equal(np_from_dev(vd, np.uint16)[:, 0], qkv[:, 2 * H:]), (t, l)
                kc[l] = oat.append(kc[l], qkv[:, H:2 * H])
                vc[l] = oat.append(vc[l], qkv[:, 2 * H:])
            # the oracle's own chain from the same input and caches
            want, _, ref_k, ref_v = oat.decode_step_kv(x, layers, H, dtype, ref_k, ref_v, D)
            assert rel_err(oracle.decode(out, dtype), oracle.decode(want, dtype)) <= 2e-2, t
            x = out
    finally:
        m.free()


def test_kv_step_at_position_zero_equals_empty_cache_step(ctx):
    dtype, L, H, F = synth.BF16, 2, 256, 512
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        x = synth.normal((3, H), dtype, 0, synth.act_id(4))
        want = m.step(x)
        hg.hetegen_model_kv_create(ctx, m.m, 8, 128)
        assert np.array_equal(m.step_kv(x, 0), want)
    finally:
        m.free()


@pytest.mark.parametrize("mode", ["streamed", "hetero"])
def test_kv_step_with_host_linears(ctx, mode):
    dtype, L, H, F, B, P, D = synth.F16, 2, 256, 1024, 2, 100, 128
    alpha = 0.0 if mode == "streamed" else [0.4, 0.3, 0.5, 0.2] * L
    m = Model(ctx, L, H, F, dtype, alpha, 0)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, 128, D)
        kc, vc = _fill_cache(m, B, P)
        x = synth.normal((B, H), dtype, 0, synth.act_id(9))
        out, tr = m.step_kv(x, P, trace=True)
        last, _ = m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, D))
        assert np.array_equal(out, last)
    finally:
        m.free()


def test_kv_opt67b_shape_one_layer_context_512(ctx):
    # OPT-6.7B layer shapes (32 heads of 128), a 512-position context
    dtype, L, H, F, B, P, D = synth.F16, 1, 4096, 16384, 1, 512, 128
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, 576, D)
        kc, vc = _fill_cache(m, B, P)
        x = synth.normal((B, H), dtype, 0, synth.act_id(3))
        out, tr = m.step_kv(x, P, trace=True)
        m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, D))
    finally:
        m.free()


def test_kv_largest_cache_last_position(ctx):
    # the largest cache the header allows (16384 positions), decoding its last position: 256
    # chunks, all but the first 16 merged through the kernel's tail loop
    dtype, L, H, F, B, D, S = synth.F16, 1, 256, 512, 2, 128, 16384
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=2)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, S, D)
        kc, vc = _fill_cache(m, B, S - 1)
        x = synth.normal((B, H), dtype, 0, synth.act_id(S))
        out, tr = m.step_kv(x, S - 1, trace=True)
        last, _ = m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, D))
        assert np.array_equal(out, last)
        with pytest.raises(hg.HetegenError):  # one past the cache
            hg.hetegen_decode_step_kv(ctx, m.m, torch_dev_from_np(x).data_ptr(),
                                      torch.zeros((B, H), dtype=torch.int16, device="cuda").data_ptr(), B, S,
                                      torch.cuda.current_stream().cuda_stream)
    finally:
        m.free()
    m = Model(ctx, L, H, F, dtype, 0.0, 1, max_batch=1)
    try:
        with pytest.raises(hg.HetegenError) as e:  # larger than the kernel supports
            hg.hetegen_model_kv_create(ctx, m.m, S + 1, D)
        assert e.value.status == hg.ERR_INVALID_ARG
    finally:
        m.free()


def test_kv_argument_errors(ctx):
    dtype, L, H, F = synth.F16, 1, 256, 512
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        x = torch.zeros((1, H), dtype=torch.int16, device="cuda")
        o = torch.zeros((1, H), dtype=torch.int16, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        with pytest.raises(hg.HetegenError):  # no cache yet
            hg.hetegen_decode_step_kv(ctx, m.m, x.data_ptr(), o.data_ptr(), 1, 0, s)
        with pytest.raises(hg.HetegenError) as e:
            hg.hetegen_model_kv_create(ctx, m.m, 16, 96)
        assert e.value.status == hg.ERR_UNSUPPORTED
        hg.hetegen_model_kv_create(ctx, m.m, 16, 64)
        with pytest.raises(hg.HetegenError):  # only once
            hg.hetegen_model_kv_create(ctx, m.m, 16, 64)
        for pos in (-1, 16):
            with pytest.raises(hg.HetegenError) as e:
                hg.hetegen_decode_step_kv(ctx, m.m, x.data_ptr(), o.data_ptr(), 1, pos, s)
            assert e.value.status == hg.ERR_INVALID_ARG
        with pytest.raises(hg.HetegenError):  # past the cache end
            hg.hetegen_model_kv_write(ctx, m.m, 0, 1, 10, 7, x.data_ptr(), x.data_ptr(), s)
        hg.hetegen_decode_step_kv(ctx, m.m, x.data_ptr(), o.data_ptr(), 1, 15, s)
        torch.cuda.synchronize()
    finally:
        m.free()


@pytest.mark.parametrize("P", [1023, 1100, 2046, 2047, 2175])
def test_kv_long_context_merge(ctx, P):
    # more chunks than the merge requests at once (16 x 64 positions), and around the
    # switch to 128-position chunks at 2048 positions (2175: 17 chunks of 128)
    dtype, L, H, F, B, D = synth.BF16, 1, 256, 512, 2, 128
    m = Model(ctx, L, H, F, dtype, 0.0, 1)
    try:
        hg.hetegen_model_kv_create(ctx, m.m, 2200, D)
        kc, vc = _fill_cache(m, B, P)
        x = synth.normal((B, H), dtype, 0, synth.act_id(P))
        out, tr = m.step_kv(x, P, trace=True)
        last, _ = m.check_teacher_forced(x, tr, attn=_attn_ref(m, kc, vc, D))
        assert np.array_equal(out, last)
    finally:
        m.free()
