"""GPU parity of hetegen_linear against the oracle (through the C ABI).

Random inputs: max relative error <= 2e-3 on binary32 outputs, for every alpha,
resident and streamed.  Integer inputs: outputs bit-identical to the oracle and
across alphas.  Placement: a row-id encoding makes y[j] == j exactly.
"""
import numpy as np
import pytest

import oracle
import synth
from common import TOL, U_ACT, Pinned, np_from_dev, rel_err, torch_dev_from_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")

ALPHAS = [0.0, 0.25, 0.5, 1.0]


@pytest.fixture(scope="module")
def ctx():
    c = hg.hetegen_create(0)
    yield c
    hg.hetegen_destroy(c)


@pytest.fixture(scope="module")
def ctx_tiny():
    # 4 KiB chunks and a ring of 2: many chunks, slots reused as often as possible
    c = hg.hetegen_create(0, chunk_bytes=4096, ring_depth=2)
    yield c
    hg.hetegen_destroy(c)


class Problem:
    """Pinned W / bias, device x / W copy / bias for one linear."""

    def __init__(self, ctx, B, K, N, dtype, kind="normal", seed=0):
        self.ctx, self.B, self.K, self.N, self.dtype = ctx, B, K, N, dtype
        self.W = Pinned(hg, ctx, (N, K), np.uint16)
        self.bias = Pinned(hg, ctx, (N,), np.uint16)
        if kind == "normal":
            synth.fill_normal_ptr(self.W.ptr, N * K, dtype, seed, 2, 0.0, 0.02)
            synth.fill_normal_ptr(self.bias.ptr, N, dtype, seed, 3, 0.0, 0.02)
            self.x = synth.normal((B, K), dtype, seed, 1, 0.0, 1.0)
        elif kind == "int":
            synth.fill_int_ptr(self.W.ptr, N * K, dtype, seed, 2, -1, 1)
            synth.fill_int_ptr(self.bias.ptr, N, dtype, seed, 3, -4, 4)
            self.x = synth.integers((B, K), dtype, seed, 1, -1, 1)
        elif kind == "rowid":
            # x = [1, base, 0, ...], W[j, 0] = j mod base, W[j, 1] = j div base -> y[j] = j exactly
            base = 2048 if dtype == synth.F16 else 256
            j = np.arange(N)
            Wf = np.zeros((N, K), np.float32)
            Wf[:, 0] = j % base
            Wf[:, 1] = j // base
            self.W.a[:] = synth.encode(Wf, dtype)
            self.bias.a[:] = 0
            xf = np.zeros((B, K), np.float32)
            xf[:, 0] = 1.0
            xf[:, 1] = base
            self.x = synth.encode(xf, dtype)
        self.x_dev = torch_dev_from_np(self.x)
        self.W_dev = torch_dev_from_np(self.W.a)
        self.b_dev = torch_dev_from_np(self.bias.a)
        self._ref = None

    def ref(self):
        if self._ref is None:
            self._ref = oracle.linear(self.x, self.W.a, self.bias.a, self.dtype)
        return self._ref

    def run(self, alpha, resident, y_f32=True, ctx=None, bias=True):
        c = ctx or self.ctx
        ydt = hg.F32 if y_f32 else self.dtype
        y = torch.full((self.B, self.N), float("nan"), dtype=torch.float32, device="cuda") if y_f32 else \
            torch.full((self.B, self.N), -1, dtype=torch.int16, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        hg.hetegen_linear(c, self.x_dev.data_ptr(), self.B, self.K, self.W.ptr,
                          self.W_dev.data_ptr() if resident else 0, self.N, self.dtype,
                          self.bias.ptr if bias else 0, self.b_dev.data_ptr() if bias else 0, alpha,
                          y.data_ptr(), ydt, s)
        torch.cuda.synchronize()
        return y.cpu().numpy() if y_f32 else np_from_dev(y, np.uint16)

    def free(self):
        self.W.free()
        self.bias.free()


@pytest.fixture(scope="module")
def cfg1(ctx):
    # single Linear, batch 1: x fp16 [1,1024] N(0,1); W fp16 [4096,1024] N(0,0.02); bias N(0,0.02)
    p = Problem(ctx, 1, 1024, 4096, synth.F16)
    yield p
    p.free()


@pytest.mark.parametrize("resident", [True, False])
@pytest.mark.parametrize("alpha", ALPHAS)
def test_single_linear_batch1_parity(cfg1, alpha, resident):
    y = cfg1.run(alpha, resident)
    assert not np.isnan(y).any()
    assert rel_err(y, cfg1.ref()) <= TOL


@pytest.mark.parametrize("resident", [True, False])
def test_single_linear_alpha_pairs_agree(cfg1, resident):
    ys = [cfg1.run(a, resident) for a in ALPHAS]
    for a in ys[1:]:
        assert rel_err(a, ys[0]) <= TOL


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 8])
@pytest.mark.parametrize("resident", [True, False])
def test_batches_and_dtypes(ctx, dtype, B, resident):
    p = Problem(ctx, B, 1032, 777, dtype, seed=B)
    try:
        for alpha in (0.0, 0.37, 1.0):
            y = p.run(alpha, resident)
            assert rel_err(y, p.ref()) <= TOL, (alpha, rel_err(y, p.ref()))
            # act-dtype output: the same values rounded to nearest even
            ya = oracle.decode(p.run(alpha, resident, y_f32=False), dtype)
            assert rel_err(ya, p.ref()) <= TOL + U_ACT[dtype]
    finally:
        p.free()


@pytest.mark.parametrize("dtype,K", [(synth.F16, 2040), (synth.BF16, 248)])
@pytest.mark.parametrize("B", [1, 4, 8])
def test_integer_inputs_bit_exact_across_alpha(ctx, ctx_tiny, dtype, K, B):
    p = Problem(ctx, B, K, 1001, dtype, kind="int", seed=3)
    try:
        ref = p.ref()
        assert np.array_equal(ref, np.round(ref))
        for c in (ctx, ctx_tiny):
            for alpha in (0.0, 0.25, 0.5, 0.999, 1.0, 0.123):
                for resident in (True, False):
                    y = p.run(alpha, resident, ctx=c)
                    assert np.array_equal(y, ref), (alpha, resident)
                    ya = p.run(alpha, resident, y_f32=False, ctx=c)
                    assert np.array_equal(oracle.decode(ya, dtype), ref)
    finally:
        p.free()


@pytest.mark.parametrize("dtype", [synth.F16, synth.BF16])
def test_row_id_placement(ctx_tiny, dtype):
    # K = 2048: one row is 4 KiB = one chunk, so every row is its own chunk
    N = 4099 if dtype == synth.F16 else 257 * 16 + 3
    p = Problem(ctx_tiny, 2, 2048, N, dtype, kind="rowid")
    try:
        want = np.tile(np.arange(N, dtype=np.float32), (2, 1))
        assert np.array_equal(p.ref(), want)
        for alpha in (0.0, 1.0 / N, 0.5, 1.0 - 1.0 / N, 1.0, 0.3):
            for resident in (False, True):
                y = p.run(alpha, resident, bias=False)
                assert np.array_equal(y, want), (alpha, resident)
    finally:
        p.free()


@pytest.mark.parametrize("depth", [2, 3])
def test_pipeline_many_chunks_ring_depth(depth):
    c = hg.hetegen_create(0, chunk_bytes=8192, ring_depth=depth)
    p = Problem(c, 2, 1024, 3001, synth.F16, kind="int", seed=5)
    try:
        for alpha in (0.0, 0.4):
            y = p.run(alpha, False)
            assert np.array_equal(y, p.ref())
    finally:
        p.free()
        hg.hetegen_destroy(c)


def test_ragged_shapes(ctx):
    for (B, K, N) in [(1, 8, 1), (1, 8, 5), (3, 520, 63), (7, 4104, 129), (2, 16392, 33)]:
        p = Problem(ctx, B, K, N, synth.F16, seed=K)
        try:
            for alpha in (0.0, 0.5, 1.0):
                for resident in (True, False):
                    assert rel_err(p.run(alpha, resident), p.ref()) <= TOL, (B, K, N, alpha)
        finally:
            p.free()


def test_no_bias(ctx):
    p = Problem(ctx, 2, 256, 100, synth.BF16, seed=9)
    try:
        ref = oracle.linear(p.x, p.W.a, None, p.dtype)
        for alpha in (0.0, 0.5, 1.0):
            assert rel_err(p.run(alpha, False, bias=False), ref) <= TOL
    finally:
        p.free()


def test_argument_errors(ctx):
    p = Problem(ctx, 1, 64, 16, synth.F16)
    s = torch.cuda.current_stream().cuda_stream
    y = torch.empty((1, 16), dtype=torch.float32, device="cuda")
    base = [p.x_dev.data_ptr(), 1, 64, p.W.ptr, 0, 16, synth.F16, p.bias.ptr, p.b_dev.data_ptr(), 0.5,
            y.data_ptr(), hg.F32, s]

    def status(**kw):
        args = list(base)
        names = ["x", "B", "K", "W", "Wd", "N", "dt", "bh", "bd", "alpha", "y", "ydt", "s"]
        for k, v in kw.items():
            args[names.index(k)] = v
        return hg.hetegen_linear_status(ctx, *args)

    try:
        assert status() == hg.OK
        assert status(alpha=float("nan")) == hg.ERR_INVALID_ARG
        assert status(alpha=1.5) == hg.ERR_INVALID_ARG
        assert status(alpha=-0.1) == hg.ERR_INVALID_ARG
        assert status(B=0) == hg.ERR_UNSUPPORTED
        assert status(B=9) == hg.ERR_UNSUPPORTED
        assert status(K=60) == hg.ERR_UNSUPPORTED
        assert status(K=0) == hg.ERR_UNSUPPORTED
        assert status(x=0) == hg.ERR_INVALID_ARG
        assert status(N=0) == hg.ERR_INVALID_ARG
        assert status(ydt=hg.BF16) == hg.ERR_UNSUPPORTED
        assert status(bh=0) == hg.ERR_INVALID_ARG
        torch.cuda.synchronize()
        assert status() == hg.OK  # the context still works after errors
        torch.cuda.synchronize()
    finally:
        p.free()


@pytest.mark.parametrize("N,K,dtype,alpha,resident", [
    (16384, 4096, synth.F16, 0.0, True),     # OPT-6.7B fc1, resident
    (4096, 16384, synth.F16, 0.0, True),     # OPT-6.7B fc2, resident
    (20480, 5120, synth.F16, 0.62, False),   # OPT-13B fc1, streamed + CPU
    (7168, 28672, synth.F16, 0.6, False),    # OPT-30B fc2, streamed + CPU
    (36864, 9216, synth.BF16, 0.3, False),   # OPT-66B fc1 bf16, streamed + CPU
])
@pytest.mark.parametrize("B", [1, 2, 4, 8])
def test_full_size_opt_linears(ctx, N, K, dtype, alpha, resident, B):
    p = Problem(ctx, B, K, N, dtype, seed=N + K)
    try:
        y = p.run(alpha, resident)
        assert rel_err(y, p.ref()) <= TOL
    finally:
        p.free()


def test_alpha_benchmark_runs_in_bracket_and_keeps_parity(ctx):
    # OPT-13B fc1 shape; the closed-form start is the probe's Eq. 5 CPU fraction
    p = Problem(ctx, 1, 5120, 20480, synth.F16, seed=11)
    try:
        bw = hg.hetegen_probe(ctx, p.W.ptr, p.N, p.K, p.dtype, 1, 2)
        a0 = hg.hetegen_layer_plan([(p.N, p.K, p.dtype, 0)], [(bw["cpu_Bps"], bw["h2d_Bps"], bw["hbm_gemv_Bps"], 0.0)])[0]
        y = torch.empty((1, p.N), dtype=torch.float32, device="cuda")
        a, crossed = hg.hetegen_alpha_benchmark(ctx, p.x_dev.data_ptr(), 1, p.K, p.W.ptr, p.N, p.dtype, p.bias.ptr,
                                                p.b_dev.data_ptr(), y.data_ptr(), a0, 0.05, 0.01, 2, 1,
                                                torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert max(0.0, a0 - 0.05) - 1e-9 <= a <= min(1.0, a0 + 0.05) + 1e-9
        assert rel_err(y.cpu().numpy(), p.ref()) <= TOL          # the last measured run's output
        assert rel_err(p.run(a, False), p.ref()) <= TOL
    finally:
        p.free()


def test_probe_concurrent_rates(ctx):
    p = Problem(ctx, 1, 2048, 4096, synth.F16)
    try:
        alone = hg.hetegen_probe(ctx, p.W.ptr, p.N, p.K, p.dtype, 1, 2)
        both = hg.hetegen_probe(ctx, p.W.ptr, p.N, p.K, p.dtype, 1, 2, hg.PROBE_CONCURRENT)
        for bw in (alone, both):
            assert all(np.isfinite(bw[f]) and bw[f] > 0 for f in ("cpu_Bps", "h2d_Bps", "hbm_gemv_Bps"))
            assert bw["pin_Bps"] == 0
    finally:
        p.free()


def test_probe_hbm_read_bandwidth(ctx):
    bps = hg.hetegen_probe_hbm(ctx, 256 << 20, 3)
    assert 5e11 < bps < 9e12  # between a slow link and above the nominal 8 TB/s peak
    with pytest.raises(hg.HetegenError):
        hg.hetegen_probe_hbm(ctx, 1000, 3)


def test_probe_launch_round_trip(ctx):
    # an empty launch plus a stream synchronisation takes microseconds
    s = torch.cuda.current_stream().cuda_stream
    us = hg.hetegen_probe_launch(ctx, 200, s)
    assert 0.5 < us < 1000
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_probe_launch(ctx, 0, s)
    assert e.value.status == hg.ERR_INVALID_ARG


def _page_node(addr):
    """NUMA node of the page at `addr` (get_mempolicy with MPOL_F_NODE | MPOL_F_ADDR)."""
    import ctypes
    libc = ctypes.CDLL(None, use_errno=True)
    node = ctypes.c_int(-1)
    sys_get_mempolicy = 239  # x86-64
    rc = libc.syscall(sys_get_mempolicy, ctypes.byref(node), None, ctypes.c_ulong(0), ctypes.c_void_p(addr),
                      ctypes.c_ulong(1 | 2))
    return node.value if rc == 0 else None


def test_numa_node_placement_of_pinned_memory():
    import os
    nodes = sorted(int(d[4:]) for d in os.listdir("/sys/devices/system/node") if d.startswith("node") and d[4:].isdigit())
    c = hg.hetegen_create(0, numa_node=nodes[-1], chunk_bytes=65536, ring_depth=2)
    try:
        p = Problem(c, 2, 520, 1001, synth.F16, seed=3)
        try:
            got = _page_node(p.W.ptr)
            if got is not None:
                assert got == nodes[-1]
            for alpha, resident in ((0.0, False), (0.4, False), (0.4, True), (1.0, False)):
                assert rel_err(p.run(alpha, resident), p.ref()) <= TOL, (alpha, resident)
        finally:
            p.free()
    finally:
        hg.hetegen_destroy(c)
    with pytest.raises(hg.HetegenError):
        hg.hetegen_create(0, numa_node=nodes[-1] + 1)
    with pytest.raises(hg.HetegenError):
        hg.hetegen_create(0, numa_node=5000)
