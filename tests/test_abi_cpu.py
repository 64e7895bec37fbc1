"""CPU-only checks of the C-ABI library: it loads, exports every declared call,
its host-only planner matches the oracle's distribution law, and calls that need a
device fail with a status instead of crashing."""
import math
import os
import re

import numpy as np
import pytest

import paper_2403_01164_amd as hg
from oracle import planner

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "hetegen.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"HETEGEN_API\s+[\w\s\*]+?\b(hetegen_\w+)\s*\(", src)))


def test_header_declares_the_calls():
    names = _declared()
    for must in ("hetegen_linear", "hetegen_layer_plan", "hetegen_decode_step", "hetegen_model_create",
                 "hetegen_create", "hetegen_host_alloc", "hetegen_probe"):
        assert must in names


def test_cpu_share_isa_is_reported():
    # the CPU share's instruction set, chosen when the library loads (no device needed)
    assert hg.hetegen_cpu_share_isa() in ("avx512+bf16", "avx512", "avx2", "scalar")


def test_every_declared_symbol_is_exported():
    import ctypes
    lib = ctypes.CDLL(hg.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(hg.EXPORTED)


def test_planner_matches_oracle_distribution_law():
    rng = np.random.default_rng(1)
    shapes, bws, want = [], [], []
    for i in range(64):
        vc, vm, vg = 10 ** rng.uniform(9, 11.5), 10 ** rng.uniform(9, 11), 10 ** rng.uniform(11, 13)
        pin = 0.0 if i % 3 else 10 ** rng.uniform(9, 11)
        res = 1 if i % 7 == 0 else 0
        shapes.append((4096, 1024, hg.F16, res))
        bws.append((vc, vm, vg, pin))
        want.append(planner.plan_cpu_fraction(vc, vm, vg, pin_Bps=pin, resident=bool(res)))
    got = hg.hetegen_layer_plan(shapes, bws)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-15)
    got_a = hg.hetegen_layer_plan(shapes, bws, flags=hg.PLAN_APPROX)
    want_a = [planner.plan_cpu_fraction(b[0], b[1], b[2], pin_Bps=b[3], resident=bool(s[3]), approx=True)
              for s, b in zip(shapes, bws)]
    assert np.allclose(got_a, want_a, rtol=1e-12, atol=1e-15)


def test_planner_shared_bandwidth_entry():
    got = hg.hetegen_layer_plan([(10, 8, 0, 0), (20, 8, 0, 1), (30, 8, 0, 0)], [(1e11, 5e10, 1e300, 0.0)])
    assert math.isclose(got[0], 2 / 3, rel_tol=1e-12) and got[1] == 0.0 and math.isclose(got[2], 2 / 3, rel_tol=1e-12)


@pytest.mark.parametrize("bw", [(0.0, 5e10, 6e12, 0.0), (1e11, -1.0, 6e12, 0.0), (1e11, 5e10, float("nan"), 0.0),
                                (1e11, 5e10, float("inf"), 0.0)])
def test_planner_rejects_bad_speeds(bw):
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_layer_plan([(10, 8, 0, 0)], [bw])
    assert e.value.status == hg.ERR_INVALID_ARG


def test_planner_rejects_bad_bandwidth_count():
    with pytest.raises(hg.HetegenError):
        hg.hetegen_layer_plan([(10, 8, 0, 0), (10, 8, 0, 0)], [(1e11, 5e10, 6e12, 0)] * 3)


def test_create_without_device_reports_status():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_create(0)
    assert e.value.status == hg.ERR_HIP
    assert "device" in str(e.value)


def test_create_rejects_bad_config():
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_create(0, ring_depth=1)
    assert e.value.status == hg.ERR_INVALID_ARG
    with pytest.raises(hg.HetegenError) as e:
        hg.hetegen_create(0, chunk_bytes=100)
    assert e.value.status == hg.ERR_INVALID_ARG


def test_single_hip_runtime_in_process():
    # the binding imports torch before the library, so only one libamdhip64 is mapped
    import torch  # noqa: F401
    maps = open("/proc/self/maps").read()
    paths = {l.split()[-1] for l in maps.splitlines() if "libamdhip64" in l}
    assert len(paths) == 1, paths
