"""Pins of the module scheduler oracle (HeteGen Sec. 4.5, Eq. 13) and parity of the
library's scheduler with it (pure host arithmetic, no GPU)."""
import itertools
import os

import numpy as np
import pytest

from oracle import scheduler as osched

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "module_schedule_cases.txt")


def _golden():
    cases, cur = [], None
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        f = line.split()
        if f[0] == "case":
            cur = {"name": f[1], "mods": [], "checks": []}
            cases.append(cur)
        elif f[0] == "modules":
            cur["mods"].append((int(f[1]), int(f[2]), float(f[3]), float(f[4])))
        elif f[0] == "budget":
            res = [] if f[4] == "-" else [int(v) for v in f[4].split(",")]
            cur["checks"].append((float(f[1]), res, float(f[6])))
    out = []
    for c in cases:
        mods = sorted(c["mods"])
        assert [m[0] for m in mods] == list(range(len(mods)))
        layer = [m[1] for m in mods]
        t = [m[2] for m in mods]
        mem = [m[3] for m in mods]
        for budget, res, used in c["checks"]:
            out.append(pytest.param(t, mem, layer, budget, res, used, id="%s-%g" % (c["name"], budget)))
    return out


@pytest.mark.parametrize("t,mem,layer,budget,res,used", _golden())
def test_golden_cases(t, mem, layer, budget, res, used):
    got, u = osched.schedule(t, mem, layer, budget)
    assert [i for i, r in enumerate(got) if r] == res
    assert u == used


def test_empty_and_limits():
    assert osched.schedule([], [], [], 10.0) == ([], 0.0)
    t, mem, layer = [1.0, 2.0, 3.0], [2.0, 3.0, 4.0], [0, 0, 1]
    assert osched.schedule(t, mem, layer, 0.0)[0] == [0, 0, 0]
    assert osched.schedule(t, mem, layer, 1.9)[0] == [0, 0, 0]  # below the smallest module
    assert osched.schedule(t, mem, layer, 9.0)[0] == [1, 1, 1]  # exactly everything
    assert osched.schedule(t, mem, layer, float("inf"))[0] == [1, 1, 1]


@pytest.mark.parametrize("seed", range(20))
def test_equal_sizes_identical_layers_is_knapsack_optimal(seed):
    """Identical layers and equal module sizes: the walk takes the modules with the
    largest times, which is the 0/1 knapsack optimum (brute force over all subsets)."""
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 4))
    kinds = int(rng.integers(2, 5))
    tk = rng.uniform(0.1, 5.0, kinds)
    t = [float(tk[i % kinds]) for i in range(L * kinds)]
    layer = [i // kinds for i in range(L * kinds)]
    mem = [1.0] * (L * kinds)
    k = int(rng.integers(0, L * kinds + 1))
    res, used = osched.schedule(t, mem, layer, float(k))
    assert used == sum(res) == k
    best = max(sum(t[i] for i in S) for S in itertools.combinations(range(L * kinds), k))
    assert abs(sum(t[i] for i in range(len(t)) if res[i]) - best) <= 1e-12 * max(1.0, best)


@pytest.mark.parametrize("seed", range(20))
def test_budget_respected_and_maximal(seed):
    """Never over budget; every module left out could not have been added when it was
    visited (its size exceeds what was free at that point of the walk)."""
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 13))
    layer = [int(v) for v in rng.integers(0, 4, n)]
    t = [float(v) for v in rng.uniform(0, 3, n)]
    mem = [float(v) for v in rng.integers(1, 6, n)]
    budget = float(rng.integers(0, 20))
    res, used = osched.schedule(t, mem, layer, budget)
    assert used <= budget
    assert used == sum(m for m, r in zip(mem, res) if r)
    free = budget
    for i in osched.visit_order(t, mem, layer):
        if res[i]:
            free -= mem[i]
        else:
            assert mem[i] > free
    # each layer's modules are visited by non-increasing gain
    g = osched.gains(t, mem)
    order = osched.visit_order(t, mem, layer)
    assert sorted(order) == list(range(n))
    for l in set(layer):
        seq = [g[i] for i in order if layer[i] == l]
        assert all(a >= b for a, b in zip(seq, seq[1:]))


# ---- library parity (host arithmetic, exact decisions) ----
hg = pytest.importorskip("paper_2403_01164_amd")


@pytest.mark.parametrize("t,mem,layer,budget,res,used", _golden())
def test_library_golden(t, mem, layer, budget, res, used):
    got, u = hg.hetegen_module_schedule(t, mem, layer, budget)
    assert [i for i, r in enumerate(got) if r] == res
    assert u == used


@pytest.mark.parametrize("seed", range(40))
def test_library_matches_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(0, 40))
    layer = [int(v) for v in rng.integers(0, 6, n)]
    if seed % 2:  # integer times and sizes: many equal gains
        t = [float(v) for v in rng.integers(0, 4, n)]
        mem = [float(v) for v in rng.integers(1, 4, n)]
    else:
        t = [float(v) for v in rng.uniform(0, 1e-2, n)]
        mem = [float(v) for v in rng.uniform(1e6, 7e8, n)]
    budget = float(rng.uniform(0, 1.1) * sum(mem)) if n else 1.0
    assert hg.hetegen_module_schedule(t, mem, layer, budget) == osched.schedule(t, mem, layer, budget)


def test_library_opt_shapes():
    """OPT-30B-shaped layers with per-shape heterogeneous times: the library and the
    oracle agree, and the budget of the first half of the weights is respected."""
    H, F, L = 7168, 28672, 48
    sizes = [3 * H * H * 2, H * H * 2, F * H * 2, H * F * 2]
    rate = [30e9, 25e9, 33e9, 34e9]  # heterogeneous bytes/s per kind
    t = [sizes[i % 4] / rate[i % 4] for i in range(4 * L)]
    mem = [float(sizes[i % 4]) for i in range(4 * L)]
    layer = [i // 4 for i in range(4 * L)]
    budget = sum(mem) / 2
    got = hg.hetegen_module_schedule(t, mem, layer, budget)
    assert got == osched.schedule(t, mem, layer, budget)
    assert got[1] <= budget


@pytest.mark.parametrize("bad", [
    dict(t=[float("nan")]), dict(t=[-1.0]), dict(mem=[0.0]), dict(mem=[float("inf")]), dict(layer=[-1]),
    dict(budget=-1.0), dict(budget=float("nan")),
])
def test_library_rejects(bad):
    a = dict(t=[1.0], mem=[1.0], layer=[0], budget=1.0)
    a.update(bad)
    with pytest.raises(hg.HetegenError):
        hg.hetegen_module_schedule(a["t"], a["mem"], a["layer"], a["budget"])
