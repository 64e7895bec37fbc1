"""Pins of the planner oracle (Eq. 4-9) against closed forms, limits and brute force."""
import math

import numpy as np
import pytest

from oracle import planner

RNG = np.random.default_rng(0)
CASES = [(10 ** RNG.uniform(9, 11.5), 10 ** RNG.uniform(11, 13), 10 ** RNG.uniform(9, 11)) for _ in range(50)]


@pytest.mark.parametrize("Vc,Vg,Vm", CASES)
def test_eq5_balances_eq4(Vc, Vg, Vm):
    a = planner.alpha_gpu_eq5(Vc, Vg, Vm)
    assert 0.0 < a < 1.0
    r = planner.balance_residual(a, Vc, Vg, Vm)
    assert abs(r) <= 1e-12 * ((1 - a) / Vc)


@pytest.mark.parametrize("Vc,Vg,Vm", CASES[:10])
def test_eq5_second_form(Vc, Vg, Vm):
    a = planner.alpha_gpu_eq5(Vc, Vg, Vm)
    assert math.isclose(a, 1.0 / (Vc / Vm + Vc / Vg + 1.0), rel_tol=1e-13)


@pytest.mark.parametrize("Vc,Vg,Vm", CASES[:10])
def test_eq5_is_bruteforce_argmin(Vc, Vg, Vm):
    grid = np.linspace(0.0, 1.0, 100001)
    T = np.maximum((1 - grid) / Vc, grid / Vg + grid / Vm)
    best = grid[np.argmin(T)]
    assert abs(best - planner.alpha_gpu_eq5(Vc, Vg, Vm)) <= 2e-5


def test_limits():
    # GPU compute infinitely fast -> Eq. 6
    assert math.isclose(planner.alpha_gpu_eq5(3e10, 1e200, 5e10), planner.alpha_gpu_eq6(3e10, 5e10), rel_tol=1e-12)
    # equal CPU and link speed, free GPU -> half on each side
    assert math.isclose(planner.alpha_gpu_eq5(5e10, 1e200, 5e10), 0.5, rel_tol=1e-12)
    # CPU nearly useless -> everything on the GPU (CPU fraction -> 0)
    assert planner.plan_cpu_fraction(1e-3, 5e10, 6e12) < 1e-12
    # link nearly closed -> everything on the CPU
    assert planner.plan_cpu_fraction(5e10, 1e-3, 6e12) > 1 - 1e-12
    # resident module -> no CPU share
    assert planner.plan_cpu_fraction(5e10, 5e10, 6e12, resident=True) == 0.0


def test_eq7_is_eq6_with_whole_module_times():
    W = 2.9e8
    for Vc, _, Vm in CASES[:10]:
        assert math.isclose(planner.alpha_gpu_eq7(W / Vc, W / Vm), planner.alpha_gpu_eq6(Vc, Vm), rel_tol=1e-12)


def test_eq8_pin_transfer_concurrency():
    assert planner.v_com(5.5e10, 0.0) == 5.5e10
    assert planner.v_com(5.5e10, 2e10) == 2e10
    assert planner.v_com(5.5e10, 9e10) == 5.5e10


def test_cpu_fraction_is_one_minus_paper_alpha():
    Vc, Vg, Vm = 1.0e11, 5.0e12, 5.5e10
    a = planner.alpha_gpu_eq5(Vc, Vg, Vm)
    assert math.isclose(planner.plan_cpu_fraction(Vc, Vm, Vg), 1 - a, rel_tol=1e-14)
    # CPU twice as fast as the link and GPU time negligible: 2/3 of the rows on the CPU
    assert math.isclose(planner.plan_cpu_fraction(1e11, 5e10, 1e200), 2.0 / 3.0, rel_tol=1e-12)


def _golden_rows():
    import os
    from fractions import Fraction
    path = os.path.join(os.path.dirname(__file__), "golden", "planner_closed_forms.txt")
    rows = []
    for line in open(path):
        line = line.split("#")[0].strip()
        if line:
            vc, vg, vm, a, c = line.split()
            rows.append((float(vc), float(vg), float(vm), float(Fraction(a)), float(Fraction(c))))
    return rows


@pytest.mark.parametrize("Vc,Vg,Vm,a,c", _golden_rows())
def test_golden_closed_forms(Vc, Vg, Vm, a, c):
    assert math.isclose(planner.alpha_gpu_eq5(Vc, Vg, Vm), a, rel_tol=1e-15)
    assert math.isclose(planner.plan_cpu_fraction(Vc, Vm, Vg), c, rel_tol=1e-15)
