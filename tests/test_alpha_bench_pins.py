"""Pins of the alpha-benchmark oracle (Sec. 4.4, Eq. 10-12) and parity of the
library's host-only fit-and-solve against it (CPU only)."""
import math

import numpy as np
import pytest

from oracle import alpha_bench as ab
from oracle import planner
import paper_2403_01164_amd as hg


def _grid(a0, gamma, lam):
    return np.round(np.arange(a0 - gamma, a0 + gamma + lam / 2, lam), 12)


def test_linear_time_model_reduces_to_closed_form():
    # times proportional to bytes (no contention): CPU side alpha*W/Vc, GPU side
    # (1-alpha)*W*(1/Vm + 1/Vg); the crossing is Eq. 5 as a CPU fraction
    Vc, Vm, Vg, Wb = 3.3e11, 5.6e10, 6.0e12, 2.9e8
    a_star = planner.plan_cpu_fraction(Vc, Vm, Vg)
    a = _grid(round(a_star, 2), 0.05, 0.01)
    tc = a * Wb / Vc
    tg = (1 - a) * Wb * (1 / Vm + 1 / Vg)
    for deg in (1, 2):
        got, crossed = ab.solve(a, tc, tg, deg, a[0], a[-1])
        assert crossed and abs(got - a_star) < 1e-9


def test_exact_quadratics_recover_the_analytic_crossing():
    a = _grid(0.5, 0.1, 0.01)
    tc = 2.0 * a ** 2 + 1.0 * a + 0.1          # increasing on the bracket
    tg = -1.0 * a ** 2 - 0.5 * a + 1.2          # decreasing
    # 3 a^2 + 1.5 a - 1.1 = 0
    want = (-1.5 + math.sqrt(1.5 ** 2 + 4 * 3 * 1.1)) / (2 * 3)
    got, crossed = ab.solve(a, tc, tg, 2, a[0], a[-1])
    assert crossed and abs(got - want) < 1e-12
    tcb, tgb = ab.balanced_times(a, tc, tg, 2, got)
    assert abs(tcb - tgb) < 1e-12


def test_no_crossing_takes_the_best_bracket_end():
    a = _grid(0.5, 0.05, 0.01)
    tc = 0.1 + 0.2 * a        # CPU always faster than the GPU side: move right
    tg = 2.0 - 0.1 * a
    got, crossed = ab.solve(a, tc, tg, 1, a[0], a[-1])
    assert not crossed and abs(got - a[-1]) < 1e-12


def test_noisy_samples_stay_close():
    rng = np.random.default_rng(3)
    a = _grid(0.8, 0.05, 0.01)
    tc = a * 1.0 + rng.normal(0, 1e-3, a.size)
    tg = (1 - a) * 4.0 + rng.normal(0, 1e-3, a.size)
    got, crossed = ab.solve(a, tc, tg, 2, a[0], a[-1])
    assert crossed and abs(got - 0.8) < 5e-3


@pytest.mark.parametrize("deg", [1, 2, 3])
def test_library_fit_matches_oracle(deg):
    rng = np.random.default_rng(deg)
    for trial in range(20):
        a0 = rng.uniform(0.2, 0.9)
        a = _grid(round(a0, 2), 0.05, 0.01)
        tc = np.polyval(rng.uniform(0.1, 1.0, deg + 1), a) * 1e-3 + a * 1e-3
        tg = np.polyval(rng.uniform(0.1, 1.0, deg + 1), a) * 1e-3 + (1 - a) * 3e-3
        want, crossed = ab.solve(a, tc, tg, deg, a[0], a[-1])
        got, got_crossed = hg.hetegen_alpha_fit(a, tc, tg, deg, a[0], a[-1])
        assert got_crossed == crossed
        assert abs(got - want) < 1e-6, (trial, got, want)


def test_library_fit_rejects_bad_input():
    with pytest.raises(hg.HetegenError):
        hg.hetegen_alpha_fit([0.1, 0.2], [1.0, 2.0], [2.0, 1.0], 2, 0.1, 0.2)   # fewer points than degree+1
    with pytest.raises(hg.HetegenError):
        hg.hetegen_alpha_fit([0.1, 0.2, 0.3], [1, 2, 3], [3, 2, 1], 1, 0.3, 0.1)  # empty bracket


def test_minimize_recovers_parabola_vertex_and_ends():
    a = np.round(np.arange(-0.06, 0.0601, 0.02), 12)
    t = 3.0 * (a - 0.013) ** 2 + 0.19
    assert abs(ab.minimize(a, t, 2, a[0], a[-1]) - 0.013) <= 1.2e-5     # grid spacing 1.2e-5
    t2 = 0.19 - 0.5 * a                                                    # decreasing: right end
    assert ab.minimize(a, t2, 1, a[0], a[-1]) == a[-1]


@pytest.mark.parametrize("deg", [1, 2, 3])
def test_library_minimize_matches_oracle(deg):
    rng = np.random.default_rng(10 + deg)
    for trial in range(20):
        a = np.round(np.arange(-0.06, 0.0601, 0.02), 12)
        t = np.polyval(rng.uniform(-1, 1, deg + 1), a) + rng.normal(0, 1e-3, a.size)
        want = ab.minimize(a, t, deg, a[0], a[-1])
        got = hg.hetegen_alpha_minimize(a, t, deg, a[0], a[-1])
        assert abs(got - want) <= 2e-5, (trial, got, want)
