"""ORACLE - test infrastructure only: the alpha benchmark's fit-and-solve step.

HeteGen Sec. 4.4 "Alpha Benchmark": starting from the closed-form ratio, the ratio
is varied over a small bracket around it in fixed steps; at each point the CPU time
and the communication time are measured; polynomials F_CPU and F_COM are fitted to
the two series, and the refined ratio is the one where the fitted curves meet
(Eq. 10); Eq. 11-12 read the balanced times off the fitted curves.

Readings (the paper leaves them open): the ratio is the library's CPU fraction;
the "communication" side is the whole GPU side of the module (transfer plus GPU
compute, as in the balance of Eq. 2/4); the fit is least squares of a given degree;
the meeting point is the root of F_CPU - F_COM inside the bracket; when the fitted
curves do not cross inside the bracket, the point of the bracket with the smallest
max(F_CPU, F_COM) (on a grid of 10^4 intervals) is taken instead.
"""
import numpy as np


def fit(alphas, times, degree):
    """Least-squares polynomial coefficients (highest power first), numpy.polyfit."""
    return np.polyfit(np.asarray(alphas, float), np.asarray(times, float), degree)


def solve(alphas, t_cpu, t_com, degree, lo, hi):
    """Refined CPU fraction and whether the fitted curves cross in [lo, hi]."""
    pc = fit(alphas, t_cpu, degree)
    pg = fit(alphas, t_com, degree)
    diff = np.polysub(pc, pg)
    roots = [r.real for r in np.roots(diff) if abs(r.imag) < 1e-12 and lo - 1e-12 <= r.real <= hi + 1e-12]
    if np.all(np.abs(diff) < 1e-300):
        roots = []
    if roots:
        # one crossing expected; take the one with the smallest balanced time
        best = min(roots, key=lambda a: np.polyval(pc, a))
        return float(min(max(best, lo), hi)), True
    grid = np.linspace(lo, hi, 10001)
    m = np.maximum(np.polyval(pc, grid), np.polyval(pg, grid))
    return float(grid[np.argmin(m)]), False


def balanced_times(alphas, t_cpu, t_com, degree, alpha):
    """Eq. 11-12: T_CPU and T_COM read off the fitted curves at the refined ratio."""
    return float(np.polyval(fit(alphas, t_cpu, degree), alpha)), float(np.polyval(fit(alphas, t_com, degree), alpha))


def minimize(alphas, t_wall, degree, lo, hi):
    """Step-level reading: the ratio minimising a least-squares polynomial fitted to the
    measured step times, on a grid of 10^4 intervals of [lo, hi]."""
    pw = fit(alphas, t_wall, degree)
    grid = np.linspace(lo, hi, 10001)
    return float(grid[np.argmin(np.polyval(pw, grid))])
