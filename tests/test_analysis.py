"""Derived statistics of the measurement (host arithmetic, CPU only): the
linear iteration-time fit, the quadratic fit of K(r), the convexity index and
the crossover definitions, checked on synthetic curves with known answers."""
import numpy as np
import pytest

from paper_2606_00516_amd import analysis as A


def test_linear_fit_recovers_line_and_r2():
    n = np.array([512, 1024, 2048, 4096], float)
    a, b, r2 = A.linear_fit(n, 0.3 + 2e-3 * n)
    assert a == pytest.approx(0.3) and b == pytest.approx(2e-3) and r2 == pytest.approx(1.0)
    rng = np.random.default_rng(0)
    _, _, r2n = A.linear_fit(n, 0.3 + 2e-3 * n + rng.normal(0, 0.5, 4))
    assert r2n < 1.0


def test_gap_is_minus_c2_r_one_minus_r():
    # K(r) - K_bar(r) = -c2 r (1 - r) for any quadratic (App. A.3)
    c0, c1, c2 = 1.3, 4.0, -2.5
    r = np.linspace(0, 1, 11)
    k = c0 + c1 * r + c2 * r * r
    gap = k - A.eb_line(r, k[0], k[-1])
    assert np.allclose(gap, -c2 * r * (1 - r))
    f = A.quad_fit(r, k)
    assert np.allclose(f, (c0, c1, c2))
    assert A.kappa(*f) == pytest.approx(2 * c2 / (c0 + c1 + c2))
    rep = A.sweep_report(r, k)
    assert rep["kappa"] < 0 and rep["r_at_max_gap"] == pytest.approx(0.5)
    assert rep["max_gap"] == pytest.approx(-c2 * 0.25)
    # a concave curve lies above its chord: the mixed step is dearer than the
    # EB line everywhere inside (0, 1)
    assert A.eb_favoured(r, k, 1e-9) == pytest.approx(list(r[1:-1]))


def test_convex_curve_has_positive_kappa_and_no_eb_interval():
    r = np.linspace(0, 1, 11)
    k = 1 + 2 * r + 3 * r * r
    assert A.kappa(*A.quad_fit(r, k)) > 0
    assert A.eb_favoured(r, k, 0.0) == []


def test_crossover_primary():
    r = np.linspace(0, 1, 11)
    beta = np.where(r < 0.55, 1.0 + r, 1.2)     # exceeds beta(1) = 1.2 from r = 0.2
    assert A.crossover_primary(r, beta) == pytest.approx(0.2)
    assert A.crossover_primary(r, 1.0 + 0.1 * r) is None             # rising to the end: none
    b2 = np.array([1.0, 1.1, 1.25, 1.3, 1.2, 1.2, 1.2, 1.2, 1.2, 1.2, 1.2])
    assert A.crossover_primary(r, b2) == pytest.approx(0.1 + 0.1 * (1.2 - 1.1) / (1.25 - 1.1))
