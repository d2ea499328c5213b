"""Pins of the batching cost model (host arithmetic) against brute force,
Monte Carlo and closed forms rather than against itself."""
import math

import numpy as np
import pytest

from paper_2606_00516_amd import cost_model as CM


def _costs(rng=None, **kw):
    rng = rng or np.random.default_rng(0)
    c = CM.StepCosts(alpha_p=float(rng.uniform(5e-3, 5e-2)), beta_p=float(rng.uniform(1e-6, 1e-4)),
                     alpha_d=float(rng.uniform(5e-3, 3e-2)), beta_d=float(rng.uniform(1e-6, 1e-4)),
                     alpha_mb=float(rng.uniform(5e-3, 5e-2)),
                     beta_mb=(float(rng.uniform(1e-6, 1e-4)), float(rng.uniform(-5e-5, 5e-5)),
                              float(rng.uniform(-5e-5, 5e-5))))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("gamma", [1e-4, 1e-2, 0.3, 1.0, 7.5, 120.0])
def test_theta0_is_the_root_of_the_increasing_psi(gamma):
    th = CM.solve_theta0(gamma)
    assert 0.0 < th < 1.0
    assert abs(CM.psi(th) - gamma) <= 1e-9 * max(1.0, gamma)
    # Psi' = theta / (1 - theta)^2 > 0 (App. "Existence and Uniqueness"):
    # a finite-difference check on a grid
    g = np.linspace(1e-4, 0.999, 2000)
    v = np.array([CM.psi(t) for t in g])
    assert np.all(np.diff(v) > 0)
    assert CM.solve_theta0(gamma * 1.01) > th


@pytest.mark.parametrize("seed", range(6))
def test_theta0_maximises_the_fluid_throughput_by_brute_force(seed):
    # theta0 from the closed form equals the maximiser of R(theta) =
    # theta / T(theta) found by a grid search, and does not move when the
    # per-token costs, N or mu_L change (App. "Parameter Independence")
    rng = np.random.default_rng(seed)
    c = _costs(rng)
    p0 = 1.0 / float(rng.uniform(50, 2000))
    th0 = CM.solve_theta0(p0 * c.alpha_p / c.alpha_d)
    grid = np.linspace(1e-5, 1 - 1e-5, 200001)
    for N, mu_L, bscale in ((64, 100.0, 1.0), (4096, 900.0, 0.3), (512, 5.0, 7.0)):
        cc = CM.StepCosts(c.alpha_p, c.beta_p * bscale, c.alpha_d, c.beta_d * bscale, c.alpha_mb, c.beta_mb)
        R = grid / np.array([CM.cycle_time(t, N, cc, p0, mu_L) for t in grid])
        assert abs(grid[int(np.argmax(R))] - th0) < 2e-4, (N, mu_L, bscale)


def test_fluid_decode_phase_matches_the_death_process():
    # pure death process: every active request completes with prob p0 per
    # iteration; iterations until k = theta N completions and the summed
    # batch size against the fluid forms t* = zeta / p0 and N theta / p0
    rng = np.random.default_rng(1)
    N, p0, theta = 20000, 0.01, 0.3
    k = int(theta * N)
    iters, summed = [], []
    for _ in range(20):
        n, t, s = N, 0, 0
        while N - n < k:
            s += n
            n -= rng.binomial(n, p0)
            t += 1
        iters.append(t)
        summed.append(s)
    assert abs(np.mean(iters) - CM.zeta_of(theta) / p0) / (CM.zeta_of(theta) / p0) < 0.02
    assert abs(np.mean(summed) - N * theta / p0) / (N * theta / p0) < 0.02
    # and the phase time with per-iteration cost alpha_d + beta_d n
    ad, bd = 0.02, 3e-5
    sim = np.mean([ad * t + bd * s for t, s in zip(iters, summed)])
    assert abs(sim - CM.decode_phase_time(theta, N, ad, bd, p0)) / sim < 0.02


@pytest.mark.parametrize("seed", range(20))
def test_crossover_condition_is_the_throughput_comparison(seed):
    # Prop. "comparison": the inequality holds exactly when the MB throughput
    # formula exceeds the EB one (both computed from their own formulas)
    rng = np.random.default_rng(100 + seed)
    c = _costs(rng)
    mu_L, mu_O = float(rng.uniform(10, 2000)), float(rng.uniform(10, 2000))
    N = int(rng.integers(16, 8192))
    d = CM.compare(c, mu_L, mu_O, N)
    direct = CM.tp_mb(N, c, mu_L, mu_O) > CM.tp_eb(d.k0, N, c, mu_L, mu_O)
    if abs(d.lhs - d.rhs) > 1e-12 * max(abs(d.lhs), abs(d.rhs), 1e-30):
        assert d.mb_favoured == direct
    assert d.tp_eb == pytest.approx(CM.tp_eb(d.k0, N, c, mu_L, mu_O))


def test_eb_plus_rule_reverses_the_condition_at_continuous_k():
    # with k0* = theta0 N taken continuously and no margin, EB+ runs EB
    # exactly when MB is not favoured; a positive margin delta favours MB
    rng = np.random.default_rng(7)
    agree = 0
    for _ in range(200):
        c = _costs(rng)
        mu_L, mu_O = float(rng.uniform(10, 2000)), float(rng.uniform(10, 2000))
        N = int(rng.integers(2000, 100000))
        d = CM.compare(c, mu_L, mu_O, N)
        if abs(d.lhs - d.rhs) > 1e-3 * abs(d.rhs) + 1e-12:
            agree += int(d.eb_plus_runs_eb == (not d.mb_favoured))
            big = CM.compare(c, mu_L, mu_O, N, delta=abs(d.lhs) + abs(d.rhs) + 1.0)
            assert not big.eb_plus_runs_eb
    assert agree >= 190


@pytest.mark.parametrize("seed", range(10))
def test_ifr_correction_positive_and_its_beta_d_zero_form(seed):
    rng = np.random.default_rng(200 + seed)
    p0 = 1.0 / float(rng.uniform(20, 2000))
    gamma = float(10 ** rng.uniform(-3, 1.5))
    th = CM.solve_theta0(gamma)
    eta = float(rng.uniform(1e-3, 1.0)) * p0 * p0
    N, ad, bd = float(rng.integers(16, 4096)), 0.02, float(rng.uniform(0, 1e-4))
    assert CM.delta_theta(eta, p0, th, bd, N, ad) > 0
    z = CM.zeta_of(th)
    special = eta * (1 - th) ** 2 / (p0 * p0 * th) * z * (gamma + z / 2)
    assert CM.delta_theta(eta, p0, th, 0.0, N, ad) == pytest.approx(special, rel=1e-9)


def _ifr_optimum(c, N, p0, eta, mu_L):
    """Maximiser of theta / T(theta) for the exact fluid model under the
    linear hazard p0 + eta t (no expansion): decode time from
    p0 T + eta T^2 / 2 = zeta, cumulative batch by quadrature."""
    from scipy import integrate, optimize

    def cycle(theta):
        z = -math.log1p(-theta)
        T = (-p0 + math.sqrt(p0 * p0 + 2 * eta * z)) / eta
        I = N * integrate.quad(lambda s: math.exp(-p0 * s - eta * s * s / 2), 0.0, T, epsabs=0, epsrel=1e-13)[0]
        return c.alpha_d * T + c.beta_d * I + c.alpha_p + c.beta_p * N * mu_L * theta

    res = optimize.minimize_scalar(lambda t: -t / cycle(t), bounds=(1e-6, 1 - 1e-6), method="bounded",
                                   options={"xatol": 1e-12})
    return res.x


@pytest.mark.parametrize("rho", [0.0, 0.5, 4.0])
def test_ifr_correction_matches_the_exact_fluid_optimum(rho):
    # first-order accuracy of Eq. delta_theta: (theta*(eta) - theta0) / eta
    # from a brute-force optimisation of the exact IFR fluid cycle converges
    # to Delta theta / eta as eta -> 0
    p0, N = 1.0 / 300.0, 1024.0
    c = CM.StepCosts(alpha_p=0.05, beta_p=2e-5, alpha_d=0.02, beta_d=rho * 0.02 / N, alpha_mb=0.0,
                     beta_mb=(0.0, 0.0, 0.0))
    th0 = CM.solve_theta0(p0 * c.alpha_p / c.alpha_d)
    errs = []
    for scale in (4e-3, 2e-3, 1e-3):
        eta = scale * p0 * p0
        got = (_ifr_optimum(c, N, p0, eta, 200.0) - th0) / eta
        want = CM.delta_theta(eta, p0, th0, c.beta_d, N, c.alpha_d) / eta
        errs.append(abs(got - want) / want)
    assert errs[-1] < 0.02, errs
    assert errs[-1] < errs[0]


def test_batch_size_bounds_are_ordered():
    rng = np.random.default_rng(3)
    for _ in range(200):
        p0 = 1.0 / float(rng.uniform(20, 2000))
        mu_L = float(rng.uniform(1, 4000))
        theta = float(rng.uniform(0.01, 0.99))
        C = float(rng.uniform(1e5, 1e8))
        eps = float(10 ** rng.uniform(-6, -1))
        a, b, s = (CM.n_star(C, eps, theta, p0, mu_L), CM.n_star_expected(C, theta, p0, mu_L),
                   CM.n_star_static(C, theta, p0, mu_L))
        assert a <= b <= s


def test_memory_bound_against_the_random_walk():
    # the supremum bound (App. "Supremum Bound") on Monte Carlo walks with the
    # model's increments (n tokens added per iteration, Binomial(n, p0)
    # completions each releasing L + O): the mean supremum stays below
    # v / (2 |d|) and the tail below exp(-2 |d| x / v), i.e. the bound is
    # conservative
    rng = np.random.default_rng(5)
    n, p0, mu_L = 400, 0.02, 50.0
    steps = 20000
    sups = []
    for _ in range(200):
        j = rng.binomial(n, p0, size=steps)
        released = np.array([rng.geometric(p0, size=k).sum() + k * mu_L for k in j])
        walk = np.cumsum(n - released)
        sups.append(max(0.0, float(walk.max())))
    d = n * p0 * mu_L
    v = n * p0 * (1 - p0) / p0 ** 2 + n * p0 * (1 - p0) * (mu_L + 1 / p0) ** 2
    sups = np.asarray(sups)
    assert np.mean(sups) <= v / (2 * d)
    for x in (0.5, 1.0, 2.0):
        x = x * v / (2 * d)
        assert np.mean(sups > x) <= math.exp(-2 * d * x / v) + 0.05


def test_kv_gate_fraction_clips():
    assert CM.kv_gate_fraction(10, 10, 16, 10 ** 9) == 0.05
    assert CM.kv_gate_fraction(10 ** 6, 10 ** 4, 16, 100) == 0.6
    f = CM.kv_gate_fraction(1000, 200, 16, 100000)
    assert f == pytest.approx(1000 * 200 * 0.5 / (16 * 100000))


def test_calibration_recovers_planted_coefficients():
    # steps generated from known coefficients are fitted back
    true = CM.StepCosts(0.002, 3e-7, 0.0015, 2.5e-6, 0.0021, (4e-7, 1.5e-6, 1e-6))
    pts = []
    for n in (512, 1024, 2048, 4096):
        pts.append({"mode": "prefill", "n_tok": n, "ms": 1e3 * (true.alpha_p + true.beta_p * n)})
        pts.append({"mode": "decode", "n_tok": n, "ms": 1e3 * (true.alpha_d + true.beta_d * n)})
        for r in np.linspace(0, 1, 11):
            pts.append({"mode": "mixed", "n_tok": n, "r": float(r),
                        "ms": 1e3 * (true.alpha_mb + true.beta_mb_at(r) * n)})
    c = CM.calibrate(pts)
    assert c.alpha_p == pytest.approx(true.alpha_p, rel=1e-9)
    assert c.beta_d == pytest.approx(true.beta_d, rel=1e-9)
    assert c.alpha_mb == pytest.approx(true.alpha_mb, rel=1e-9)
    assert np.allclose(c.beta_mb, true.beta_mb, rtol=1e-6, atol=1e-15)


def test_committed_mi355x_profile_loads():
    # the calibration the benchmark wrote from MI355X step times: linear fits
    # as close as the paper's own within the practical budget (R^2 above
    # 0.986 up to 8K tokens, App. A.1; the GEMM kernel and its K split change
    # with the row count here), positive fixed and per-token costs
    c = CM.load_profile()
    assert c.alpha_p > 0 and c.alpha_d > 0 and c.alpha_mb > 0
    assert c.beta_p > 0 and c.beta_d > 0 and c.beta_mb_at(0.5) > 0
    assert c.r2["prefill"] > 0.98 and c.r2["decode"] > 0.98
    assert min(c.r2.values()) > 0.97
    rows = CM.evaluate(c)
    assert len(rows) == len(CM.PAPER_MIXES) * 4
