"""Pins of the serving-loop simulator and the online controller against the
closed forms they must reproduce and against planted parameters."""
import numpy as np
import pytest

from paper_2606_00516_amd import cost_model as CM
from paper_2606_00516_amd import scheduler_sim as S

COSTS = CM.StepCosts(alpha_p=0.03, beta_p=2e-5, alpha_d=0.01, beta_d=5e-5, alpha_mb=0.02, beta_mb=(6e-5, 0.0, 0.0))


def test_hazard_fit_recovers_planted_parameters():
    rng = np.random.default_rng(0)
    o = S.geometric_outputs(200)(rng, 40000)
    p0, eta = S.fit_linear_hazard(o)
    assert p0 == pytest.approx(1 / 200, rel=0.05)
    assert abs(eta) * np.percentile(o, 95) < 0.1 / 200
    o = S.linear_hazard_outputs(2e-3, 2e-5)(rng, 40000)
    p0, eta = S.fit_linear_hazard(o)
    assert p0 == pytest.approx(2e-3, rel=0.15)
    assert eta == pytest.approx(2e-5, rel=0.1)


def test_linear_hazard_sampler_has_the_planted_hazard():
    # empirical hazard #{O = t} / #{O >= t} against p0 + eta t at a few t
    rng = np.random.default_rng(1)
    o = S.linear_hazard_outputs(0.01, 1e-4)(rng, 200000)
    for t in (1, 20, 60):
        h = np.mean(o == t) / np.mean(o >= t)
        assert h == pytest.approx(0.01 + 1e-4 * t, rel=0.1)


def test_eb_simulation_matches_the_fluid_throughput_and_optimum():
    # geometric outputs: simulated EB(theta N, N) throughput at theta0 is
    # within 2 % of Eq. throughput_EB, within 1 % of the best threshold on a
    # grid, and clearly above a late switch
    mu_O, mu_L, N = 100, 50, 512
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    th0 = CM.solve_theta0(COSTS.alpha_p / (COSTS.alpha_d * mu_O))
    grid = list(np.arange(0.1, 0.75, 0.05)) + [th0]
    res = dict(S.sweep_threshold(COSTS, wl, N, grid, seed=0, max_completions=4000))
    at0 = res[max(1, int(round(th0 * N))) / N]
    formula = CM.tp_eb(max(1, int(th0 * N)), N, COSTS, mu_L, mu_O)
    assert at0 == pytest.approx(formula, rel=0.02)
    assert at0 >= 0.99 * max(res.values())
    assert at0 >= 1.08 * res[round(0.7 * N) / N]


def _best_theta(shape, mu_O, seed):
    """Vertex of a parabola through the simulated throughputs within 2 % of
    the best threshold on a grid (less sensitive to noise than the argmax)."""
    wl = S.Workload(S.fixed_inputs(32), S.gamma_outputs(shape, mu_O))
    grid = np.arange(0.2, 0.85, 0.04)
    costs = CM.StepCosts(alpha_p=0.2, beta_p=1e-6, alpha_d=0.01, beta_d=1e-5, alpha_mb=0.0, beta_mb=(0, 0, 0))
    th, tp = np.array(S.sweep_threshold(costs, wl, 256, grid, seed=seed, max_completions=6000)).T
    top = tp >= 0.98 * tp.max()
    a, b, _ = np.polyfit(th[top], tp[top], 2)
    return -b / (2 * a)


def test_increasing_hazard_moves_the_best_threshold_up():
    # Gamma outputs with the same mean: shape 1 (constant hazard) against
    # shape 2 (increasing hazard); the best threshold of the simulated EB
    # loop is higher for the increasing hazard (Thm. "IFR Threshold
    # Correction": Delta theta > 0), and the constant-hazard one sits near
    # theta0
    cfr = np.mean([_best_theta(1.0, 64, s) for s in range(2)])
    ifr = np.mean([_best_theta(2.0, 64, s) for s in range(2)])
    assert ifr > cfr + 0.03, (cfr, ifr)
    assert cfr == pytest.approx(CM.solve_theta0(0.2 / (0.01 * 64)), abs=0.06)


def test_mb_simulation_matches_the_mb_throughput():
    # r-independent mixed cost: the simulated MB loop reaches
    # [alpha_MB (1 + mu_O) / N + beta_MB (mu_L + mu_O)]^-1 (Sec. 3.5) when
    # every prompt fits one iteration's budget
    mu_O, mu_L, N = 100, 50, 512
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    res = S.Simulator(COSTS, wl, S.SimCfg(N=N, B=1 << 20, policy="mb", max_completions=6000), seed=0).run()
    assert res.throughput == pytest.approx(CM.tp_mb(N, COSTS, mu_L, mu_O), rel=0.03)


def test_adaptive_controller_settles_on_the_closed_forms():
    # Alg. "Online Joint Adaptation": on geometric outputs the controller's
    # threshold approaches theta0 of the true p0 and its batch size N* of
    # Eq. Nstar once the batch size has stopped growing (while it grows, the
    # window of recent completions over-represents long requests)
    mu_O, mu_L = 120, 40
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    C = 200_000.0
    ctl = S.ControllerCfg(C=C, eps=1e-3, window=3000, min_window=300, update_every=200, N_default=256, N_max=4096)
    sim = S.Simulator(COSTS, wl, S.SimCfg(N=256, policy="eb", adaptive=ctl, max_completions=30000), seed=2)
    sim.run()
    c = sim.ctrl
    th0 = CM.solve_theta0(COSTS.alpha_p / (COSTS.alpha_d * mu_O))
    assert c.updates > 5
    assert c.p0 == pytest.approx(1.0 / mu_O, rel=0.1)
    assert c.theta0 == pytest.approx(th0, abs=0.03)
    want_N = min(ctl.N_max, CM.n_star(C, 1e-3, c.theta, 1.0 / mu_O, mu_L))
    assert c.N == pytest.approx(want_N, rel=0.1)
    assert c.N < ctl.N_max
    assert c.k == int(c.theta * c.N)


def test_kv_gate_lowers_the_memory_peak():
    # a cache too small for the batch: with the gate the decode -> prefill
    # switch waits for blocks to free up, and the peak footprint is lower
    mu_O, mu_L, N = 200, 400, 512
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    cap = 260_000
    k = int(0.3 * N)
    free = S.Simulator(COSTS, wl, S.SimCfg(N=N, k=k, policy="eb", max_completions=3000), seed=3).run()
    gated = S.Simulator(COSTS, wl, S.SimCfg(N=N, k=k, policy="eb", kv_capacity=cap, max_completions=3000),
                        seed=3).run()
    assert gated.peak_kv_tokens < free.peak_kv_tokens


@pytest.mark.parametrize("mb_cost,expect", [(1.0, "mb"), (3.0, "eb")])
def test_eb_plus_runs_the_better_discipline(mb_cost, expect):
    # mixed rows priced at 1x or 3x the weighted EB marginal cost: EB+ runs
    # mostly the discipline the crossover condition favours, and reaches at
    # least 95 % of the better of EB(k0*) and MB
    mu_O, mu_L, N = 100, 50, 512
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    bw = COSTS.beta_eb_w(mu_L, mu_O)
    c = CM.StepCosts(COSTS.alpha_p, COSTS.beta_p, COSTS.alpha_d, COSTS.beta_d, alpha_mb=0.004,
                     beta_mb=(mb_cost * bw, 0.0, 0.0))
    k0 = max(1, int(CM.solve_theta0(c.alpha_p / (c.alpha_d * mu_O)) * N))
    eb = S.Simulator(c, wl, S.SimCfg(N=N, k=k0, policy="eb", max_completions=4000), seed=4).run()
    mb = S.Simulator(c, wl, S.SimCfg(N=N, B=1 << 20, policy="mb", max_completions=4000), seed=4).run()
    ebp = S.Simulator(c, wl, S.SimCfg(N=N, k=k0, B=1 << 20, policy="ebplus", max_completions=4000), seed=4).run()
    d = CM.compare(c, mu_L, mu_O, N)
    assert ("mb" if d.mb_favoured else "eb") == expect
    share_eb = ebp.eb_iterations / ebp.iterations
    assert (share_eb > 0.8) if expect == "eb" else (share_eb < 0.2)
    assert ebp.throughput >= 0.95 * max(eb.throughput, mb.throughput)


def test_kv_gate_reads_the_controller_window():
    # with the online controller on, the KV gate takes the mean output length
    # from the controller's window of completions: the gated run completes as
    # the ungated one does, and the controller refreshes from a window whose
    # mean output matches the workload (the controller's own N* already keeps
    # the footprint near the capacity, so the peaks of the two runs are close)
    mu_O, mu_L = 200, 400
    wl = S.Workload(S.fixed_inputs(mu_L), S.geometric_outputs(mu_O))
    cap = 260_000
    ctl = S.ControllerCfg(C=float(cap), window=1000, min_window=100, update_every=100, N_default=256, N_max=1024)
    free = S.Simulator(COSTS, wl, S.SimCfg(N=256, policy="eb", adaptive=ctl, max_completions=2000), seed=1)
    gated = S.Simulator(COSTS, wl, S.SimCfg(N=256, policy="eb", kv_capacity=cap, adaptive=ctl, max_completions=2000),
                        seed=1)
    rf, rg = free.run(), gated.run()
    assert gated.ctrl.updates > 5 and gated.ctrl.window.mean_output() == pytest.approx(mu_O, rel=0.15)
    assert min(rg.completed, rf.completed) >= 2000
    assert rg.peak_kv_tokens <= 1.1 * cap and rf.peak_kv_tokens <= 1.1 * cap
