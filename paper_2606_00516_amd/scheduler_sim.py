"""Iteration-level simulator of the serving loop under exclusive batching
EB(k, N), mixed batching MB, and the adaptive EB+ rule, priced by a step-time
model (host-side; the step times come from layer steps measured on this GPU).

What is simulated follows the paper's system model (Sec. 3.1): N slots, a
saturated queue, exclusive phases (a decode phase runs until k slots are
idle, then one prefill batch refills them while the other requests wait),
linear iteration times, output lengths from a distribution with hazard h(t).
MB runs chunked-prefill iterations of at most B rows, every decode request
contributing one row (Sec. 3.5).  EB+ chooses EB or MB before every iteration
with Eq. eb_plus_switch on online estimates.  The online controller
(Alg. "Online Joint Adaptation of (k*, N*)") keeps a window of completed
requests, estimates the hazard h(t) = p0 + eta t from it by weighted least
squares over t in [1, t95] (Sec. 3.4), and maps the estimates to a
threshold (Eqs. theta_base and delta_theta), a batch size (Eq. Nstar) and
k* = floor(theta* N*).  A KV-aware gate defers a
decode -> prefill switch while fewer than f_KV of the cache blocks are free
(App. "Runtime Refinement: KV-aware Feasibility Gate").
"""
from __future__ import annotations

import dataclasses
import math
from collections import deque
from typing import Callable, Deque, Dict, List, Optional, Tuple

import numpy as np

from . import cost_model as CM


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    """Input and output length samplers (positive integers)."""
    sample_L: Callable[[np.random.Generator, int], np.ndarray]
    sample_O: Callable[[np.random.Generator, int], np.ndarray]
    label: str = ""


def geometric_outputs(mu_O: float) -> Callable:
    """CFR: P(O = t) = p0 (1 - p0)^(t-1), p0 = 1 / mu_O."""
    p0 = 1.0 / mu_O
    return lambda rng, n: rng.geometric(p0, size=n)


def gamma_outputs(shape: float, mu_O: float) -> Callable:
    """Gamma(shape, rate shape / mu_O) rounded up to whole tokens: shape 1 is
    the CFR case, shape > 1 has an increasing hazard (App. "Empirical
    Evidence for Delta theta > 0 under IFR")."""
    return lambda rng, n: np.maximum(1, np.ceil(rng.gamma(shape, mu_O / shape, size=n))).astype(np.int64)


def linear_hazard_outputs(p0: float, eta: float) -> Callable:
    """Discrete lengths with hazard h(t) = min(1, p0 + eta t) (Sec. 3.2)."""
    def draw(rng, n):
        out = np.empty(n, np.int64)
        u = rng.random((n,))
        # inverse transform on the survival function S(t) = prod (1 - h(s))
        tmax = 1
        while True:
            t = np.arange(1, tmax + 1)
            h = np.minimum(1.0, p0 + eta * t)
            S = np.cumprod(1.0 - h)
            if S[-1] < 1e-12 or h[-1] >= 1.0:
                break
            tmax *= 2
        cdf = 1.0 - S
        out[:] = np.searchsorted(cdf, u, side="left") + 1
        return out
    return draw


def fixed_inputs(mu_L: int) -> Callable:
    return lambda rng, n: np.full(n, int(mu_L), np.int64)


# ----------------------------------------------------------------------------
# online estimation (Sec. 3.4)
# ----------------------------------------------------------------------------

def fit_linear_hazard(outputs: np.ndarray) -> Tuple[float, float]:
    """(p0, eta) of h(t) = p0 + eta t fitted by weighted least squares to the
    empirical hazard #{O = t} / #{O >= t} over t in [1, t95], each t weighted
    by its risk set #{O >= t}."""
    o = np.asarray(outputs, np.int64)
    if o.size < 2:
        raise ValueError("need at least two output lengths")
    t95 = max(2, int(np.percentile(o, 95)))
    counts = np.bincount(o, minlength=t95 + 2)
    at_risk = counts[::-1].cumsum()[::-1]            # #{O >= t}
    t = np.arange(1, t95 + 1)
    w = at_risk[t].astype(np.float64)
    keep = w > 0
    t, w = t[keep], w[keep]
    h = counts[t] / w
    A = np.stack([np.ones_like(t, dtype=np.float64), t.astype(np.float64)], axis=1)
    sw = np.sqrt(w)
    (p0, eta), *_ = np.linalg.lstsq(A * sw[:, None], h * sw, rcond=None)
    return float(p0), float(eta)


@dataclasses.dataclass
class ControllerCfg:
    C: float                     # KV capacity in tokens
    eps: float = 1e-3            # OOM risk level
    window: int = 2000           # W
    min_window: int = 200        # W_min
    update_every: int = 100      # T_upd
    theta_min: float = 0.02
    theta_max: float = 0.95
    theta_default: float = 0.3
    N_default: int = 256
    N_max: int = 8192


@dataclasses.dataclass
class LengthEstimates:
    """What the controller knows of the workload: the linear hazard
    h(t) = p0 + eta t of output lengths and the mean input length."""
    p0: float
    eta: float
    mu_L: float


class CompletionWindow:
    """Input and output lengths of the most recently completed requests (a
    bounded window) and the estimates taken from them (Sec. 3.4)."""

    def __init__(self, size: int):
        self._inputs: Deque[int] = deque(maxlen=size)
        self._outputs: Deque[int] = deque(maxlen=size)

    def add(self, L: int, O: int):
        self._inputs.append(int(L))
        self._outputs.append(int(O))

    def __len__(self) -> int:
        return len(self._outputs)

    def mean_output(self) -> float:
        return float(np.mean(self._outputs))

    def estimates(self) -> LengthEstimates:
        p0, eta = fit_linear_hazard(np.asarray(self._outputs))
        # a hazard below zero or falling with t is outside the model's IFR /
        # CFR family: clamp to the CFR boundary
        return LengthEstimates(p0=max(p0, 1e-6), eta=max(eta, 0.0), mu_L=float(np.mean(self._inputs)))


@dataclasses.dataclass
class OperatingPoint:
    """Threshold theta, batch size N and switch count k of EB(k, N)."""
    theta0: float
    theta: float
    N: int
    k: int


def operating_point(costs: CM.StepCosts, est: LengthEstimates, N_prev: int, cfg: ControllerCfg) -> OperatingPoint:
    """The operating point the estimates call for: the CFR threshold of
    Eq. theta_base at the ratio p0 alpha_p / alpha_d, raised by the IFR
    correction of Eq. delta_theta (taken at the batch size in use, N_prev),
    kept within [theta_min, theta_max]; the largest batch Eq. Nstar allows at
    that threshold under the KV capacity and risk level, within [1, N_max];
    and k = floor(theta N)."""
    th0 = CM.solve_theta0(est.p0 * costs.alpha_p / costs.alpha_d)
    correction = CM.delta_theta(est.eta, est.p0, th0, costs.beta_d, N_prev, costs.alpha_d) if est.eta > 0 else 0.0
    theta = min(cfg.theta_max, max(cfg.theta_min, th0 + correction))
    N = int(min(cfg.N_max, max(1, CM.n_star(cfg.C, cfg.eps, theta, est.p0, est.mu_L))))
    return OperatingPoint(theta0=th0, theta=theta, N=N, k=max(1, int(math.floor(theta * N))))


class AdaptiveController:
    """The online controller (Alg. "Online Joint Adaptation of (k*, N*)"):
    a window of completions as the estimator, and the operating-point rule
    above re-applied to its estimates every update_every completions once
    the window holds at least min_window of them."""

    def __init__(self, costs: CM.StepCosts, cfg: ControllerCfg):
        self.c = costs
        self.cfg = cfg
        self.window = CompletionWindow(cfg.window)
        self.point = OperatingPoint(theta0=cfg.theta_default, theta=cfg.theta_default, N=cfg.N_default,
                                    k=max(1, int(cfg.theta_default * cfg.N_default)))
        self.est: Optional[LengthEstimates] = None
        self._since_refresh = 0
        self.updates = 0

    def observe(self, L: int, O: int):
        """Record one completed request; refresh the operating point when due."""
        self.window.add(L, O)
        self._since_refresh += 1
        if self._since_refresh >= self.cfg.update_every and len(self.window) >= self.cfg.min_window:
            self.est = self.window.estimates()
            self.point = operating_point(self.c, self.est, self.point.N, self.cfg)
            self.updates += 1
            self._since_refresh = 0

    # the current operating point and estimates, as the simulator reads them
    @property
    def N(self) -> int:
        return self.point.N

    @property
    def k(self) -> int:
        return self.point.k

    @property
    def theta(self) -> float:
        return self.point.theta

    @property
    def theta0(self) -> float:
        return self.point.theta0

    @property
    def p0(self) -> Optional[float]:
        return self.est.p0 if self.est else None

    @property
    def eta(self) -> float:
        return self.est.eta if self.est else 0.0

    @property
    def mu_L(self) -> Optional[float]:
        return self.est.mu_L if self.est else None


# ----------------------------------------------------------------------------
# the simulator
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class SimResult:
    policy: str
    time_s: float
    completed: int
    decoded_tokens: int
    prefilled_tokens: int
    iterations: int
    eb_iterations: int
    mb_iterations: int
    peak_kv_tokens: int
    mean_decode_batch: float
    k: int
    N: int

    @property
    def throughput(self) -> float:
        """Completed requests per second."""
        return self.completed / self.time_s

    @property
    def token_throughput(self) -> float:
        return (self.decoded_tokens + self.prefilled_tokens) / self.time_s


@dataclasses.dataclass
class SimCfg:
    N: int
    k: int = 1
    B: int = 8192                        # MB token budget per iteration
    policy: str = "eb"                   # 'eb' | 'mb' | 'ebplus'
    kv_capacity: Optional[int] = None    # tokens; enables the KV gate
    block: int = 16
    s_kv: float = 0.5
    f0: float = 0.0
    delta: float = 0.0                   # EB+ priority margin
    ema: float = 0.05                    # EB+ occupancy smoothing
    adaptive: Optional[ControllerCfg] = None
    max_completions: int = 5000
    warmup: int = 200
    beta_ctx: float = 0.0                # optional cost per cached token of a decode row


class Simulator:
    """Slots hold (input length L, output length O, generated g, prefilled
    tokens); a request is a decode request once fully prefilled."""

    def __init__(self, costs: CM.StepCosts, wl: Workload, cfg: SimCfg, seed: int = 0):
        self.c, self.wl, self.cfg = costs, wl, cfg
        self.rng = np.random.default_rng(seed)
        self.ctrl = AdaptiveController(costs, cfg.adaptive) if cfg.adaptive else None
        cap = cfg.N if not self.ctrl else max(cfg.N, cfg.adaptive.N_max)
        self.cap = cap
        # completed requests' lengths, for the EB+ estimates without a controller
        self.seen_O: Deque[int] = deque(maxlen=2000)
        self.seen_L: Deque[int] = deque(maxlen=2000)
        self.L = np.zeros(cap, np.int64)
        self.O = np.zeros(cap, np.int64)
        self.g = np.zeros(cap, np.int64)
        self.pf = np.zeros(cap, np.int64)       # prefilled tokens
        self.busy = np.zeros(cap, bool)
        self.time = 0.0
        self.done = 0
        self.dec_tok = 0
        self.pre_tok = 0
        self.iters = self.eb_iters = self.mb_iters = 0
        self.peak_kv = 0
        self.batch_sum = 0
        self.batch_n = 0
        self.n_obs = None
        self.in_decode_phase = True
        self.t0 = None
        self.done0 = self.dec0 = self.pre0 = 0

    # -- bookkeeping --------------------------------------------------------
    def _limits(self):
        if self.ctrl:
            return self.ctrl.N, self.ctrl.k
        return self.cfg.N, self.cfg.k

    def _admit(self, n_max: int) -> np.ndarray:
        idle = np.nonzero(~self.busy)[0][:n_max]
        m = idle.size
        if m:
            self.L[idle] = self.wl.sample_L(self.rng, m)
            self.O[idle] = self.wl.sample_O(self.rng, m)
            self.g[idle] = 0
            self.pf[idle] = 0
            self.busy[idle] = True
        return idle

    def _kv_tokens(self) -> int:
        return int((self.pf[self.busy] + self.g[self.busy]).sum())

    def _finish(self, idx: np.ndarray):
        for i in idx:
            self.seen_O.append(int(self.O[i]))
            self.seen_L.append(int(self.L[i]))
            if self.ctrl:
                self.ctrl.observe(int(self.L[i]), int(self.O[i]))
        self.done += idx.size
        self.busy[idx] = False
        if self.t0 is None and self.done >= self.cfg.warmup:
            self.t0, self.done0, self.dec0, self.pre0 = self.time, self.done, self.dec_tok, self.pre_tok

    def _decode_rows(self) -> np.ndarray:
        return np.nonzero(self.busy & (self.pf >= self.L))[0]

    # -- iterations ---------------------------------------------------------
    def _decode_iteration(self):
        rows = self._decode_rows()
        n = rows.size
        ctx = int((self.L[rows] + self.g[rows]).sum())
        self.time += self.c.alpha_d + self.c.beta_d * n + self.cfg.beta_ctx * ctx
        self.g[rows] += 1
        self.dec_tok += n
        self.batch_sum += n
        self.batch_n += 1
        self.iters += 1
        self.eb_iters += 1
        self.peak_kv = max(self.peak_kv, self._kv_tokens())
        self._finish(rows[self.g[rows] >= self.O[rows]])

    def _prefill_phase(self):
        N, _ = self._limits()
        self._admit(max(0, N - int(self.busy.sum())))
        todo = np.nonzero(self.busy & (self.pf < self.L))[0]
        tokens = int((self.L[todo] - self.pf[todo]).sum())
        if todo.size == 0:
            return
        self.time += self.c.alpha_p + self.c.beta_p * tokens
        self.pf[todo] = self.L[todo]
        self.pre_tok += tokens
        self.iters += 1
        self.eb_iters += 1
        self.peak_kv = max(self.peak_kv, self._kv_tokens())

    def _mixed_iteration(self):
        N, _ = self._limits()
        self._admit(max(0, N - int(self.busy.sum())))
        rows = self._decode_rows()
        n_d = rows.size
        budget = max(0, self.cfg.B - n_d)
        # chunked prefill, first come first served in slot order
        pend = np.nonzero(self.busy & (self.pf < self.L))[0]
        taken = 0
        for i in pend:
            if taken >= budget:
                break
            t = int(min(self.L[i] - self.pf[i], budget - taken))
            self.pf[i] += t
            taken += t
        n_tok = n_d + taken
        if n_tok == 0:
            return
        r = n_d / n_tok
        ctx = int((self.L[rows] + self.g[rows]).sum())
        self.time += self.c.alpha_mb + self.c.beta_mb_at(r) * n_tok + self.cfg.beta_ctx * ctx
        self.g[rows] += 1
        self.dec_tok += n_d
        self.pre_tok += taken
        self.batch_sum += n_d
        self.batch_n += 1
        self.iters += 1
        self.mb_iters += 1
        self.peak_kv = max(self.peak_kv, self._kv_tokens())
        self._finish(rows[self.g[rows] >= self.O[rows]])

    # -- policies -----------------------------------------------------------
    def _gate_ok(self) -> bool:
        cap = self.cfg.kv_capacity
        if cap is None:
            return True
        total_blocks = cap // self.cfg.block
        used = int(np.ceil((self.pf[self.busy] + self.g[self.busy]) / self.cfg.block).sum())
        N, _ = self._limits()
        mu_O = self.ctrl.window.mean_output() if (self.ctrl and len(self.ctrl.window)) else float(np.mean(self.O[self.busy]))
        f = CM.kv_gate_fraction(N, mu_O, self.cfg.block, total_blocks, self.cfg.s_kv, self.cfg.f0)
        return (total_blocks - used) >= f * total_blocks

    def _eb_step(self):
        N, k = self._limits()
        idle = self.cap - int(self.busy.sum()) - (self.cap - N)
        decoding = self._decode_rows().size
        if (idle >= k and self._gate_ok()) or decoding == 0:
            self._prefill_phase()
        else:
            self._decode_iteration()

    def _ebplus_runs_eb(self) -> bool:
        occ = int(self.busy.sum())
        self.n_obs = occ if self.n_obs is None else (1 - self.cfg.ema) * self.n_obs + self.cfg.ema * occ
        if self.ctrl and self.ctrl.p0:
            mu_O, mu_L, th0 = 1.0 / self.ctrl.p0, self.ctrl.mu_L, self.ctrl.theta0
        elif len(self.seen_O) >= 20:
            # mean lengths of the completed requests seen so far
            mu_O, mu_L = float(np.mean(self.seen_O)), float(np.mean(self.seen_L))
            th0 = CM.solve_theta0(self.c.alpha_p / (self.c.alpha_d * mu_O))
        else:
            return False    # nothing known yet: MB, the default
        z = CM.zeta_of(th0)
        r = mu_O / (mu_L + mu_O)
        lhs = self.c.beta_mb_at(r) - self.c.beta_eb_w(mu_L, mu_O)
        rhs = ((self.c.alpha_p + self.c.alpha_d * z * mu_O) / th0 - self.c.alpha_mb * (1 + mu_O)) / (
            max(self.n_obs, 1.0) * (mu_L + mu_O))
        return lhs > rhs + self.cfg.delta

    def run(self) -> SimResult:
        N, k = self._limits()
        self._admit(N)
        self._prefill_phase() if self.cfg.policy != "mb" else None
        guard = 0
        while self.done < self.cfg.max_completions + self.cfg.warmup:
            if self.cfg.policy == "eb":
                self._eb_step()
            elif self.cfg.policy == "mb":
                self._mixed_iteration()
            else:
                if self._ebplus_runs_eb():
                    self._eb_step()
                else:
                    self._mixed_iteration()
            guard += 1
            if guard > 50_000_000:
                raise RuntimeError("simulation did not finish")
        t = self.time - (self.t0 or 0.0)
        N, k = self._limits()
        return SimResult(self.cfg.policy, t, self.done - self.done0, self.dec_tok - self.dec0,
                         self.pre_tok - self.pre0, self.iters, self.eb_iters, self.mb_iters, self.peak_kv,
                         self.batch_sum / max(1, self.batch_n), k, N)


def sweep_threshold(costs: CM.StepCosts, wl: Workload, N: int, thetas, seed: int = 0, **kw) -> List[Tuple[float, float]]:
    """Simulated EB(k = theta N, N) throughput over a grid of thresholds."""
    out = []
    for th in thetas:
        k = max(1, int(round(th * N)))
        res = Simulator(costs, wl, SimCfg(N=N, k=k, policy="eb", **kw), seed=seed).run()
        out.append((k / N, res.throughput))
    return out
