"""Cost model of the exclusive-vs-mixed batching decision, evaluated on step
times measured on this GPU (host-side arithmetic, no kernels).

The paper prices a serving iteration linearly in its rows (Sec. 1;
Sec. 3.1 "Timing Model"): a prefill phase of k requests costs
``T_p = alpha_p + beta_p * sum L_i``, a decode iteration over n requests
``t_d(n) = alpha_d + beta_d * n``, and a mixed iteration
``alpha_MB + beta_MB^e(r) * n_tok`` with a decode-ratio-dependent marginal
cost (Sec. 3.5, App. "Empirical Calibration of beta_MB^e(r)").  On these
coefficients it derives

* the CFR base threshold theta_0, the unique root of
  ``Psi(theta) = theta / (1 - theta) + ln(1 - theta) = p0 alpha_p / alpha_d``
  (Prop. "Base Threshold under CFR", Eq. theta_base), with
  ``zeta = -ln(1 - theta_0)``;
* the fluid decode-phase duration, cycle time ``T(theta)`` and normalised
  throughput ``R(theta) = theta / T(theta)`` whose maximiser theta_0 is (App.
  "Proof of Proposition threshold_cfr");
* the EB throughput at ``k0* = floor(theta_0 N)`` (Eq. throughput_EB) with the
  workload-weighted marginal cost beta_EB^w, the MB throughput (Sec. 3.5), the
  crossover condition (Prop. "comparison", Eq. comparison_condition) and the
  EB+ rule (Eq. eb_plus_switch);
* the IFR correction Delta theta (Thm. "IFR Threshold Correction",
  Eq. delta_theta) and its beta_d = 0 form (App. "Physical Interpretation");
* the memory-safe batch size N* (Prop. "Memory-Safe Batch Size", Eq. Nstar)
  and the static / expected-peak bounds (App. "Comparison of Batch Size
  Bounds"), and the KV-aware gate threshold f_KV (App. "Runtime Refinement:
  KV-aware Feasibility Gate").

Units: seconds and tokens.  Coefficients measured on one decoder layer
price a model of n identical layers n times over; every decision below
compares ratios or differences of such prices, so it does not depend on the
layer count.
"""
from __future__ import annotations

import dataclasses
import json
import math
import os
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

from . import analysis as AN


# ----------------------------------------------------------------------------
# step-cost coefficients
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class StepCosts:
    """Linear step-time coefficients (seconds, per token / per request).

    beta_mb: (c0, c1, c2) of beta_MB^e(r) = c0 + c1 r + c2 r^2.
    """
    alpha_p: float
    beta_p: float
    alpha_d: float
    beta_d: float
    alpha_mb: float
    beta_mb: Tuple[float, float, float]
    label: str = ""
    r2: Dict[str, float] = dataclasses.field(default_factory=dict)

    def beta_mb_at(self, r: float) -> float:
        c0, c1, c2 = self.beta_mb
        return c0 + c1 * r + c2 * r * r

    def beta_eb_w(self, mu_L: float, mu_O: float) -> float:
        """Workload-weighted EB marginal cost (Sec. 3.2, below the EB
        throughput)."""
        return (self.beta_p * mu_L + self.beta_d * mu_O) / (mu_L + mu_O)

    def to_dict(self) -> dict:
        return dataclasses.asdict(self)


def calibrate(points: Sequence[dict], label: str = "") -> StepCosts:
    """Fit the coefficients from measured steps.

    points: dicts with ``mode`` ('prefill' | 'decode' | 'mixed'), ``n_tok``,
    ``ms`` and, for mixed steps, ``r``.  EB-prefill steps give
    (alpha_p, beta_p) against their rows; EB-decode steps give
    (alpha_d, beta_d) against their requests; mixed steps are fitted per decode
    share (alpha(r), beta(r)) and beta(r) by a quadratic in r (App. "Empirical
    Calibration of beta_MB^e(r)"); alpha_MB is the mean alpha(r) over the
    shares strictly inside (0, 1).
    """
    def lin(mode):
        pts = [p for p in points if p["mode"] == mode]
        if len(pts) < 2:
            raise ValueError(f"need at least two {mode} steps")
        a, b, r2 = AN.linear_fit([p["n_tok"] for p in pts], [p["ms"] * 1e-3 for p in pts])
        return a, b, r2

    ap, bp, r2p = lin("prefill")
    ad, bd, r2d = lin("decode")
    mixed = [p for p in points if p["mode"] == "mixed"]
    shares = sorted({round(float(p["r"]), 6) for p in mixed})
    rs, betas, alphas, r2m = [], [], [], {}
    for r in shares:
        pts = [p for p in mixed if abs(p["r"] - r) < 1e-9]
        if len(pts) < 2:
            continue
        a, b, r2 = AN.linear_fit([p["n_tok"] for p in pts], [p["ms"] * 1e-3 for p in pts])
        rs.append(r)
        betas.append(b)
        alphas.append(a)
        r2m[f"mixed_r{r:.2f}"] = r2
    if len(rs) < 3:
        raise ValueError("need mixed steps at three or more decode shares")
    c = AN.quad_fit(rs, betas)
    inner = [a for r, a in zip(rs, alphas) if 0.0 < r < 1.0] or alphas
    r2 = {"prefill": r2p, "decode": r2d, **r2m}
    return StepCosts(ap, bp, ad, bd, float(np.mean(inner)), c, label, r2)


PROFILE_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calibration")


def load_profile(path: Optional[str] = None) -> StepCosts:
    """Step costs from a calibration profile written by the benchmark's
    policy workload (default: the MI355X profile of the 8B-shaped layer)."""
    path = path or os.path.join(PROFILE_DIR, "mi355x_llama3_8b_layer.json")
    with open(path) as f:
        prof = json.load(f)
    c = prof["costs"]
    return StepCosts(c["alpha_p"], c["beta_p"], c["alpha_d"], c["beta_d"], c["alpha_mb"], tuple(c["beta_mb"]),
                     c.get("label", ""), c.get("r2", {}))


# ----------------------------------------------------------------------------
# threshold (CFR) and the fluid cycle
# ----------------------------------------------------------------------------

def psi(theta: float) -> float:
    """theta / (1 - theta) + ln(1 - theta): strictly increasing on (0, 1),
    from 0 to infinity (App. "Existence and Uniqueness")."""
    return theta / (1.0 - theta) + math.log1p(-theta)


def solve_theta0(gamma: float, tol: float = 1e-15) -> float:
    """The unique theta_0 in (0, 1) with Psi(theta_0) = gamma > 0
    (Eq. theta_base), by bisection on the increasing Psi."""
    if not gamma > 0:
        raise ValueError("gamma = p0 alpha_p / alpha_d must be positive")
    lo, hi = 0.0, 1.0
    # Psi(theta) ~ theta^2 / 2 near 0 and ~ 1 / (1 - theta) near 1
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mid <= 0.0 or mid >= 1.0:
            break
        if psi(mid) < gamma:
            lo = mid
        else:
            hi = mid
        if hi - lo < tol:
            break
    return 0.5 * (lo + hi)


def zeta_of(theta: float) -> float:
    return -math.log1p(-theta)


def decode_phase_time(theta: float, N: float, alpha_d: float, beta_d: float, p0: float) -> float:
    """Fluid decode-phase duration until a fraction theta of N requests has
    completed under hazard p0: [beta_d N theta - alpha_d ln(1 - theta)] / p0
    (Sec. 3.2, "Base Threshold Under CFR")."""
    return (beta_d * N * theta + alpha_d * zeta_of(theta)) / p0


def cycle_time(theta: float, N: float, c: StepCosts, p0: float, mu_L: float) -> float:
    """Decode phase plus the prefill of the theta N replacements (App.
    "Complete Cycle Time")."""
    return decode_phase_time(theta, N, c.alpha_d, c.beta_d, p0) + c.alpha_p + c.beta_p * N * mu_L * theta


def normalized_throughput(theta: float, N: float, c: StepCosts, p0: float, mu_L: float) -> float:
    """R(theta) = theta / T(theta) (App. "Throughput Optimization")."""
    return theta / cycle_time(theta, N, c, p0, mu_L)


# ----------------------------------------------------------------------------
# EB vs MB
# ----------------------------------------------------------------------------

def tp_eb(k: int, N: int, c: StepCosts, mu_L: float, mu_O: float) -> float:
    """EB throughput (requests per second) at threshold k under CFR with
    p0 = 1 / mu_O: [(alpha_p - alpha_d mu_O ln(1 - k/N)) / k
    + beta_EB^w (mu_L + mu_O)]^-1 (Sec. 3.2; Eq. throughput_EB at k = k0*)."""
    theta = k / N
    return 1.0 / ((c.alpha_p + c.alpha_d * mu_O * zeta_of(theta)) / k + c.beta_eb_w(mu_L, mu_O) * (mu_L + mu_O))


def tp_mb(N: int, c: StepCosts, mu_L: float, mu_O: float, r: Optional[float] = None) -> float:
    """MB throughput (requests per second) at effective batch size N:
    [alpha_MB (1 + mu_O) / N + beta_MB^e(r) (mu_L + mu_O)]^-1 (Sec. 3.5), with
    r = mu_O / (mu_L + mu_O) unless given."""
    r = mu_O / (mu_L + mu_O) if r is None else r
    return 1.0 / (c.alpha_mb * (1.0 + mu_O) / N + c.beta_mb_at(r) * (mu_L + mu_O))


@dataclasses.dataclass
class Decision:
    mu_L: float
    mu_O: float
    N: int
    r: float
    gamma: float
    theta0: float
    k0: int
    lhs: float          # beta_MB^e(r) - beta_EB^w          [s / token]
    rhs: float          # amortised fixed-cost advantage of MB [s / token]
    tp_eb: float        # requests / s
    tp_mb: float
    mb_favoured: bool   # Eq. comparison_condition
    eb_plus_runs_eb: bool  # Eq. eb_plus_switch (with the given delta)


def compare(c: StepCosts, mu_L: float, mu_O: float, N: int, delta: float = 0.0) -> Decision:
    """The crossover condition (Prop. "comparison"): MB beats EB(k0*) iff
    beta_MB^e - beta_EB^w < [(alpha_p + alpha_d zeta mu_O) / k0* -
    alpha_MB (1 + mu_O) / N] / (mu_L + mu_O); and the EB+ rule
    (Eq. eb_plus_switch), which runs EB when the left side exceeds the right
    side with k0* = theta_0 N (continuous) plus the margin delta."""
    p0 = 1.0 / mu_O
    gamma = p0 * c.alpha_p / c.alpha_d
    th = solve_theta0(gamma)
    z = zeta_of(th)
    k0 = max(1, int(math.floor(th * N)))
    r = mu_O / (mu_L + mu_O)
    lhs = c.beta_mb_at(r) - c.beta_eb_w(mu_L, mu_O)
    rhs = ((c.alpha_p + c.alpha_d * z * mu_O) / k0 - c.alpha_mb * (1.0 + mu_O) / N) / (mu_L + mu_O)
    rhs_plus = ((c.alpha_p + c.alpha_d * z * mu_O) / th - c.alpha_mb * (1.0 + mu_O)) / (N * (mu_L + mu_O))
    return Decision(mu_L, mu_O, N, r, gamma, th, k0, lhs, rhs, tp_eb(k0, N, c, mu_L, mu_O),
                    tp_mb(N, c, mu_L, mu_O, r), lhs < rhs, lhs > rhs_plus + delta)


# ----------------------------------------------------------------------------
# IFR correction and memory
# ----------------------------------------------------------------------------

def delta_theta(eta: float, p0: float, theta0: float, beta_d: float, N: float, alpha_d: float) -> float:
    """Delta theta = eta (1 - theta0)^2 / (p0^2 theta0) [zeta (theta0 / (1 -
    theta0) - zeta / 2) + (beta_d N / alpha_d)(zeta - theta0)]
    (Eq. delta_theta)."""
    z = zeta_of(theta0)
    rho = beta_d * N / alpha_d
    return eta * (1.0 - theta0) ** 2 / (p0 * p0 * theta0) * (z * (theta0 / (1.0 - theta0) - z / 2.0) + rho * (z - theta0))


def _nstar_den(theta: float, p0: float, mu_L: float) -> float:
    return mu_L + (1.0 - theta) / (theta * p0) * math.log(1.0 / (1.0 - theta))


def vbar(p0: float, mu_L: float) -> float:
    """Memory volatility (p0^2 mu_L)^-1 (App. "Supremum Bound")."""
    return 1.0 / (p0 * p0 * mu_L)


def n_star(C: float, eps: float, theta: float, p0: float, mu_L: float) -> int:
    """Memory-safe batch size (Eq. Nstar): OOM probability at most eps for a
    KV capacity of C tokens."""
    return int(math.floor((C - math.log(1.0 / eps) * vbar(p0, mu_L)) / _nstar_den(theta, p0, mu_L)))


def n_star_expected(C: float, theta: float, p0: float, mu_L: float) -> int:
    return int(math.floor((C - vbar(p0, mu_L)) / _nstar_den(theta, p0, mu_L)))


def n_star_static(C: float, theta: float, p0: float, mu_L: float) -> int:
    return int(math.floor(C / _nstar_den(theta, p0, mu_L)))


def kv_gate_fraction(N: int, mu_O: float, block: int, total_blocks: int, s_kv: float = 0.5, f0: float = 0.0) -> float:
    """f_KV = min(0.6, max(0.05, N mu_O s_KV / (b total_blocks) + f0))
    (App. "Runtime Refinement: KV-aware Feasibility Gate")."""
    return min(0.6, max(0.05, N * mu_O * s_kv / (block * total_blocks) + f0))


# ----------------------------------------------------------------------------
# reports
# ----------------------------------------------------------------------------

# the paper's synthetic input/output mixes (mu_L, mu_O) (Sec. 4.1)
PAPER_MIXES = ((128, 1024), (512, 512), (1024, 128))


def evaluate(c: StepCosts, mixes: Iterable[Tuple[float, float]] = PAPER_MIXES,
             Ns: Sequence[int] = (64, 256, 1024, 4096), delta: float = 0.0) -> List[dict]:
    """The decision table: for each mix and batch size, theta_0, k0*, the two
    sides of the crossover condition, both throughputs and the choices."""
    out = []
    for mu_L, mu_O in mixes:
        for N in Ns:
            d = compare(c, mu_L, mu_O, N, delta)
            out.append({k: (float(v) if isinstance(v, (float, np.floating)) else v)
                        for k, v in dataclasses.asdict(d).items()})
    return out


def crossover_in_r(c: StepCosts, total: float, N: int, rs: Optional[Sequence[float]] = None) -> dict:
    """With mu_L + mu_O fixed, the decode shares at which MB is favoured by
    the crossover condition, and the smallest share at which EB wins (None if
    MB wins everywhere on the grid)."""
    rs = np.linspace(0.02, 0.98, 49) if rs is None else rs
    fav = []
    for r in rs:
        mu_O = r * total
        d = compare(c, total - mu_O, mu_O, N)
        fav.append(bool(d.mb_favoured))
    eb = [float(r) for r, f in zip(rs, fav) if not f]
    return {"total": total, "N": N, "r": [float(r) for r in rs], "mb_favoured": fav,
            "first_eb_r": eb[0] if eb else None}
