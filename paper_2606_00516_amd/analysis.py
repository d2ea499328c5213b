"""Derived statistics of measured step times (host-side arithmetic).

These are the quantities the paper builds its EB-vs-MB decision on, computed
from step latencies measured on this GPU:

* the linear iteration-time model T_iter = alpha + beta * n_tok and the decode
  ratio r = n_decode / n_tok (Sec. 1), with the R^2 of the fit (App. A.1,
  Table linear-r2-practical);
* the crossover decode ratio: the smallest r at which the mixed-batch marginal
  cost beta(r) reaches the pure-decode one beta(1) (Sec. 1, Fig. marginal_cost);
* the EB cost line K_bar(r) = (1 - r) K(0) + r K(1) between pure-prefill and
  pure-decode kernel time, the quadratic fit K(r) = c0 + c1 r + c2 r^2, the gap
  K(r) - K_bar(r) = -c2 r (1 - r) and the interference convexity index
  kappa = 2 c2 / (c0 + c1 + c2) (App. A.3, Eqs. gap_proportional, fL_diff,
  convexity_index).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


def linear_fit(n_tok: Sequence[float], t: Sequence[float]) -> Tuple[float, float, float]:
    """Least-squares T = alpha + beta n_tok; returns (alpha, beta, R^2)."""
    x = np.asarray(n_tok, np.float64)
    y = np.asarray(t, np.float64)
    A = np.stack([np.ones_like(x), x], axis=1)
    (alpha, beta), *_ = np.linalg.lstsq(A, y, rcond=None)
    pred = alpha + beta * x
    ss_res = float(np.sum((y - pred) ** 2))
    ss_tot = float(np.sum((y - y.mean()) ** 2))
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0
    return float(alpha), float(beta), r2


def quad_fit(r: Sequence[float], k: Sequence[float]) -> Tuple[float, float, float]:
    """Least-squares K(r) = c0 + c1 r + c2 r^2; returns (c0, c1, c2)."""
    r = np.asarray(r, np.float64)
    k = np.asarray(k, np.float64)
    A = np.stack([np.ones_like(r), r, r * r], axis=1)
    (c0, c1, c2), *_ = np.linalg.lstsq(A, k, rcond=None)
    return float(c0), float(c1), float(c2)


def kappa(c0: float, c1: float, c2: float) -> float:
    """Interference convexity index: 2 c2 normalised by K(1) = c0 + c1 + c2."""
    return 2.0 * c2 / (c0 + c1 + c2)


def eb_line(r: Sequence[float], k0: float, k1: float) -> np.ndarray:
    """Linear interpolation between the pure-prefill and pure-decode costs."""
    r = np.asarray(r, np.float64)
    return (1.0 - r) * k0 + r * k1


def crossover_primary(r: Sequence[float], beta: Sequence[float]) -> Optional[float]:
    """Smallest r in [0, 1) with beta(r) >= beta(1), linearly interpolated
    between grid points; None if beta stays below beta(1) on [0, 1)."""
    r = np.asarray(r, np.float64)
    b = np.asarray(beta, np.float64)
    order = np.argsort(r)
    r, b = r[order], b[order]
    assert abs(r[-1] - 1.0) < 1e-9, "the grid must end at r = 1"
    target = b[-1]
    for i in range(len(r) - 1):
        if b[i] >= target:
            if i == 0:
                return float(r[0])
            # interpolate between i-1 (below) and i (at or above)
            r0, r1, b0, b1 = r[i - 1], r[i], b[i - 1], b[i]
            return float(r0 + (target - b0) * (r1 - r0) / (b1 - b0)) if b1 != b0 else float(r1)
    return None


def eb_favoured(r: Sequence[float], k: Sequence[float], noise: float) -> List[float]:
    """Grid points where the mixed step costs more than the EB line by more
    than ``noise`` (the saturated-limit reading of Eq. comparison_condition)."""
    r = np.asarray(r, np.float64)
    k = np.asarray(k, np.float64)
    kb = eb_line(r, k[np.argmin(r)], k[np.argmax(r)])
    return [float(x) for x, g in zip(r, k - kb) if g > noise]


def sweep_report(r: Sequence[float], k: Sequence[float]) -> Dict[str, float]:
    """Quadratic fit, kappa and the largest gap K - K_bar of a decode-share sweep."""
    c0, c1, c2 = quad_fit(r, k)
    r_arr = np.asarray(r, np.float64)
    k_arr = np.asarray(k, np.float64)
    gap = k_arr - eb_line(r_arr, k_arr[np.argmin(r_arr)], k_arr[np.argmax(r_arr)])
    i = int(np.argmax(gap))
    return {"c0": c0, "c1": c1, "c2": c2, "kappa": kappa(c0, c1, c2),
            "max_gap": float(gap[i]), "r_at_max_gap": float(r_arr[i])}
