"""Calibration constants of the method (test infrastructure only).

Sec. 3.4, Eq. "scale":  scale^(l) = alpha * sigma^(l) * (d / sqrt(d_h)) / (eta_fp8 * R_max),
with R_safe = eta_fp8 * R_max = 0.8 * 448 = 358.4 in all of the paper's runs.

Sec. 3.2, Prop. "Rank-aware overflow probability bound" and the selection
rule that follows it (Eqs. "gamma_selection", "alpha_selection"):

    T1 = L exp(-(d_h / 2) h(gamma)),   h(gamma) = gamma - 1 - ln gamma
    T2 = 2 L^2 exp(-d^2 alpha^2 / (2 gamma d_h))
    gamma: smallest gamma > 1 with h(gamma) >= (2 / d_h) ln(2 N L / delta*)
    alpha_min = sqrt(2 gamma d_h) / d * sqrt(ln(4 N L^2 / delta*))

N = n_layers * n_heads (the union bound over heads).
"""

from __future__ import annotations

import math


def scale_factor(sigma_layer: float, alpha: float, d: int, head_dim: int,
                 eta_fp8: float = 0.8, r_max: float = 448.0) -> float:
    b_alpha = alpha * sigma_layer * d / math.sqrt(head_dim)     # calibrated bound B_alpha
    r_safe = eta_fp8 * r_max
    return b_alpha / r_safe


def h_gamma(gamma: float) -> float:
    return gamma - 1.0 - math.log(gamma)


def gamma_select(head_dim: int, n_heads_total: int, seq_len: int, delta: float) -> float:
    """Smallest gamma > 1 meeting Eq. "gamma_selection" (h is increasing on
    (1, inf), so bisection on [1, 1e6])."""
    rhs = 2.0 / head_dim * math.log(2.0 * n_heads_total * seq_len / delta)
    lo, hi = 1.0, 1.0e6
    for _ in range(400):
        mid = 0.5 * (lo + hi)
        if h_gamma(mid) >= rhs:
            hi = mid
        else:
            lo = mid
    return hi


def alpha_min(d: int, head_dim: int, n_heads_total: int, seq_len: int, delta: float) -> float:
    gamma = gamma_select(head_dim, n_heads_total, seq_len, delta)
    return math.sqrt(2.0 * gamma * head_dim) / d * math.sqrt(
        math.log(4.0 * n_heads_total * seq_len ** 2 / delta))


def overflow_terms(d: int, head_dim: int, seq_len: int, alpha: float, gamma: float):
    """(T1, T2) of Prop. "Rank-aware overflow probability bound"."""
    t1 = seq_len * math.exp(-0.5 * head_dim * h_gamma(gamma))
    t2 = 2.0 * seq_len ** 2 * math.exp(-(d * d * alpha * alpha) / (2.0 * gamma * head_dim))
    return t1, t2


def rank_aware_improvement(d: int, head_dim: int, gamma: float) -> float:
    """Exponent ratio d / (gamma d_h) of Table "concentration"."""
    return d / (gamma * head_dim)


def slack_ratio(max_abs_logit: float, sigma_layer: float, d: int, head_dim: int) -> float:
    """r_t = max|S| / B_max (Sec. 3.5), B_max = sigma * d / sqrt(d_h) (Eq. "bound")."""
    return max_abs_logit / (sigma_layer * d / math.sqrt(head_dim))


def auto_alpha(slack_ratios, quantile: float = 0.9999, kappa: float = 1.0) -> float:
    """Algorithm "Auto-alpha Calibration" (App. M): Quantile_q(R) * kappa.
    The quantile is numpy's default (linear interpolation between order
    statistics); the paper does not name an estimator."""
    import numpy as np

    return float(np.quantile(np.asarray(slack_ratios, dtype=np.float64), quantile)) * kappa


def utilization(max_abs_logit: float, scale: float, r_max: float = 448.0) -> float:
    """FP8 range utilisation max|S| / (scale * R_max) (Sec. 1, "Utilization")."""
    return max_abs_logit / (scale * r_max)
