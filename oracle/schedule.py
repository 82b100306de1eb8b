"""Noise schedule and scheduler coefficients (oracle).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The reverse step in §I updates the noisy sample as
    x_t = (alpha_t / alpha_{t+1}) x_{t+1} - s(t, t-1) eps + sigma_{t+1} z ,
and Lemma 1 (Eq. (1), §II-A) fixes the eps coefficient of the first-order
solver (DDIM): with lambda = log(alpha / sigma) and h = lambda_target -
lambda_source, the coefficient is sigma_target * (e^h - 1).

Readings (the paper leaves these open):
  * alpha_t = sqrt(abar_t), sigma_t = sqrt(1 - abar_t) (variance preserving),
    abar_n = prod_{i<=n} (1 - beta_i), beta = linspace(beta_start, beta_end, T)
    with both ends included.
  * The target index -1 means abar = 1 (alpha = 1, sigma = 0): the final step.
  * Eq. (1) is evaluated in the rearranged form
        Bc = alpha_p * sigma_s / alpha_s - sigma_p ,
    algebraically equal to sigma_p (e^h - 1) and finite at sigma_p = 0.
  * The z term: for eta > 0 the eta-DDIM form with
        c = eta * sqrt((1 - abar_p) / (1 - abar_s)) * sqrt(1 - abar_s / abar_p)
    and Bc = alpha_p sigma_s / alpha_s - sqrt(1 - abar_p - c^2); eta = 0
    gives c = 0 and Eq. (1) exactly.
  * DDIM grid: tau_k = k * T / M, k = 0..M-1, sampled in descending order.
"""
from __future__ import annotations

import math
from typing import List, Tuple

import numpy as np


def betas(T: int = 1000, beta_start: float = 1e-4, beta_end: float = 2e-2) -> np.ndarray:
    return np.linspace(beta_start, beta_end, T, dtype=np.float64)


def alpha_bar(T: int = 1000, beta_start: float = 1e-4, beta_end: float = 2e-2) -> np.ndarray:
    return np.cumprod(1.0 - betas(T, beta_start, beta_end))


def _abar(ab: np.ndarray, t: int) -> float:
    return 1.0 if t < 0 else float(ab[t])


def alpha_sigma(ab: np.ndarray, t: int) -> Tuple[float, float]:
    a = _abar(ab, t)
    return math.sqrt(a), math.sqrt(1.0 - a)


def log_snr(ab: np.ndarray, t: int) -> float:
    """lambda_t = log(alpha_t / sigma_t)."""
    a, s = alpha_sigma(ab, t)
    return math.log(a / s)


def ddim_coefficients(ab: np.ndarray, t: int, t_prev: int, eta: float = 0.0
                      ) -> Tuple[float, float, float]:
    """(A, Bc, C) with x_prev = A x - Bc eps + C z for the step t -> t_prev."""
    ab_s, ab_p = _abar(ab, t), _abar(ab, t_prev)
    a_s, s_s = math.sqrt(ab_s), math.sqrt(1.0 - ab_s)
    a_p = math.sqrt(ab_p)
    c = 0.0
    if eta > 0.0:
        c = eta * math.sqrt((1.0 - ab_p) / (1.0 - ab_s)) * math.sqrt(1.0 - ab_s / ab_p)
    A = a_p / a_s
    Bc = a_p * s_s / a_s - math.sqrt(max(0.0, 1.0 - ab_p - c * c))
    return A, Bc, c


def lemma1_coefficients(ab: np.ndarray, t: int, t_prev: int) -> Tuple[float, float]:
    """Eq. (1) as printed: A = alpha_p/alpha_s, Bc = sigma_p (e^h - 1),
    h = lambda_p - lambda_s.  Undefined at t_prev = -1 (sigma_p = 0)."""
    if t_prev < 0:
        raise ValueError("Eq. (1) as printed is 0 * inf at the final step")
    a_s, _ = alpha_sigma(ab, t)
    a_p, s_p = alpha_sigma(ab, t_prev)
    h = log_snr(ab, t_prev) - log_snr(ab, t)
    return a_p / a_s, s_p * math.expm1(h)


def scheduler_update(x: np.ndarray, eps: np.ndarray, A: float, Bc: float,
                     C: float = 0.0, z: np.ndarray | None = None) -> np.ndarray:
    """The elementwise update of §I: x_prev = A x - Bc eps + C z."""
    out = A * np.asarray(x, dtype=np.float64) - Bc * np.asarray(eps, dtype=np.float64)
    if C != 0.0:
        out = out + C * np.asarray(z, dtype=np.float64)
    return out


def ddim_grid(T: int, M: int) -> List[int]:
    """tau_k = k T / M for k = 0..M-1 (ascending)."""
    return [k * T // M for k in range(M)]


def step_pairs(T: int, M: int) -> List[Tuple[int, int]]:
    """Descending (t, t_prev) pairs of the M-step sampler; the last target is -1."""
    g = ddim_grid(T, M)
    seq = list(reversed(g)) + [-1]
    return [(seq[m], seq[m + 1]) for m in range(M)]


def tiered_step_count(M_base: int, M_warmup: int) -> int:
    """Eq. (2), middle case: steps of a device in the reduced tier,
    M_base/2 + M_warmup/2 rounded up -- M_warmup single steps, then the rest
    of the grid in steps of two intervals (the last one single when
    M_base - M_warmup is odd)."""
    return -(-(M_base + M_warmup) // 2)


def tiered_schedule(T: int, M_base: int, M_warmup: int
                    ) -> List[Tuple[int, int, int, bool]]:
    """Executed steps of a reduced-tier device (Algorithm 1, slow branch; Eq. (2)).

    The first M_warmup grid steps run one by one; after that the device
    covers the remaining grid with steps of two intervals (Theorem 2 with
    n = 2), refreshing its buffer on every executed step.
    Returns (m, t, t_prev, refresh) for each executed step.
    """
    g = ddim_grid(T, M_base)
    seq = list(reversed(g)) + [-1]          # seq[m] = t_m, seq[M_base] = -1
    out = []
    m = 0
    while m < M_base:
        stride = 1 if m < M_warmup else 2
        nxt = min(m + stride, M_base)
        out.append((m, seq[m], seq[nxt], True))
        m = nxt
    return out
