"""Device planning of the method (oracle): temporal and spatial adaptation.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Temporal adaptation (Eq. (2), §III-C): with v_max the largest effective
speed, a device keeps M_base steps when a*v_max < v_i, takes the reduced tier
M_base/2 + M_warmup/2 when b*v_max < v_i <= a*v_max, and is excluded when
v_i <= b*v_max (0 < b < a < 1).  The evaluation (§V-A) uses a = 0.75,
b = 0.25.

Spatial adaptation, patch mending (Eq. (3), §III-D): device i gets the share
(v_i/M_i) / sum_j (v_j/M_j) of the image, over the devices not excluded.

Readings (the paper leaves these open):
  * The effective speed is v_i = c_i * (1 - rho_i) (capability times idle
    fraction); the planner also takes v directly.
  * The reduced tier has ceil((M_base + M_warmup) / 2) steps: M_warmup single
    steps, then the rest of the grid in steps of two intervals, the last one
    single when M_base - M_warmup is odd -- the count the reduced-tier
    schedule executes (Table II's 100:52 and 50:27 at M_warmup = 4; 63 for
    M_base = 100, M_warmup = 25).
  * A device whose share rounds to no rows has no work: it runs 0 steps.
  * Shares are turned into whole token rows by largest remainders: each device
    gets floor(P_i), the rows left over go to the largest fractional parts,
    ties to the lower index; the rows always sum to P_total.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np


def effective_speed(c: float, rho: float) -> float:
    return c * (1.0 - rho)


def speed_from_profile(rows: Sequence[int], ms: Sequence[float], ref_rows: int) -> float:
    """Effective speed from an inference time profile (§V-A: speeds derived
    from historical inference times; the paper gives no formula).  Reading:
    the step times are a fixed per-step cost plus a per-row cost, fitted by
    least squares, t = alpha + beta * rows; the speed is the rows per unit time
    at the reference band height, ref_rows / (alpha + beta * ref_rows).  A
    single height fixes only beta = mean(t / rows) with alpha = 0."""
    r = np.asarray(rows, dtype=np.float64)
    t = np.asarray(ms, dtype=np.float64)
    if np.all(r == r[0]):
        alpha, beta = 0.0, t.sum() / r.sum()
    else:
        A = np.stack([np.ones_like(r), r], axis=1)
        alpha, beta = np.linalg.lstsq(A, t, rcond=None)[0]
    return ref_rows / (alpha + beta * ref_rows)


def reduced_steps(M_base: int, M_warmup: int) -> int:
    """Eq. (2), middle case: M_warmup single steps, then ceil of half the rest."""
    return M_warmup + (M_base - M_warmup + 1) // 2


def step_counts(v: Sequence[float], M_base: int, M_warmup: int, a: float, b: float) -> List[int]:
    """Eq. (2): steps per device, 0 for an excluded device."""
    vmax = max(v)
    out = []
    for vi in v:
        if vi > a * vmax:
            out.append(M_base)
        elif vi > b * vmax:
            out.append(reduced_steps(M_base, M_warmup))
        else:
            out.append(0)
    return out


def patch_shares(v: Sequence[float], steps: Sequence[int]) -> List[float]:
    """Eq. (3) with P_total = 1: (v_i/M_i) / sum_j (v_j/M_j); 0 when excluded."""
    rate = [vi / m if m > 0 else 0.0 for vi, m in zip(v, steps)]
    tot = sum(rate)
    return [r / tot for r in rate]


def whole_rows(shares: Sequence[float], total: int) -> List[int]:
    """Largest-remainder rounding of shares * total to integers summing to total."""
    exact = [s * total for s in shares]
    rows = [int(math.floor(e)) for e in exact]
    left = total - sum(rows)
    order = sorted(range(len(exact)), key=lambda i: (-(exact[i] - rows[i]), i))
    for i in order[:left]:
        rows[i] += 1
    return rows


def plan(v: Sequence[float], M_base: int, M_warmup: int, a: float, b: float, total_rows: int
         ) -> Tuple[List[int], List[int]]:
    """(steps, rows) per device: Eq. (2) then Eq. (3) in whole rows."""
    steps = step_counts(v, M_base, M_warmup, a, b)
    rows = whole_rows(patch_shares(v, steps), total_rows)
    steps = [m if r > 0 else 0 for m, r in zip(steps, rows)]
    return steps, rows
