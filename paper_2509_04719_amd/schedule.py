"""Host-side step schedules of the sampler (no device work).

* Uniform DDIM grid: tau_k = k T / M, k = 0..M-1, sampled in descending
  order; the final target is -1 (alpha_bar = 1).
* Reduced tier of the tiered step reduction (Algorithm 1, slow branch; Eq. (2)
  middle case): the first M_warmup grid steps run one by one, then steps of
  two grid intervals (Theorem 2 with n = 2) until the end; the buffer is
  refreshed on every executed step.  That gives ceil((M_base + M_warmup)/2)
  steps (Eq. (2)'s M_base/2 + M_warmup/2, rounded up).
"""
from __future__ import annotations

from typing import List, NamedTuple


class Step(NamedTuple):
    m: int          # index on the M-step grid
    t: int          # source timestep
    t_prev: int     # target timestep (-1: final)
    refresh: bool   # write the band's fresh K/V into the buffer


def grid_desc(T: int, M: int) -> List[int]:
    """t_0 > t_1 > ... > t_{M-1}, then the final target -1."""
    return [(M - 1 - m) * T // M for m in range(M)] + [-1]


def plain_schedule(T: int, M: int) -> List[Step]:
    g = grid_desc(T, M)
    return [Step(m, g[m], g[m + 1], True) for m in range(M)]


def tiered_schedule(T: int, M_base: int, M_warmup: int) -> List[Step]:
    g = grid_desc(T, M_base)
    steps, m = [], 0
    while m < M_base:
        nxt = m + 1 if m < M_warmup else min(m + 2, M_base)
        steps.append(Step(m, g[m], g[nxt], True))
        m = nxt
    return steps


def band_rows(share: float, R: int) -> int:
    """Rows of an elastic band holding `share` of R rows (round half up, >= 1)."""
    return max(1, min(R, int(share * R + 0.5)))
