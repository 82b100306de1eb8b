"""Samplers (oracle): the plain full-image DDIM sampler and Algorithm 1's
patch-parallel sampler over N virtual devices.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Patch-parallel sampler (Algorithm 1, §III-B; stale activations of §II-B).
Device i owns the token rows [splits[i], splits[i+1]) and a tier (0: every
step of the grid, 1: the reduced tier of Eq. (2)).  Readings (the algorithm
leaves these open for a simulation on one machine):
  * Warm-up steps m < M_warmup exchange the buffer synchronously inside the
    step, so every device attends over the current step's K/V of every
    token: the warm-up step is the full-image step, and the buffer afterwards
    holds that step's K/V.
  * After warm-up the grid is covered in sync intervals of two steps (one if
    a single step is left).  In an interval every device reads the buffer as
    it was at the interval's start for the other devices' tokens (its own
    tokens are always fresh).  A tier-0 device runs t_m -> t_{m+1}, whose K/V
    it exchanges, then t_{m+1} -> t_{m+2} from its own half-step result, whose
    K/V it keeps ("no update for buffer" on odd offsets).  A tier-1 device
    runs t_m -> t_{m+2} and exchanges its K/V.  At the interval's end the
    exchanged K/V form the next buffer and the bands of x are gathered.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from . import dit


def full_sample(hdr, params, x_T, t_grid: Sequence[int], labels, cfg_scale: float,
                dtype=np.float64):
    """Full-image DDIM over the grid t_grid[0] > ... > t_grid[-1] = -1."""
    x = np.asarray(x_T, dtype=np.float64)
    for t, tp in zip(t_grid[:-1], t_grid[1:]):
        x = dit.full_step(hdr, params, x, t, tp, labels, cfg_scale, dtype=dtype)["x_out"]
    return x


def patch_parallel_sample(hdr, params, x_T, splits: Sequence[int], tiers: Sequence[int],
                          t_grid: Sequence[int], warmup: int, labels, cfg_scale: float,
                          dtype=np.float64, order: Optional[Sequence[int]] = None):
    """Algorithm 1 on len(tiers) virtual devices; returns the final latent.

    order: the order in which this simulation visits the devices within an
    interval (default: by index).  The devices of Algorithm 1 run in
    parallel, so the result does not depend on it."""
    M = len(t_grid) - 1
    if not 1 <= warmup <= M:
        raise ValueError("need 1 <= warmup <= steps")
    p = hdr["patch"]
    x = np.asarray(x_T, dtype=np.float64)
    buf = None
    for m in range(warmup):
        r = dit.full_step(hdr, params, x, t_grid[m], t_grid[m + 1], labels, cfg_scale,
                          dtype=dtype, keep_kv=True)
        x = r["x_out"]
        buf = dit.full_kv_buffer(hdr, r["kv"])
    m = warmup
    while m < M:
        m2 = min(m + 2, M)
        nxt = buf.copy()
        x_next = x.copy()
        for i in (range(len(tiers)) if order is None else order):
            tier = tiers[i]
            rb, re = splits[i], splits[i + 1]
            rows = slice(rb * p, re * p)
            if tier == 0 and m2 == m + 2:
                a = dit.patch_step(hdr, params, x, rb, re, t_grid[m], t_grid[m + 1], labels,
                                   cfg_scale, buf, dtype=dtype, keep_kv=True)
                nxt = dit.refreshed_buffer(hdr, nxt, a["kv"], rb, re)
                x_mid = x.copy()
                x_mid[:, rows, :] = a["x_out"]
                b = dit.patch_step(hdr, params, x_mid, rb, re, t_grid[m + 1], t_grid[m + 2],
                                   labels, cfg_scale, buf, dtype=dtype)
                x_next[:, rows, :] = b["x_out"]
            else:
                a = dit.patch_step(hdr, params, x, rb, re, t_grid[m], t_grid[m2], labels,
                                   cfg_scale, buf, dtype=dtype, keep_kv=True)
                nxt = dit.refreshed_buffer(hdr, nxt, a["kv"], rb, re)
                x_next[:, rows, :] = a["x_out"]
        buf, x = nxt, x_next
        m = m2
    return x
