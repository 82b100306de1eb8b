"""A convolutional (U-Net) block on a band of rows with stale activations (oracle).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper evaluates a U-Net denoiser (SDXL) under patch parallelism with
stale activation reuse (§II-B, DistriFusion): each device evaluates its patch
of the feature map and takes whatever it needs from the other patches from a
buffer filled at an earlier step.  A U-Net needs two such things a
transformer does not:
  * halo rows: a 3x3 convolution at the band's first and last rows reads one
    row above and one below the band, which belong to the neighbouring
    patches;
  * GroupNorm statistics: the mean and variance of a channel group are taken
    over the whole feature map, not the band.

This module computes the first half of a U-Net ResNet block on a band:
GroupNorm -> SiLU -> 3x3 convolution (stride 1, zero padding 1), with:
  * the band's own rows fresh;
  * halo rows read from the stale buffer of the convolution's input (the
    SiLU(GroupNorm(x)) activations of the previous step), zero outside the
    feature map;
  * the group statistics assembled from per-row partial sums: the band's
    rows fresh, every other row's from the stale buffer of partial sums.

Readings (the paper does not restate the U-Net):
  * block order GroupNorm -> SiLU -> conv3x3 (+ bias), GroupNorm with a
    per-channel affine (gamma, beta), eps 1e-5, biased variance;
  * a row's partial sums are (sum x, sum x^2) over the row's pixels and the
    group's channels; mean = S / N and var = Q / N - mean^2 with N the
    group's element count over the whole map;
  * layouts are pixel-major (NHWC): x [rows][W][C], activations [H][W][C],
    partial sums [H][G][2], conv weight [C_out][3][3][C_in].

Everything is float64; a band of every row ignores the stale buffers.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

GN_EPS = 1e-5


def silu(x):
    return x / (1.0 + np.exp(-x))


def row_group_sums(x_rows, groups: int):
    """Per row and channel group: (sum, sum of squares) over the row's
    pixels and the group's channels.  x_rows [r, W, C] -> [r, G, 2]."""
    x = np.asarray(x_rows, dtype=np.float64)
    r, W, C = x.shape
    xg = x.reshape(r, W, groups, C // groups)
    s = xg.sum(axis=(1, 3))
    q = (xg * xg).sum(axis=(1, 3))
    return np.stack([s, q], axis=-1)


def group_stats(sums_all_rows, W: int, C: int, eps: float = GN_EPS):
    """Mean and 1/sqrt(var + eps) per group from every row's partial sums
    [H, G, 2]."""
    sums = np.asarray(sums_all_rows, dtype=np.float64)
    H, G, _ = sums.shape
    n = H * W * (C // G)
    S = sums[:, :, 0].sum(axis=0)
    Q = sums[:, :, 1].sum(axis=0)
    mean = S / n
    var = Q / n - mean * mean
    return mean, 1.0 / np.sqrt(var + eps)


def gn_silu(x_rows, mean, rstd, gamma, beta):
    """SiLU(GroupNorm(x)) on rows [r, W, C] given the group statistics."""
    x = np.asarray(x_rows, dtype=np.float64)
    r, W, C = x.shape
    G = mean.shape[0]
    xg = x.reshape(r, W, G, C // G)
    y = ((xg - mean[None, None, :, None]) * rstd[None, None, :, None]).reshape(r, W, C)
    return silu(y * gamma + beta)


def conv3x3_rows(act_rows, weight, bias):
    """3x3 convolution, stride 1, of rows that already carry one halo row
    above and below: act_rows [r + 2, W, C_in] -> [r, W, C_out].  Columns are
    zero-padded; out = bias + sum over (dy, dx, c) of w[o, dy, dx, c] *
    act[y + dy - 1, x + dx - 1, c]."""
    a = np.asarray(act_rows, dtype=np.float64)
    w = np.asarray(weight, dtype=np.float64)
    r2, W, C = a.shape
    r = r2 - 2
    Co = w.shape[0]
    pad = np.zeros((r2, W + 2, C))
    pad[:, 1:W + 1] = a
    out = np.zeros((r, W, Co)) + np.asarray(bias, dtype=np.float64)
    for dy in range(3):
        for dx in range(3):
            win = pad[dy:dy + r, dx:dx + W].reshape(r * W, C)
            out += (win @ w[:, dy, dx, :].T).reshape(r, W, Co)
    return out


def band_step(params: Dict, x_band, H: int, row_begin: int, row_end: int, groups: int,
              stale_act=None, stale_sums=None, eps: float = GN_EPS) -> Dict:
    """GroupNorm -> SiLU -> conv3x3 on the band's rows [row_begin, row_end) of
    an H-row feature map.

    x_band      [r, W, C]: the block input on the band's rows (fresh).
    stale_act   [H, W, C]: the convolution input of an earlier step (read for
                the halo rows outside the band).
    stale_sums  [H, G, 2]: per-row partial sums of an earlier step (read for
                every row outside the band).
    Returns out [r, W, C_out], act [r, W, C] (the band's conv input, what a
    refresh stores) and sums [r, G, 2] (the band's partial sums).
    """
    x = np.asarray(x_band, dtype=np.float64)
    r, W, C = x.shape
    if r != row_end - row_begin or not (0 <= row_begin < row_end <= H):
        raise ValueError("band rows do not match x_band")
    full = row_begin == 0 and row_end == H
    if not full and (stale_act is None or stale_sums is None):
        raise ValueError("a band of fewer than all rows needs the stale buffers")
    fresh = row_group_sums(x, groups)
    if full:
        all_sums = fresh
    else:
        all_sums = np.array(stale_sums, dtype=np.float64, copy=True)
        all_sums[row_begin:row_end] = fresh
    mean, rstd = group_stats(all_sums, W, C, eps)
    act = gn_silu(x, mean, rstd, params["gamma"], params["beta"])
    # convolution input rows row_begin - 1 .. row_end: fresh band, stale halo
    rows = np.zeros((r + 2, W, C))
    rows[1:r + 1] = act
    for k, y in ((0, row_begin - 1), (r + 1, row_end)):
        if 0 <= y < H:
            rows[k] = np.asarray(stale_act[y], dtype=np.float64)
    out = conv3x3_rows(rows, params["weight"], params["bias"])
    return {"out": out, "act": act, "sums": fresh, "mean": mean, "rstd": rstd}


def full_step(params: Dict, x_full, groups: int, eps: float = GN_EPS) -> Dict:
    """The unpartitioned block: the band is every row, nothing is stale."""
    H = np.asarray(x_full).shape[0]
    return band_step(params, x_full, H, 0, H, groups, eps=eps)
