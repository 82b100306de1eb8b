"""Pins of the U-Net band block oracle (GroupNorm -> SiLU -> conv3x3 with
stale halo rows and stale group statistics), against torch's own GroupNorm
and conv2d, brute force, and the invariants of a band step (all rows,
stitching, locality)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import unet
from oracle.blob import bf16_to_float
from seeded_inputs import configs, generate

CFG = configs.UNET_TINY


@pytest.fixture(scope="module")
def block():
    pr = generate.make_unet_params(CFG, 0)
    params = {"gamma": pr["gamma"].astype(np.float64), "beta": pr["beta"].astype(np.float64),
              "weight": bf16_to_float(pr["weight_bits"]).astype(np.float64),
              "bias": pr["bias"].astype(np.float64)}
    x = generate.make_unet_input(CFG, 0).astype(np.float64)
    return params, x


def _torch_block(params, x, groups):
    """GroupNorm -> SiLU -> conv3x3 by torch routines (NCHW)."""
    t = torch.tensor(x).permute(2, 0, 1)[None]
    y = F.group_norm(t, groups, torch.tensor(params["gamma"]), torch.tensor(params["beta"]),
                     eps=unet.GN_EPS)
    y = F.silu(y)
    w = torch.tensor(params["weight"]).permute(0, 3, 1, 2)       # [Co][C][3][3]
    o = F.conv2d(y, w, torch.tensor(params["bias"]), padding=1)
    return o[0].permute(1, 2, 0).numpy(), y[0].permute(1, 2, 0).numpy()


def test_full_map_equals_torch_groupnorm_silu_conv(block):
    params, x = block
    got = unet.full_step(params, x, CFG.groups)
    ref_out, ref_act = _torch_block(params, x, CFG.groups)
    np.testing.assert_allclose(got["act"], ref_act, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(got["out"], ref_out, rtol=1e-11, atol=1e-11)


def test_all_rows_band_ignores_stale_buffers(block):
    params, x = block
    H = CFG.height
    nan_act = np.full((H, CFG.width, CFG.channels), np.nan)
    nan_sums = np.full((H, CFG.groups, 2), np.nan)
    got = unet.band_step(params, x, H, 0, H, CFG.groups, nan_act, nan_sums)
    np.testing.assert_array_equal(got["out"], unet.full_step(params, x, CFG.groups)["out"])


def test_conv_brute_force():
    rng = np.random.default_rng(5)
    r, W, C, Co = 3, 5, 4, 3
    rows = rng.standard_normal((r + 2, W, C))
    w = rng.standard_normal((Co, 3, 3, C))
    b = rng.standard_normal(Co)
    ref = np.zeros((r, W, Co))
    for y in range(r):
        for xx in range(W):
            for o in range(Co):
                acc = b[o]
                for dy in range(3):
                    for dx in range(3):
                        sx = xx + dx - 1
                        if 0 <= sx < W:
                            for c in range(C):
                                acc += w[o, dy, dx, c] * rows[y + dy, sx, c]
                ref[y, xx, o] = acc
    np.testing.assert_allclose(unet.conv3x3_rows(rows, w, b), ref, rtol=1e-13, atol=1e-13)


def test_group_stats_closed_form(block):
    _, x = block
    sums = unet.row_group_sums(x, CFG.groups)
    mean, rstd = unet.group_stats(sums, CFG.width, CFG.channels)
    cg = CFG.channels // CFG.groups
    for g in range(CFG.groups):
        v = x[:, :, g * cg:(g + 1) * cg]
        assert abs(mean[g] - v.mean()) < 1e-12
        assert abs(1 / rstd[g] ** 2 - unet.GN_EPS - v.var()) < 1e-10


@pytest.mark.parametrize("cuts", [[0, 5, 16], [0, 1, 7, 8, 15, 16], [0, 16]])
def test_stitching_with_fresh_buffers_equals_full_map(block, cuts):
    """Buffers holding the full map's own activations and partial sums: every
    band reproduces its rows of the full map (fp64 rounding only)."""
    params, x = block
    full = unet.full_step(params, x, CFG.groups)
    act = full["act"]
    sums = unet.row_group_sums(x, CFG.groups)
    H = CFG.height
    for rb, re in zip(cuts[:-1], cuts[1:]):
        got = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, act, sums)
        np.testing.assert_allclose(got["out"], full["out"][rb:re], rtol=1e-12, atol=1e-12)


def test_locality(block):
    """Halo rows affect only the band's edge rows; stale rows beyond the halo
    do not affect anything; stale partial sums of any row move every output."""
    params, x = block
    H = CFG.height
    full = unet.full_step(params, x, CFG.groups)
    act, sums = full["act"].copy(), unet.row_group_sums(x, CFG.groups)
    rb, re = 5, 10
    base = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, act, sums)["out"]
    far = act.copy()
    far[:rb - 1] = np.nan
    far[re + 1:] = np.nan
    np.testing.assert_array_equal(
        unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, far, sums)["out"], base)
    halo = act.copy()
    halo[rb - 1] += 1.0
    o = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, halo, sums)["out"]
    assert np.abs(o[0] - base[0]).max() > 1e-3
    np.testing.assert_array_equal(o[1:], base[1:])
    halo = act.copy()
    halo[re] += 1.0
    o = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, halo, sums)["out"]
    assert np.abs(o[-1] - base[-1]).max() > 1e-3
    np.testing.assert_array_equal(o[:-1], base[:-1])
    s2 = sums.copy()
    s2[0, :, 0] += 50.0                     # another row's stale sum moves every mean
    o = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, act, s2)["out"]
    assert (np.abs(o - base).max(axis=2) > 1e-6).all()
    # the band's own rows of the buffers are never read
    own = act.copy()
    own[rb:re] = np.nan
    s3 = sums.copy()
    s3[rb:re] = np.nan
    np.testing.assert_array_equal(
        unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, own, s3)["out"], base)


def test_image_border_is_zero_padded(block):
    """A band at the top edge has no row above it: a stale buffer row there
    does not exist, and the output equals torch's zero-padded convolution."""
    params, x = block
    H = CFG.height
    full = unet.full_step(params, x, CFG.groups)
    sums = unet.row_group_sums(x, CFG.groups)
    for rb, re in ((0, 4), (12, 16)):
        got = unet.band_step(params, x[rb:re], H, rb, re, CFG.groups, full["act"], sums)
        np.testing.assert_allclose(got["out"], full["out"][rb:re], rtol=1e-12, atol=1e-12)
