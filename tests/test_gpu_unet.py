"""Oracle parity of the U-Net band block (GroupNorm -> SiLU -> conv3x3 with
stale halo rows and stale group statistics) through the C ABI.

The stale buffers are the oracle's full-map computation on an independent
seeded input (what the previous step of every device would leave), rounded
to the buffers' storage types; the same values go to both sides.  Tolerance:
relative L2 <= 1e-2 on the output, whole band and every row (the GPU rounds
the convolution input to bf16; the oracle is float64), 1e-2 on the refreshed
activations (bf16) and 1e-5 on the refreshed partial sums (fp32).
"""
import functools

import numpy as np
import pytest
import torch

from oracle import unet
from oracle.blob import bf16_to_float
from seeded_inputs import configs, generate
from tests._gpu_util import DEV, rel_l2, to_host

pytestmark = pytest.mark.gpu

EPS = 1e-5


@functools.lru_cache(maxsize=2)
def _setup(name):
    cfg = {c.name: c for c in configs.UNET_CONFIGS}[name]
    pr = generate.make_unet_params(cfg, 0)
    params = {"gamma": pr["gamma"].astype(np.float64), "beta": pr["beta"].astype(np.float64),
              "weight": bf16_to_float(pr["weight_bits"]).astype(np.float64),
              "bias": pr["bias"].astype(np.float64)}
    x = generate.make_unet_input(cfg, 0)
    # stale buffers: the full map of an independent input, in storage types
    prev = unet.full_step(params, generate.make_unet_input(cfg, 1).astype(np.float64), cfg.groups)
    act_bits = generate.f32_to_bf16_bits(prev["act"].astype(np.float32))
    sums = unet.row_group_sums(generate.make_unet_input(cfg, 1), cfg.groups).astype(np.float32)
    return cfg, pr, params, x, act_bits, sums


def _dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def _row_rel(got, ref):
    g = got.reshape(got.shape[0], -1)
    r = ref.reshape(ref.shape[0], -1)
    return float((np.linalg.norm(g - r, axis=1) / np.linalg.norm(r, axis=1)).max())


def _run(orch_lib, name, rb, re, refresh):
    cfg, pr, params, x, act_bits, sums = _setup(name)
    H, W, C, Co, G = cfg.height, cfg.width, cfg.channels, cfg.out_channels, cfg.groups
    print(f"\n[{name} band [{rb},{re}) of {H} rows, refresh {refresh}]", flush=True)
    shape = orch_lib.unet_shape(cfg, EPS)
    act_d = _dev_bf16(act_bits)
    sums_d = torch.from_numpy(sums).to(DEV)
    ws = torch.empty(orch_lib.unet_conv_workspace_bytes(shape, re - rb), dtype=torch.uint8, device=DEV)
    out = torch.full((re - rb, W, Co), float("nan"), device=DEV)
    orch_lib.unet_conv_band(shape, rb, re, torch.from_numpy(x[rb:re].copy()).to(DEV),
                            torch.from_numpy(pr["gamma"]).to(DEV), torch.from_numpy(pr["beta"]).to(DEV),
                            _dev_bf16(pr["weight_bits"]), torch.from_numpy(pr["bias"]).to(DEV),
                            act_d, sums_d, refresh, out, ws)
    got = to_host(out)
    ref = unet.band_step(params, x[rb:re].astype(np.float64), H, rb, re, G,
                         bf16_to_float(act_bits).astype(np.float64), sums.astype(np.float64), EPS)
    e, m = rel_l2(got, ref["out"]), _row_rel(got, ref["out"])
    print(f"  out rel-L2 {e:.2e}, worst row {m:.2e}", flush=True)
    assert e <= 1e-2 and m <= 1e-2, (e, m)
    act_h = to_host(act_d)
    sums_h = to_host(sums_d)
    old_act = bf16_to_float(act_bits).astype(np.float64)
    if refresh:
        assert rel_l2(act_h[rb:re], ref["act"]) <= 1e-2
        assert rel_l2(sums_h[rb:re], ref["sums"]) <= 1e-5
    else:
        np.testing.assert_array_equal(act_h[rb:re], old_act[rb:re])
        np.testing.assert_array_equal(sums_h[rb:re], sums[rb:re])
    np.testing.assert_array_equal(np.delete(act_h, np.s_[rb:re], 0), np.delete(old_act, np.s_[rb:re], 0))
    np.testing.assert_array_equal(np.delete(sums_h, np.s_[rb:re], 0), np.delete(sums, np.s_[rb:re], 0))


@pytest.mark.parametrize("rb,re,refresh", [(0, 5, 1), (5, 11, 0), (11, 16, 1), (0, 16, 0), (7, 8, 1)])
def test_unet_tiny(orch_lib, rb, re, refresh):
    _run(orch_lib, "unet_tiny", rb, re, refresh)


# SDXL-sized first stage at 1024px: 1/8 interior, the evaluation's 14 and 18
# patch units (56 and 72 rows) at the head and the tail, every row
@pytest.mark.parametrize("rb,re,refresh", [(56, 72, 1), (0, 56, 0), (56, 128, 1), (0, 128, 1)],
                         ids=["1/8", "14/32", "18/32", "all"])
def test_unet_sdxl_stage1(orch_lib, rb, re, refresh):
    _run(orch_lib, "unet_sdxl_1024_stage1", rb, re, refresh)


# the deeper stages: 64 x 64 x 640 and 32 x 32 x 1280 (bands at the same shares)
@pytest.mark.parametrize("name,rows", [("unet_sdxl_1024_stage2", 64), ("unet_sdxl_1024_stage3", 32)],
                         ids=["stage2", "stage3"])
@pytest.mark.parametrize("share", ["1/8", "14/32", "18/32", "all"])
def test_unet_sdxl_deeper_stages(orch_lib, name, rows, share):
    rb, re, refresh = {"1/8": (7 * rows // 16, 9 * rows // 16, 1), "14/32": (0, 14 * rows // 32, 0),
                       "18/32": (14 * rows // 32, rows, 1), "all": (0, rows, 1)}[share]
    _run(orch_lib, name, rb, re, refresh)


# 120 x 120 x 192 -> 320: every row (the whole map in 160-channel tiles, the
# last pixel tile partial), an interior band (64-channel tiles) and a 26-row
# band (160-channel tiles, k-tiles split three ways, the last pixel tile
# partial)
@pytest.mark.parametrize("rb,re,refresh", [(0, 120, 1), (30, 90, 0), (40, 66, 1)],
                         ids=["all", "interior", "26 rows"])
def test_unet_ragged_320_channels(orch_lib, rb, re, refresh):
    _run(orch_lib, "unet_ragged_320", rb, re, refresh)


def test_unet_stitching_with_own_buffers(orch_lib):
    """The all-rows pass with refresh fills both buffers; bands then read
    their halo rows and the other rows' sums from them.  Refreshing, the
    bands rewrite both buffers bit for bit (a row's sums and the group
    statistics are added in an order fixed by the rows alone), and their
    outputs stitch to the all-rows output up to the order of the
    convolution's sums: a launch with few tiles splits its k-tiles over more
    workgroups and adds their partial sums (the all-rows pass of this stage
    does not split).  A repeated band gives the same bits."""
    cfg, pr, _, x, _, _ = _setup("unet_sdxl_1024_stage1")
    H, W, C, Co, G = cfg.height, cfg.width, cfg.channels, cfg.out_channels, cfg.groups
    shape = orch_lib.unet_shape(cfg, EPS)
    dev = {k: torch.from_numpy(v).to(DEV) for k, v in pr.items() if k != "weight_bits"}
    wt = _dev_bf16(pr["weight_bits"])
    xd = torch.from_numpy(x).to(DEV)
    act = torch.full((H, W, C), float("nan"), dtype=torch.bfloat16, device=DEV)
    sums = torch.full((H, G, 2), float("nan"), device=DEV)
    cut_sets = ([0, 56, 128], [0, 16, 40, 72, 73, 128])
    heights = {H} | {b - a for cuts in cut_sets for a, b in zip(cuts[:-1], cuts[1:])}
    ws = torch.empty(max(orch_lib.unet_conv_workspace_bytes(shape, r) for r in heights), dtype=torch.uint8,
                     device=DEV)
    full = torch.empty((H, W, Co), device=DEV)
    orch_lib.unet_conv_band(shape, 0, H, xd, dev["gamma"], dev["beta"], wt, dev["bias"], act, sums,
                            1, full, ws)
    torch.cuda.synchronize()
    assert not torch.isnan(full).any()
    act0, sums0 = act.clone(), sums.clone()

    def stitch(cuts, refresh):
        out = torch.empty_like(full)
        for rb, re in zip(cuts[:-1], cuts[1:]):
            o = torch.empty((re - rb, W, Co), device=DEV)
            orch_lib.unet_conv_band(shape, rb, re, xd[rb:re].contiguous(), dev["gamma"], dev["beta"],
                                    wt, dev["bias"], act, sums, refresh, o, ws)
            out[rb:re] = o
        torch.cuda.synchronize()
        return out
    for cuts in cut_sets:
        got = stitch(cuts, 1)
        assert torch.equal(act, act0) and torch.equal(sums, sums0), cuts
        assert rel_l2(to_host(got), to_host(full)) <= 1e-6, cuts
    assert torch.equal(stitch(cut_sets[1], 0), stitch(cut_sets[1], 0))


def test_unet_rejects_bad_arguments(orch_lib):
    cfg = configs.UNET_TINY
    shape = orch_lib.unet_shape(cfg, EPS)
    t = torch.zeros(1 << 16, device=DEV)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.unet_conv_band(shape, 4, 4, t, t, t, t, t, t, t, 0, t[:100], ws)
    assert "band" in str(e.value)
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.unet_conv_band(shape, 2, 6, t, t, t, t, t, None, None, 0, t[:100], ws)
    assert "stale" in str(e.value)
    bad = orch_lib.UNetConvShape(16, 16, 96, 8, 64, EPS)
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.unet_conv_band(bad, 0, 4, t, t, t, t, t, t, t, 0, t[:100], ws)
    assert "multiple of 64" in str(e.value)
