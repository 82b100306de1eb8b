"""The patch-parallel sampler on virtual devices (Algorithm 1) against the
oracle sampler, end to end: the whole trajectory runs free on both sides.
Tolerance (relative L2 of the final latent): 1e-5 for the fp32
configuration, 2e-2 for bf16."""
import functools

import numpy as np
import pytest
import torch

from oracle import blob as oblob
from oracle import sampler as osampler
from oracle import schedule as osched
from seeded_inputs import configs, generate
from tests._gpu_util import DEV, rel_l2, to_dev, to_host

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=2)
def _model(name):
    cfg = {c.name: c for c in configs.ALL_CONFIGS}[name]
    blob = generate.make_weight_blob(cfg, 0)
    hdr, params = oblob.read_blob(blob, np.float64)
    return cfg, blob, hdr, params


def _grid(cfg, M):
    return [t for t, _ in osched.step_pairs(cfg.T, M)] + [-1]


def _run(orch_lib, cfg, blob, x0, splits, tiers, grid, warmup, labels):
    ctx = orch_lib.DiTStep(cfg, blob)
    try:
        n = ctx.stale_kv_bytes()
        kv_a = torch.empty(n, dtype=torch.uint8, device=DEV)
        kv_b = torch.empty(n, dtype=torch.uint8, device=DEV)
        lat = to_dev(x0)
        ctx.sample_patch_parallel(lat, splits, tiers, grid, warmup, labels, cfg.cfg_scale, kv_a, kv_b)
        torch.cuda.synchronize()
        return to_host(lat)
    finally:
        ctx.close()


@pytest.mark.parametrize("splits,tiers,M,warmup", [
    ([0, 3, 5, 8], [0, 1, 0], 8, 2),
    ([0, 2, 8], [1, 0], 7, 2),         # odd remainder: the last interval is one step
    ([0, 8], [0], 6, 2),                # one device on every row: the full sampler
    ([0, 1, 2, 3, 4, 5, 6, 7, 8], [0, 1, 0, 1, 0, 1, 0, 1], 6, 1),
])
def test_sampler_fp32_tiny(orch_lib, splits, tiers, M, warmup):
    cfg, blob, hdr, params = _model("tiny")
    x0 = generate.make_latent(cfg, 3)
    labels = generate.make_labels(cfg, 3)
    grid = _grid(cfg, M)
    got = _run(orch_lib, cfg, blob, x0, splits, tiers, grid, warmup, labels)
    ref = osampler.patch_parallel_sample(hdr, params, x0, splits, tiers, grid, warmup, labels,
                                         cfg.cfg_scale)
    assert rel_l2(got, ref) <= 1e-5
    if len(tiers) == 1:
        full = osampler.full_sample(hdr, params, x0, grid, labels, cfg.cfg_scale)
        assert rel_l2(got, full) <= 1e-5


def test_sampler_bf16_dit_s2(orch_lib):
    cfg, blob, hdr, params = _model("dit_s2_256")
    x0 = generate.make_latent(cfg, 4)
    labels = generate.make_labels(cfg, 4)
    grid = _grid(cfg, 10)
    splits, tiers = [0, 6, 11, 16], [0, 1, 0]
    got = _run(orch_lib, cfg, blob, x0, splits, tiers, grid, 2, labels)
    ref = osampler.patch_parallel_sample(hdr, params, x0, splits, tiers, grid, 2, labels,
                                         cfg.cfg_scale)
    assert rel_l2(got, ref) <= 2e-2


@pytest.mark.parametrize("kw,word", [
    (dict(splits=[1, 8]), "row_splits"), (dict(splits=[0, 5, 5, 8], tiers=[0, 0, 0]), "increase"),
    (dict(tiers=[2]), "tiers"), (dict(warmup=0), "warmup"), (dict(warmup=7), "warmup"),
    (dict(grid=[900, 950, -1]), "t_grid"), (dict(grid=[900, 400, 0]), "t_grid[steps]"),
])
def test_sampler_rejects_bad_arguments(orch_lib, kw, word):
    cfg, blob, _, _ = _model("tiny")
    a = dict(splits=[0, 8], tiers=[0], grid=[900, 600, 300, -1], warmup=1)
    a.update(kw)
    ctx = orch_lib.DiTStep(cfg, blob)
    try:
        n = ctx.stale_kv_bytes()
        kv_a = torch.zeros(n, dtype=torch.uint8, device=DEV)
        kv_b = torch.zeros(n, dtype=torch.uint8, device=DEV)
        lat = to_dev(generate.make_latent(cfg, 0))
        before = lat.clone()
        with pytest.raises(orch_lib.OrchError) as e:
            ctx.sample_patch_parallel(lat, a["splits"], a["tiers"], a["grid"], a["warmup"],
                                      generate.make_labels(cfg, 0), cfg.cfg_scale, kv_a, kv_b)
        assert e.value.code == orch_lib.ORCH_EINVAL and word in orch_lib.last_error()
        torch.cuda.synchronize()
        assert torch.equal(lat, before)
    finally:
        ctx.close()
