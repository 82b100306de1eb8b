"""Pins of the patch-parallel sampler oracle (Algorithm 1 on virtual devices):
cases that reduce to the plain full-image DDIM sampler, and the O(1/M)
behaviour of the stale-activation error (Theorems 1 and 2)."""
import numpy as np
import pytest

from oracle import blob as oblob, dit, sampler, schedule as osched
from seeded_inputs import configs, generate

CFG = configs.TINY


@pytest.fixture(scope="module")
def model():
    hdr, params = oblob.read_blob(generate.make_weight_blob(CFG, 0))
    return hdr, params


def _grid(M):
    return [t for t, _ in osched.step_pairs(CFG.T, M)] + [-1]


def _inputs():
    return generate.make_latent(CFG, 1), generate.make_labels(CFG, 1)


def test_one_device_every_step_is_the_full_sampler(model):
    hdr, params = model
    x, lab = _inputs()
    g = _grid(6)
    got = sampler.patch_parallel_sample(hdr, params, x, [0, CFG.R], [0], g, 2, lab, CFG.cfg_scale)
    want = sampler.full_sample(hdr, params, x, g, lab, CFG.cfg_scale)
    assert np.array_equal(got, want)


def test_one_device_reduced_tier_is_the_tiered_full_sampler(model):
    """A lone tier-1 device runs the tiered schedule of the whole image."""
    hdr, params = model
    x, lab = _inputs()
    M, w = 9, 3
    g = _grid(M)
    got = sampler.patch_parallel_sample(hdr, params, x, [0, CFG.R], [1], g, w, lab, CFG.cfg_scale)
    pairs = [(t, tp) for _, t, tp, _ in osched.tiered_schedule(CFG.T, M, w)]
    want = sampler.full_sample(hdr, params, x, [t for t, _ in pairs] + [-1], lab, CFG.cfg_scale)
    assert np.array_equal(got, want)


def test_all_warmup_is_the_full_sampler(model):
    hdr, params = model
    x, lab = _inputs()
    g = _grid(4)
    got = sampler.patch_parallel_sample(hdr, params, x, [0, 3, CFG.R], [0, 1], g, 4, lab,
                                        CFG.cfg_scale)
    assert np.array_equal(got, sampler.full_sample(hdr, params, x, g, lab, CFG.cfg_scale))


@pytest.mark.parametrize("tiers", [[0, 0, 0], [0, 1, 0]])
def test_error_to_full_sampler_is_order_one_over_M(model, tiers):
    """Theorems 1/2: with the warm-up a fixed fraction of the grid, the gap
    between the patch-parallel and the full-image sample halves when M
    doubles (stale activations alone, and with a reduced-tier device)."""
    hdr, params = model
    x, lab = _inputs()
    errs = []
    for M in (8, 16, 32):
        g = _grid(M)
        pp = sampler.patch_parallel_sample(hdr, params, x, [0, 3, 5, CFG.R], tiers, g, M // 4,
                                           lab, CFG.cfg_scale)
        full = sampler.full_sample(hdr, params, x, g, lab, CFG.cfg_scale)
        errs.append(dit.rel_l2(pp, full))
    assert errs[0] > 0
    for e1, e2 in zip(errs, errs[1:]):
        assert 0.35 < e2 / e1 < 0.65, errs


@pytest.mark.parametrize("tiers", [[0, 0, 1], [1, 0, 0]])
def test_device_order_does_not_matter(model, tiers):
    """Algorithm 1's devices run in parallel: visiting them in another order
    within an interval gives the same latent bit for bit."""
    hdr, params = model
    x, lab = _inputs()
    g = _grid(7)
    splits = [0, 3, 5, CFG.R]
    a = sampler.patch_parallel_sample(hdr, params, x, splits, tiers, g, 2, lab, CFG.cfg_scale)
    b = sampler.patch_parallel_sample(hdr, params, x, splits, tiers, g, 2, lab, CFG.cfg_scale,
                                      order=[2, 0, 1])
    assert np.array_equal(a, b)
