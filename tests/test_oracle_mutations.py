"""Planted mistakes in the oracle (on the CPU) must be caught by its pins.

Each case patches one plausible slip into the oracle -- a dropped term, a
wrong scale, a swapped operand -- and checks that an independent reference
no longer agrees.  Nothing here touches the GPU path.
"""
import math

import numpy as np
import pytest

from oracle import blob as oblob
from oracle import dit, schedule
from seeded_inputs import configs, generate
from tests._torch_dit import torch_dit_eps

CFG = configs.scaled(configs.TINY, name="tiny_cfg2", cfg_batch=2)


@pytest.fixture(scope="module")
def model():
    hdr, params = oblob.read_blob(generate.make_weight_blob(CFG, 0))
    x = generate.make_latent(CFG, 0).astype(np.float64)
    return hdr, params, x, generate.make_labels(CFG, 0)


def _full_eps_agrees(hdr, params, x, labels):
    got = dit.denoiser_band(hdr, params, x, 0, CFG.R, 750, labels)["eps"]
    ref = torch_dit_eps(hdr, params, x, 750, labels)
    return np.allclose(got, ref, rtol=1e-9, atol=1e-10)


MUTATIONS = {
    "gelu_constant": ("gelu_tanh", lambda x: 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.04 * x ** 3)))),
    "gelu_exact_erf_like": ("gelu_tanh", lambda x: x / (1 + np.exp(-1.702 * x))),
    "ln_unbiased_var": ("layer_norm", lambda h, eps=1e-6: (h - h.mean(-1, keepdims=True)) /
                        np.sqrt(h.var(-1, ddof=1, keepdims=True) + eps)),
    "ln_eps_1e-5": ("layer_norm", lambda h, eps=1e-6: (h - h.mean(-1, keepdims=True)) /
                    np.sqrt(h.var(-1, keepdims=True) + 1e-2)),
    "modulate_no_one": ("modulate", lambda u, shift, scale: u * scale + shift),
    "sinusoid_sin_first": ("timestep_embedding", None),
    "silu_as_sigmoid": ("silu", lambda x: 1 / (1 + np.exp(-x))),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_caught_by_torch_reference(model, monkeypatch, name):
    hdr, params, x, labels = model
    assert _full_eps_agrees(hdr, params, x, labels)
    attr, fn = MUTATIONS[name]
    orig = getattr(dit, attr)
    if fn is None:          # [sin, cos] instead of [cos, sin]
        def fn(t, dim=256, dtype=np.float64):
            return np.roll(orig(t, dim, dtype), dim // 2)
    monkeypatch.setattr(dit, attr, fn)
    assert not _full_eps_agrees(hdr, params, x, labels)


def test_mutation_attention_scale(model, monkeypatch):
    hdr, params, x, labels = model
    orig = dit.attention

    def wrong(q, k, v, heads, q_chunk=2048):
        d = q.shape[1] // heads
        return orig(q / math.sqrt(d), k, v, heads, q_chunk)
    monkeypatch.setattr(dit, "attention", wrong)
    assert not _full_eps_agrees(hdr, params, x, labels)


def test_mutation_patch_order(model, monkeypatch):
    hdr, params, x, labels = model
    orig = dit.patchify_rows

    def wrong(hdr_, xf, rb, re):                 # (dy, dx, channel) instead of (channel, dy, dx)
        v = orig(hdr_, xf, rb, re)
        C, p = hdr_["in_ch"], hdr_["patch"]
        return v.reshape(-1, C, p, p).transpose(0, 2, 3, 1).reshape(v.shape)
    monkeypatch.setattr(dit, "patchify_rows", wrong)
    assert not _full_eps_agrees(hdr, params, x, labels)


@pytest.mark.parametrize("slip", ["offset_zero", "stale_band", "fresh_v_as_k"])
def test_mutation_band_kv_caught_by_stitching(model, monkeypatch, slip):
    """Slips in where the band's fresh K/V go break the stitching invariant
    (stale buffer = the full step's own K/V => bands reproduce the full step)."""
    hdr, params, x, labels = model
    full = dit.full_step(hdr, params, x, 500, 250, labels, 1.5, keep_kv=True)
    buf = dit.full_kv_buffer(hdr, full["kv"])
    # perturb the buffer inside the band only: unused by a correct band step
    R = hdr["grid"]
    rb, re = 2, 5
    noisy = buf.copy()
    N, H = R * R, hdr["hidden"]
    per = 2 * N * H
    d = H // hdr["heads"]
    for blk in range(hdr["n_blocks"] * 2):
        for hh in range(hdr["heads"]):
            s0 = blk * per + hh * N * d
            noisy[s0 + rb * R * d:s0 + re * R * d] += 0.5
    good = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, noisy)
    np.testing.assert_allclose(good["x_out"], full["x_out"][:, rb * 2:re * 2], rtol=1e-12, atol=1e-12)
    orig = dit.assemble_kv

    def wrong(stale, k, v, tok0):
        if slip == "offset_zero":
            return orig(stale, k, v, 0)
        if slip == "stale_band":
            return stale[0].copy(), stale[1].copy()
        return orig(stale, v, v, tok0)
    monkeypatch.setattr(dit, "assemble_kv", wrong)
    bad = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, noisy)
    assert not np.allclose(bad["x_out"], full["x_out"][:, rb * 2:re * 2], rtol=1e-6, atol=1e-8)


def test_mutation_scheduler_sign(monkeypatch):
    """A sign slip in Bc breaks the forward-marginal invariant."""
    ab = schedule.alpha_bar()
    a_s, s_s = schedule.alpha_sigma(ab, 780)
    a_p, s_p = schedule.alpha_sigma(ab, 760)
    A, Bc, C = schedule.ddim_coefficients(ab, 780, 760)
    x0, eps = 0.3, -1.25
    x = a_s * x0 + s_s * eps
    good = A * x - Bc * eps
    bad = A * x + Bc * eps
    assert abs(good - (a_p * x0 + s_p * eps)) < 1e-12
    assert abs(bad - (a_p * x0 + s_p * eps)) > 1e-3


def test_mutation_guidance_branch_swap(model, monkeypatch):
    """eps_c + g (eps_u - eps_c) (branches swapped) breaks the single-branch pin."""
    from tests.test_oracle_dit import _branch_order_holds
    hdr, params, x, labels = model
    assert _branch_order_holds(hdr, params, x, labels)

    def swapped(eps, cfg_scale):
        if eps.shape[0] == 1:
            return eps[0]
        return eps[0] + cfg_scale * (eps[1] - eps[0])
    monkeypatch.setattr(dit, "guided_eps", swapped)
    assert not _branch_order_holds(hdr, params, x, labels)


# ---- U-Net band block -------------------------------------------------------

def _unet_pins_hold():
    """The torch pin (full map) and the stitching pin (bands with the full
    map's own buffers) of the U-Net band block."""
    from oracle import unet
    from oracle.blob import bf16_to_float
    from tests.test_oracle_unet import _torch_block
    cfg = configs.UNET_TINY
    pr = generate.make_unet_params(cfg, 0)
    params = {"gamma": pr["gamma"].astype(np.float64), "beta": pr["beta"].astype(np.float64),
              "weight": bf16_to_float(pr["weight_bits"]).astype(np.float64),
              "bias": pr["bias"].astype(np.float64)}
    x = generate.make_unet_input(cfg, 0).astype(np.float64)
    full = unet.full_step(params, x, cfg.groups)
    ok = np.allclose(full["out"], _torch_block(params, x, cfg.groups)[0], rtol=1e-10, atol=1e-10)
    sums = unet.row_group_sums(x, cfg.groups)
    for rb, re in ((0, 5), (5, 11), (11, 16)):
        got = unet.band_step(params, x[rb:re], cfg.height, rb, re, cfg.groups, full["act"], sums)
        ok &= bool(np.allclose(got["out"], full["out"][rb:re], rtol=1e-10, atol=1e-10))
    return bool(ok)


def test_unet_mutation_halo_off_by_one(monkeypatch):
    from oracle import unet
    assert _unet_pins_hold()
    orig = unet.band_step

    def wrong(params, x_band, H, rb, re, groups, stale_act=None, stale_sums=None, eps=unet.GN_EPS):
        if stale_act is not None:                 # halo taken one row too far out
            stale_act = np.concatenate([stale_act[1:], stale_act[-1:]])
        return orig(params, x_band, H, rb, re, groups, stale_act, stale_sums, eps)
    monkeypatch.setattr(unet, "band_step", wrong)
    assert not _unet_pins_hold()


@pytest.mark.parametrize("slip", ["band_only_stats", "unbiased_var", "wrapped_columns",
                                  "no_silu"])
def test_unet_mutations(monkeypatch, slip):
    from oracle import unet
    assert _unet_pins_hold()
    if slip == "band_only_stats":
        orig = unet.group_stats

        def wrong(sums, W, C, eps=unet.GN_EPS):
            s = np.asarray(sums)
            keep = ~np.isclose(s, 0).all(axis=(1, 2))
            return orig(s[keep][:max(1, len(s) // 3)], W, C, eps)
        monkeypatch.setattr(unet, "group_stats", wrong)
    elif slip == "unbiased_var":
        orig = unet.group_stats

        def wrong(sums, W, C, eps=unet.GN_EPS):
            s = np.asarray(sums, dtype=np.float64)
            n = s.shape[0] * W * (C // s.shape[1])
            mean, rstd = orig(sums, W, C, eps)
            var = (1 / rstd ** 2 - eps) * n / (n - 1)
            return mean, 1 / np.sqrt(var + eps)
        monkeypatch.setattr(unet, "group_stats", wrong)
    elif slip == "wrapped_columns":
        def wrong(act_rows, weight, bias):
            a = np.asarray(act_rows, dtype=np.float64)
            r = a.shape[0] - 2
            out = np.zeros((r, a.shape[1], weight.shape[0])) + bias
            for dy in range(3):
                for dx in range(3):
                    win = np.roll(a[dy:dy + r], 1 - dx, axis=1)
                    out += win @ weight[:, dy, dx, :].T
            return out
        monkeypatch.setattr(unet, "conv3x3_rows", wrong)
    else:
        monkeypatch.setattr(unet, "silu", lambda v: v)           # GroupNorm output as is
    assert not _unet_pins_hold()


# ---- patch-parallel sampler (Algorithm 1 on virtual devices) -----------------

def _sampler_pins_hold():
    from oracle import sampler
    from oracle import schedule as osched
    cfg = configs.TINY
    hdr, params = oblob.read_blob(generate.make_weight_blob(cfg, 0))
    x, lab = generate.make_latent(cfg, 1), generate.make_labels(cfg, 1)
    g = [t for t, _ in osched.step_pairs(cfg.T, 7)] + [-1]
    splits = [0, 3, 5, cfg.R]
    ok = True
    for tiers in ([0, 0, 1], [1, 0, 0]):
        a = sampler.patch_parallel_sample(hdr, params, x, splits, tiers, g, 2, lab, 1.5)
        b = sampler.patch_parallel_sample(hdr, params, x, splits, tiers, g, 2, lab, 1.5, order=[2, 0, 1])
        ok &= bool(np.array_equal(a, b))
    g6 = [t for t, _ in osched.step_pairs(cfg.T, 6)] + [-1]
    one = sampler.patch_parallel_sample(hdr, params, x, [0, cfg.R], [0], g6, 2, lab, 1.5)
    ok &= bool(np.array_equal(one, sampler.full_sample(hdr, params, x, g6, lab, 1.5)))
    return ok


@pytest.mark.parametrize("slip", ["second_half_reads_exchanged", "second_half_from_interval_start",
                                  "reduced_tier_reads_exchanged"])
def test_sampler_mutations(monkeypatch, slip):
    """Plausible slips in which buffer or latent a half-step reads break the
    device-order invariance or the one-device reduction to the full sampler.
    In the sampler, a band step that keeps its K/V is one whose K/V are
    exchanged (a tier-0 first half-step or a tier-1 double step); the tier-0
    second half-step keeps nothing."""
    from oracle import sampler  # noqa: F401  (the pins run it)
    assert _sampler_pins_hold()
    orig_step, orig_refreshed = dit.patch_step, dit.refreshed_buffer
    interval = 1000 // 7                            # grid spacing of the pins' 7-step grid
    state = {}

    def refreshed(hdr, stale, kv, rb, re, dtype=np.float64):
        state["exchanged"] = orig_refreshed(hdr, stale, kv, rb, re, dtype)   # the next buffer so far
        return state["exchanged"]

    def step(hdr, params, x_full, rb, re, t, tp, labels, g, stale_kv=None, **kw):
        exchanges = kw.get("keep_kv", False)
        double = tp == -1 or t - tp > 1.5 * interval
        if stale_kv is not None and "exchanged" in state:
            if slip == "second_half_reads_exchanged" and not exchanges:
                stale_kv = state["exchanged"]
            if slip == "reduced_tier_reads_exchanged" and exchanges and double:
                stale_kv = state["exchanged"]
        if slip == "second_half_from_interval_start" and not exchanges and stale_kv is not None:
            x_full = state.get("x_first_half", x_full)
        if exchanges:
            state["x_first_half"] = x_full
        return orig_step(hdr, params, x_full, rb, re, t, tp, labels, g, stale_kv, **kw)

    monkeypatch.setattr(dit, "refreshed_buffer", refreshed)
    monkeypatch.setattr(dit, "patch_step", step)
    assert not _sampler_pins_hold()
