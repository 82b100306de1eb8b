"""Step-level parity of orch_patch_denoise_step against the oracle, and the
invariants of the band step on the GPU (all-rows band, stitching of bands
with fresh K/V, buffer refresh semantics).

Parity is per step and teacher-forced: the same x, t, labels and stale
buffer go to both sides.  Tolerance (relative L2 over the whole tensor):
1e-5 for the fp32 configuration, 2e-2 for bf16, on the eps of every
guidance branch and on the updated band of x.
"""
import functools

import numpy as np
import pytest
import torch

from oracle import blob as oblob
from oracle import dit
from seeded_inputs import configs, generate
from tests._gpu_util import DEV, bits_to_dev, empty, rel_l2, to_dev, to_host

pytestmark = pytest.mark.gpu

TINY2 = configs.scaled(configs.TINY, name="tiny_cfg2", cfg_batch=2)


@functools.lru_cache(maxsize=2)
def _model(name, dtype_oracle="f64"):
    cfg = {c.name: c for c in configs.ALL_CONFIGS + (TINY2,)}[name]
    blob = generate.make_weight_blob(cfg, 0)
    hdr, params = oblob.read_blob(blob, np.float64 if dtype_oracle == "f64" else np.float32)
    return cfg, blob, hdr, params


_CTX = {}


def _ctx(orch_lib, cfg, blob):
    if cfg.name not in _CTX:
        for k in list(_CTX):
            _CTX.pop(k).close()
        _CTX[cfg.name] = orch_lib.DiTStep(cfg, blob)
    return _CTX[cfg.name]


def _run_gpu(orch_lib, cfg, blob, x, rb, re, t, tp, labels, stale, refresh, z=None, eta=0.0):
    ctx = _ctx(orch_lib, cfg, blob)
    p = cfg.patch
    xd = to_dev(x)
    kv = bits_to_dev(stale)
    eps = empty((cfg.cfg_batch, cfg.out_ch, (re - rb) * p, cfg.latent))
    out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
    ctx.step(xd, rb, re, t, tp, labels, cfg.cfg_scale, kv, refresh, out, eps,
             None if z is None else to_dev(z), eta)
    return to_host(eps), to_host(out), kv


def _check(cfg, got_eps, got_x, ref, tol):
    for b in range(cfg.cfg_batch):
        e = rel_l2(got_eps[b], ref["eps"][b])
        assert e <= tol, (b, e)
    e = rel_l2(got_x, ref["x_out"])
    assert e <= tol, e


# ---- fp32: tiny DiT, tolerance 1e-5 ---------------------------------------

@pytest.mark.parametrize("name,rb,re,t,tp,refresh,eta", [
    ("tiny", 0, 4, 750, 500, 0, 0.0),
    ("tiny", 0, 4, 0, -1, 1, 0.0),
    ("tiny_cfg2", 2, 6, 500, 250, 1, 0.0),
    ("tiny_cfg2", 5, 8, 250, 0, 0, 0.7),
    ("tiny_cfg2", 0, 8, 999, 500, 1, 0.0),
])
def test_step_fp32_tiny(orch_lib, name, rb, re, t, tp, refresh, eta):
    cfg, blob, hdr, params = _model(name)
    x = generate.make_latent(cfg, 0)
    z = generate.make_noise(cfg, 0) if eta > 0 else None
    labels = generate.make_labels(cfg, 0)
    stale = generate.make_stale_kv(cfg, 0)
    eps, xo, kv = _run_gpu(orch_lib, cfg, blob, x, rb, re, t, tp, labels, stale, refresh, z, eta)
    ref = dit.patch_step(hdr, params, x, rb, re, t, tp, labels, cfg.cfg_scale, stale, eta=eta,
                         z=z, keep_kv=bool(refresh))
    _check(cfg, eps, xo, ref, 1e-5)
    kvh = to_host(kv)
    if refresh:
        want = dit.refreshed_buffer(hdr, stale, ref["kv"], rb, re)
        assert rel_l2(kvh, want) <= 1e-5
        # tokens outside the band are bitwise unchanged
        R, N, H = cfg.R, cfg.n_kv, cfg.hidden
        for l in range(cfg.n_blocks):
            for b in range(cfg.cfg_batch):
                K1, V1 = dit.stale_kv_block(hdr, kvh, cfg.cfg_batch, l, b)
                K0, V0 = dit.stale_kv_block(hdr, stale, cfg.cfg_batch, l, b)
                band = slice(rb * R, re * R)
                np.testing.assert_array_equal(np.delete(K1, band, 0), np.delete(K0, band, 0))
                np.testing.assert_array_equal(np.delete(V1, band, 0), np.delete(V0, band, 0))
    else:
        np.testing.assert_array_equal(kvh, stale.astype(np.float64))


def test_trajectory_fp32_tiny(orch_lib):
    """Four free-running full-image DDIM steps (the tiny config's sampler)."""
    cfg, blob, hdr, params = _model("tiny")
    x_gpu = generate.make_latent(cfg, 0)
    x_ref = x_gpu.astype(np.float64)
    labels = generate.make_labels(cfg, 0)
    stale = generate.make_stale_kv(cfg, 0)
    from oracle import schedule as osched
    for t, tp in osched.step_pairs(cfg.T, cfg.steps):
        _, xo, _ = _run_gpu(orch_lib, cfg, blob, x_gpu, 0, cfg.R, t, tp, labels, stale, 1)
        x_gpu = xo.astype(np.float32)
        x_ref = dit.full_step(hdr, params, x_ref, t, tp, labels, cfg.cfg_scale)["x_out"]
    assert rel_l2(x_gpu, x_ref) <= 1e-5


# ---- bf16 configs, tolerance 2e-2 ------------------------------------------

@pytest.mark.parametrize("rb,re,refresh", [(0, 6, 1), (5, 11, 0), (10, 16, 1)])
def test_step_bf16_dit_s2(orch_lib, rb, re, refresh):
    cfg, blob, hdr, params = _model("dit_s2_256")
    x = generate.make_latent(cfg, 0)
    labels = generate.make_labels(cfg, 0)
    stale = generate.make_stale_kv(cfg, 0)
    t, tp = 500, 450
    eps, xo, kv = _run_gpu(orch_lib, cfg, blob, x, rb, re, t, tp, labels, stale, refresh)
    ref = dit.patch_step(hdr, params, x, rb, re, t, tp, labels, cfg.cfg_scale, stale,
                         keep_kv=bool(refresh))
    _check(cfg, eps, xo, ref, 2e-2)
    if refresh:
        want = dit.refreshed_buffer(hdr, stale, ref["kv"], rb, re)
        assert rel_l2(to_host(kv), want) <= 2e-2


def test_trajectory_bf16_dit_s2(orch_lib):
    """The S/2 sampler's 20 steps on a 6-row band with a refreshed buffer,
    free running on both sides; checked at steps 1, 10 and 20."""
    cfg, blob, hdr, params = _model("dit_s2_256")
    from oracle import schedule as osched
    x0 = generate.make_latent(cfg, 0)
    labels = generate.make_labels(cfg, 0)
    stale = generate.make_stale_kv(cfg, 0)
    rb, re = 0, cfg.band_rows[0]
    p = cfg.patch
    ctx = _ctx(orch_lib, cfg, blob)
    xg = to_dev(x0)
    kv = bits_to_dev(stale)
    out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
    x_ref = x0.astype(np.float64)
    buf_ref = stale
    for m, (t, tp) in enumerate(osched.step_pairs(cfg.T, cfg.steps)):
        ctx.step(xg, rb, re, t, tp, labels, cfg.cfg_scale, kv, 1, out)
        xg[:, rb * p:re * p] = out
        r = dit.patch_step(hdr, params, x_ref, rb, re, t, tp, labels, cfg.cfg_scale, buf_ref,
                           keep_kv=True)
        buf_ref = dit.refreshed_buffer(hdr, buf_ref, r["kv"], rb, re)
        x_ref = x_ref.copy()
        x_ref[:, rb * p:re * p] = r["x_out"]
        if m in (0, 9, 19):
            e = rel_l2(to_host(xg)[:, rb * p:re * p], x_ref[:, rb * p:re * p])
            assert e <= 2e-2, (m, e)


@pytest.mark.parametrize("name,rows_idx,t,tp", [
    ("dit_xl2_512", 0, 780, 760),
    ("dit_xl2_512", 0, 20, -1),
    ("dit_xl2_1024", 0, 780, 760),
])
def test_step_bf16_xl(orch_lib, name, rows_idx, t, tp):
    big = name == "dit_xl2_1024"
    cfg, blob, hdr, params = _model(name, "f32" if big else "f64")
    x = generate.make_latent(cfg, 0)
    labels = generate.make_labels(cfg, 0)
    stale = generate.make_stale_kv(cfg, 0)
    r = cfg.band_rows[rows_idx]
    rb, re = (cfg.R - r) // 2, (cfg.R - r) // 2 + r       # an interior band
    eps, xo, kv = _run_gpu(orch_lib, cfg, blob, x, rb, re, t, tp, labels, stale, 0)
    ref = dit.patch_step(hdr, params, x, rb, re, t, tp, labels, cfg.cfg_scale, stale,
                         dtype=np.float32 if big else np.float64)
    _check(cfg, eps, xo, ref, 2e-2)


# ---- invariants at the full DiT-XL/2 1024px shape ----------------------------

def test_xl1024_all_rows_ignores_stale_and_stitching(orch_lib):
    cfg, blob, _, _ = _model("dit_xl2_1024", "f32")
    ctx = _ctx(orch_lib, cfg, blob)
    x = to_dev(generate.make_latent(cfg, 0))
    labels = generate.make_labels(cfg, 0)
    p, R = cfg.patch, cfg.R
    n_el = ctx.stale_kv_bytes() // 2
    t, tp = 780, 760
    # all rows: the buffer is never read (NaN-filled buffer gives the same result)
    kv_a = torch.full((n_el,), float("nan"), dtype=torch.bfloat16, device=DEV)
    kv_b = bits_to_dev(generate.make_stale_kv(cfg, 0))
    full_a = empty((cfg.in_ch, R * p, cfg.latent))
    full_b = empty((cfg.in_ch, R * p, cfg.latent))
    ctx.step(x, 0, R, t, tp, labels, cfg.cfg_scale, kv_a, 1, full_a)
    ctx.step(x, 0, R, t, tp, labels, cfg.cfg_scale, kv_b, 1, full_b)
    fa, fb = to_host(full_a), to_host(full_b)
    assert np.isfinite(fa).all()
    np.testing.assert_array_equal(fa, fb)
    # kv_a now holds this step's own K/V: bands with refresh off stitch to the full step
    assert not torch.isnan(kv_a).any()
    stitched = np.zeros_like(fa)
    for rb, re in [(0, 26), (26, 42), (42, 64)]:
        out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
        before = kv_a.clone()
        ctx.step(x, rb, re, t, tp, labels, cfg.cfg_scale, kv_a, 0, out)
        stitched[:, rb * p:re * p] = to_host(out)
        assert torch.equal(before, kv_a)                    # refresh off: buffer untouched
    # Equal up to rounding: a band's attention may cut its query tiles
    # between workgroups and its GEMMs may split K (short bands do), which
    # changes the summation order of the bf16 path.
    assert rel_l2(stitched, fa) <= 2e-3, rel_l2(stitched, fa)
    # With the work split off every output's summation order is fixed by its
    # token (GEMM tiles of every shape add k in the same order; attention
    # tiles are whole): stitched bands equal the all-rows step bit for bit.
    ctx.set_work_split(False)
    try:
        full_c = empty((cfg.in_ch, R * p, cfg.latent))
        ctx.step(x, 0, R, t, tp, labels, cfg.cfg_scale, kv_a, 1, full_c)
        stitched_c = np.zeros_like(fa)
        for rb, re in [(0, 6), (6, 26), (26, 42), (42, 64)]:
            out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
            ctx.step(x, rb, re, t, tp, labels, cfg.cfg_scale, kv_a, 0, out)
            stitched_c[:, rb * p:re * p] = to_host(out)
    finally:
        ctx.set_work_split(True)
    fc = to_host(full_c)
    np.testing.assert_array_equal(stitched_c, fc)
    assert rel_l2(fc, fa) <= 2e-3


def test_xl1024_refresh_matches_no_refresh(orch_lib):
    cfg, blob, _, _ = _model("dit_xl2_1024", "f32")
    ctx = _ctx(orch_lib, cfg, blob)
    x = to_dev(generate.make_latent(cfg, 1))
    labels = generate.make_labels(cfg, 1)
    stale = generate.make_stale_kv(cfg, 1)
    p, R = cfg.patch, cfg.R
    rb, re = 19, 45                                          # a 26-row (40%) interior band
    outs, kvs = [], []
    for refresh in (0, 1):
        kv = bits_to_dev(stale)
        out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
        ctx.step(x, rb, re, 780, 760, labels, cfg.cfg_scale, kv, refresh, out)
        outs.append(to_host(out))
        kvs.append(kv)
    np.testing.assert_array_equal(outs[0], outs[1])
    # non-band tokens of every block / branch are bitwise unchanged by the refresh
    N, H, B, L = cfg.n_kv, cfg.hidden, cfg.cfg_batch, cfg.n_blocks
    d, heads = cfg.head_dim, cfg.heads
    k1 = kvs[1].view(L, B, 2, N * H)
    k0 = kvs[0].view(L, B, 2, N * H)
    K1 = k1[:, :, 0].reshape(L, B, heads, N, d)
    K0 = k0[:, :, 0].reshape(L, B, heads, N, d)
    V1 = k1[:, :, 1].reshape(L, B, heads, d, N)
    V0 = k0[:, :, 1].reshape(L, B, heads, d, N)
    t0, t1 = rb * R, re * R
    assert torch.equal(K1[:, :, :, :t0], K0[:, :, :, :t0])
    assert torch.equal(K1[:, :, :, t1:], K0[:, :, :, t1:])
    assert torch.equal(V1[..., :t0], V0[..., :t0])
    assert torch.equal(V1[..., t1:], V0[..., t1:])
    assert not torch.equal(K1[:, :, :, t0:t1], K0[:, :, :, t0:t1])


# ---- the reduced-tier schedule (Algorithm 1 slow branch, Eq. (2)) ----------

def test_tiered_trajectory_fp32_tiny(orch_lib):
    """30 executed steps of the 50-step grid with a 10-step warm-up (steps of
    two intervals after it), one device's band with its buffer refreshed on
    executed steps only, against the oracle running the same schedule."""
    from oracle import schedule as osched
    from paper_2509_04719_amd import schedule as psched
    cfg, blob, hdr, params = _model("tiny")
    steps = psched.tiered_schedule(cfg.T, 50, 10)
    assert [(s.m, s.t, s.t_prev, s.refresh) for s in steps] == osched.tiered_schedule(cfg.T, 50, 10)
    x0 = generate.make_latent(cfg, 2)
    labels = generate.make_labels(cfg, 2)
    stale = generate.make_stale_kv(cfg, 2)
    rb, re = 2, 6
    p = cfg.patch
    ctx = _ctx(orch_lib, cfg, blob)
    xg = to_dev(x0)
    kv = bits_to_dev(stale)
    out = empty((cfg.in_ch, (re - rb) * p, cfg.latent))
    x_ref = x0.astype(np.float64)
    buf_ref = stale.astype(np.float64)
    for st in steps:
        ctx.step(xg, rb, re, st.t, st.t_prev, labels, cfg.cfg_scale, kv, int(st.refresh), out)
        xg[:, rb * p:re * p] = out
        r = dit.patch_step(hdr, params, x_ref, rb, re, st.t, st.t_prev, labels, cfg.cfg_scale,
                           buf_ref, keep_kv=True)
        if st.refresh:
            buf_ref = dit.refreshed_buffer(hdr, buf_ref, r["kv"], rb, re)
        x_ref = x_ref.copy()
        x_ref[:, rb * p:re * p] = r["x_out"]
    assert rel_l2(to_host(xg), x_ref) <= 1e-5
    assert rel_l2(to_host(kv), buf_ref) <= 1e-5
