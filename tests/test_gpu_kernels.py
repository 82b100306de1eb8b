"""Kernel-level parity of the HIP path against the oracle, through the C ABI.

Each kernel runs on seeded inputs at shapes that span several tiles with a
ragged tail, and at the full DiT-XL/2 1024px (40% band) shape in the launch
configuration of the step, where the oracle checks sampled rows.
"""
import numpy as np
import pytest
import torch

from oracle import blob as oblob
from oracle import dit, schedule as osched
from seeded_inputs import configs, generate
from tests._gpu_util import (DEV, bits_to_dev, code, empty, rel_l2, rounded, to_dev, to_host)

pytestmark = pytest.mark.gpu

XL = configs.DIT_XL2_1024
XL_M = XL.cfg_batch * XL.n_q(26)      # 3328 rows: the 40% band, both branches


# ---- adaLN LayerNorm ------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,H,rpb", [(1, 128, 1), (97, 384, 50), (3328, 1152, 1664)])
def test_layernorm_modulate(orch_lib, dtype, rows, H, rpb):
    rng = np.random.default_rng(rows + H)
    x = rng.standard_normal((rows, H)) * 2.0 + 0.5
    B = (rows + rpb - 1) // rpb
    mod = rng.standard_normal((B, 3 * H)) * 0.1
    shift, scale = mod[:, H:2 * H], mod[:, 2 * H:]
    xd, md = to_dev(x), to_dev(mod)
    out = empty((rows, H), dtype)
    orch_lib.layernorm_modulate(xd, rows, H, rpb, md[:, H:], md[:, 2 * H:], 3 * H, out, code(dtype))
    xr, mr = rounded(x, "f32"), rounded(mod, "f32")
    b = np.arange(rows) // rpb
    ref = dit.modulate(dit.layer_norm(xr), mr[b, H:2 * H], mr[b, 2 * H:])
    err = rel_l2(to_host(out), ref)
    assert err <= (1e-6 if dtype == "f32" else 4e-3), err


# ---- projection GEMMs -------------------------------------------------------

GEMM_SHAPES = [(1, 128, 128), (96, 384, 1152), (200, 1536, 384), (333, 1152, 3456)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,K,N", GEMM_SHAPES)
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_linear(orch_lib, dtype, M, K, N, epi):
    rng = np.random.default_rng(M * 7 + K + N + epi)
    A = rng.standard_normal((M, K))
    W = rng.standard_normal((N, K)) * 0.02
    bias = rng.standard_normal(N) * 0.02
    Ar, Wr, br = rounded(A, dtype), rounded(W, dtype), rounded(bias, "f32")
    y = dit.linear(Ar, Wr, br)
    Ad, Wd, bd = to_dev(A, dtype), to_dev(W, dtype), to_dev(bias)
    if epi == 2:
        rpb = max(1, M // 2)
        nb = (M + rpb - 1) // rpb
        gate = rng.standard_normal((nb, N + 16)) * 0.5
        h0 = rng.standard_normal((M, N))
        gd, out = to_dev(gate), to_dev(h0)
        orch_lib.linear(Ad, M, K, Wd, N, bd, 2, gd, N + 16, rpb, out, code(dtype))
        g = rounded(gate, "f32")[np.arange(M) // rpb, :N]
        got = to_host(out) - rounded(h0, "f32")
        err = rel_l2(got, g * y)
        assert err <= 2e-5, err
    else:
        out = empty((M, N), dtype)
        orch_lib.linear(Ad, M, K, Wd, N, bd, epi, None, 0, 1, out, code(dtype))
        ref = dit.gelu_tanh(y) if epi == 1 else y
        err = rel_l2(to_host(out), ref)
        assert err <= (1e-5 if dtype == "f32" else 5e-3), err


@pytest.mark.parametrize("K,N,epi", [(1152, 3456, 0), (1152, 1152, 2), (1152, 4608, 1), (4608, 1152, 2)])
def test_linear_full_xl_shape_sampled(orch_lib, K, N, epi):
    """The four projections of DiT-XL/2 at the 40% band (M = 3328), sampled rows."""
    M = XL_M
    rng = np.random.default_rng(K + N)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    bias = (rng.standard_normal(N) * 0.02).astype(np.float32)
    Ad, Wd, bd = to_dev(A, "bf16"), to_dev(W, "bf16"), to_dev(bias)
    rows = np.sort(rng.choice(M, 48, replace=False))
    rows[-1] = M - 1
    Ar, Wr = rounded(A[rows], "bf16"), rounded(W, "bf16")
    y = dit.linear(Ar, Wr, bias.astype(np.float64))
    if epi == 2:
        gate = (rng.standard_normal((2, N)) * 0.5).astype(np.float32)
        h0 = np.zeros((M, N), np.float32)
        out = to_dev(h0)
        orch_lib.linear(Ad, M, K, Wd, N, bd, 2, to_dev(gate), N, M // 2, out, 1)
        ref = gate.astype(np.float64)[rows // (M // 2)] * y
        err = rel_l2(to_host(out)[rows], ref)
        assert err <= 2e-5, err
    else:
        out = empty((M, N), "bf16")
        orch_lib.linear(Ad, M, K, Wd, N, bd, epi, None, 0, 1, out, 1)
        ref = dit.gelu_tanh(y) if epi == 1 else y
        err = rel_l2(to_host(out)[rows], ref)
        assert err <= 5e-3, err


# ---- QKV projection with the buffer scatter ---------------------------------

@pytest.mark.parametrize("dtype,H,heads,n_tok,kv_tokens,off", [
    ("f32", 128, 4, 32, 64, 16), ("bf16", 384, 6, 96, 256, 96), ("bf16", 1152, 16, 384, 1024, 640)])
def test_qkv_scatter(orch_lib, dtype, H, heads, n_tok, kv_tokens, off):
    B = 2
    d = H // heads
    rng = np.random.default_rng(H)
    A = rng.standard_normal((B * n_tok, H))
    W = rng.standard_normal((3 * H, H)) * 0.02
    bias = rng.standard_normal(3 * H) * 0.02
    y = dit.linear(rounded(A, dtype), rounded(W, dtype), rounded(bias, "f32"))
    stride = 2 * kv_tokens * H + 64
    canary = rng.standard_normal(B * stride)
    kv = to_dev(canary, dtype)
    q = empty((B, heads, n_tok, d), dtype)
    orch_lib.qkv_projection(to_dev(A, dtype), B, n_tok, H, to_dev(W, dtype), to_dev(bias), H, heads,
                            q, kv, stride, kv_tokens, off, code(dtype))
    tol = 1e-5 if dtype == "f32" else 5e-3
    qh = to_host(q)
    kvh = to_host(kv).reshape(B, stride)
    can = rounded(canary, dtype).reshape(B, stride)
    hdr = {"hidden": H, "heads": heads, "grid": int(np.sqrt(kv_tokens))}
    for b in range(B):
        yb = y[b * n_tok:(b + 1) * n_tok]
        qref = yb[:, :H].reshape(n_tok, heads, d).transpose(1, 0, 2)
        assert rel_l2(qh[b], qref) <= tol
        K, V = dit.stale_kv_block(hdr, kvh[b, :2 * kv_tokens * H], 1, 0, 0)
        K0, V0 = dit.stale_kv_block(hdr, can[b, :2 * kv_tokens * H], 1, 0, 0)
        band = slice(off, off + n_tok)
        assert rel_l2(K[band], yb[:, H:2 * H]) <= tol
        assert rel_l2(V[band], yb[:, 2 * H:]) <= tol
        # every other token, and the tail past the buffer, is untouched
        np.testing.assert_array_equal(np.delete(K, band, 0), np.delete(K0, band, 0))
        np.testing.assert_array_equal(np.delete(V, band, 0), np.delete(V0, band, 0))
        np.testing.assert_array_equal(kvh[b, 2 * kv_tokens * H:], can[b, 2 * kv_tokens * H:])


# ---- k-split of short GEMMs ---------------------------------------------------

@pytest.mark.parametrize("M,K,N", [(333, 4608, 768), (768, 4608, 1152), (200, 1152, 384)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_linear_split_k(orch_lib, M, K, N, epi):
    """Few output tiles: with a workspace the GEMM splits K (fp32 partials,
    then a reduction applying the epilogue); checked against the oracle and
    against the unsplit launch."""
    wsb = orch_lib.linear_workspace_bytes(M, N, K, 1)
    assert wsb > 0
    rng = np.random.default_rng(M + K + N + epi)
    A = rng.standard_normal((M, K))
    W = rng.standard_normal((N, K)) * 0.02
    bias = rng.standard_normal(N) * 0.02
    y = dit.linear(rounded(A, "bf16"), rounded(W, "bf16"), rounded(bias, "f32"))
    Ad, Wd, bd = to_dev(A, "bf16"), to_dev(W, "bf16"), to_dev(bias)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    if epi == 2:
        rpb = max(1, M // 2)
        gate = rng.standard_normal(((M + rpb - 1) // rpb, N)) * 0.5
        h0 = rng.standard_normal((M, N))
        gd = to_dev(gate)
        outs = []
        for w in (ws, None):
            out = to_dev(h0)
            orch_lib.linear(Ad, M, K, Wd, N, bd, 2, gd, N, rpb, out, 1, workspace=w)
            outs.append(to_host(out) - rounded(h0, "f32"))
        g = rounded(gate, "f32")[np.arange(M) // rpb]
        assert rel_l2(outs[0], g * y) <= 2e-5
        assert rel_l2(outs[0], outs[1]) <= 2e-5
    else:
        outs = []
        for w in (ws, None):
            out = empty((M, N), "bf16")
            orch_lib.linear(Ad, M, K, Wd, N, bd, epi, None, 0, 1, out, 1, workspace=w)
            outs.append(to_host(out))
        ref = dit.gelu_tanh(y) if epi == 1 else y
        assert rel_l2(outs[0], ref) <= 5e-3
        assert rel_l2(outs[0], outs[1]) <= 5e-3


# ---- every MFMA tile configuration ------------------------------------------

N_TILES = 4     # MFMA tile configurations of the projection GEMM, fallback last


@pytest.fixture
def force_tile(monkeypatch):
    def set_tile(t):
        monkeypatch.setenv("ORCH_GEMM_TILE", str(t))
    return set_tile


@pytest.mark.parametrize("tile", range(N_TILES))
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_linear_every_tile(orch_lib, force_tile, tile, epi):
    """Each tile shape (forced; N = 768 and K = 1152 fit all of them) on a
    ragged M, with every epilogue."""
    force_tile(tile)
    test_linear(orch_lib, "bf16", 333, 1152, 768, epi)


@pytest.mark.parametrize("tile", range(N_TILES))
def test_qkv_scatter_every_tile(orch_lib, force_tile, tile):
    force_tile(tile)
    test_qkv_scatter(orch_lib, "bf16", 768, 12, 200, 576, 192)


# ---- attention over fresh + stale K/V --------------------------------------

def _attention_case(orch_lib, dtype, B, heads, d, n_q, n_kv, fresh_begin, n_fresh, seed,
                    sample_rows=None, split=True, k_ramp=0.0, shift=0.0, k_spike=0.0):
    """k_ramp: key j's vector scaled by 1 + k_ramp j / n_kv (scores grow along
    the key stream, so the running max moves mid-stream); shift: the first
    channel of every head set to `shift` in Q and K (every score of a query
    raised by the same large amount: softmax unchanged, running max large);
    k_spike: the 32 keys from n_kv / 2 on score k_spike-proportionally higher
    (a jump of over 127 in log2 units mid-stream: exp2 of the scores overflows
    before the running max is raised)."""
    H = heads * d
    R = int(np.sqrt(n_kv))
    hdr = {"hidden": H, "heads": heads, "grid": R}
    rng = np.random.default_rng(seed)
    scale = 0.02 * np.sqrt(1152)
    q = rng.standard_normal((B, n_q, H)) * scale
    Ks = rng.standard_normal((B, n_kv, H)) * scale
    Vs = rng.standard_normal((B, n_kv, H))
    Kf = rng.standard_normal((B, max(n_fresh, 1), H)) * scale
    Vf = rng.standard_normal((B, max(n_fresh, 1), H))
    if k_ramp:
        Ks *= (1.0 + k_ramp * np.arange(n_kv) / n_kv)[None, :, None]
        Kf *= (1.0 + k_ramp * (fresh_begin + np.arange(Kf.shape[1])) / n_kv)[None, :, None]
    if shift:
        for arr in (q, Ks, Kf):
            arr[:, :, 0::d] = shift
    if k_spike:
        # channel 1 of every head: 16 in Q, k_spike in the 32 spiked keys, so
        # their scores share an offset of 16 k_spike / sqrt(d) (the offset's
        # rounding cancels in the softmax over them; the others vanish)
        j0 = n_kv // 2
        q[:, :, 1::d] = 16.0
        Ks[:, j0:j0 + 32, 1::d] = k_spike
        f0, f1 = max(j0 - fresh_begin, 0), min(j0 + 32 - fresh_begin, Kf.shape[1])
        if n_fresh and f0 < f1:
            Kf[:, f0:f1, 1::d] = k_spike
    qd = to_dev(np.stack([q[b].reshape(n_q, heads, d).transpose(1, 0, 2) for b in range(B)]), dtype)
    stale = np.concatenate([dit.kv_to_buffer_layout(hdr, Ks[b], Vs[b]) for b in range(B)])
    fresh = np.concatenate([dit.kv_to_buffer_layout(hdr, Kf[b], Vf[b]) for b in range(B)])
    out = empty((B, n_q, H), dtype)
    wsb = orch_lib.attention_workspace_bytes(B, heads, n_q, n_kv, d, code(dtype)) if split else 0
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV) if wsb else None
    orch_lib.attention(qd, to_dev(stale, dtype), 2 * n_kv * H, to_dev(fresh, dtype),
                       2 * max(n_fresh, 1) * H, fresh_begin, n_fresh, B, heads, n_q, n_kv, d, out,
                       code(dtype), workspace=ws)
    got = to_host(out)
    rows = np.arange(n_q) if sample_rows is None else sample_rows
    errs = []
    for b in range(B):
        K, V = rounded(Ks[b], dtype), rounded(Vs[b], dtype)
        if n_fresh:
            K, V = dit.assemble_kv((K, V), rounded(Kf[b][:n_fresh], dtype),
                                   rounded(Vf[b][:n_fresh], dtype), fresh_begin)
        ref = dit.attention(rounded(q[b][rows], dtype), K, V, heads)
        errs.append(rel_l2(got[b][rows], ref))
    return max(errs)


@pytest.mark.parametrize("dtype,heads,d,n_q,n_kv,fb,nf", [
    ("f32", 4, 32, 32, 64, 0, 32),
    ("f32", 4, 32, 20, 64, 24, 0),
    ("bf16", 6, 64, 96, 256, 96, 96),
    ("bf16", 6, 64, 100, 256, 0, 0),
    ("bf16", 16, 72, 384, 1024, 640, 384),
    ("bf16", 16, 72, 130, 1024, 8, 128),
    ("bf16", 2, 72, 1, 64, 0, 0),
])
def test_attention(orch_lib, dtype, heads, d, n_q, n_kv, fb, nf):
    err = _attention_case(orch_lib, dtype, 2, heads, d, n_q, n_kv, fb, nf, seed=n_q + n_kv + d)
    assert err <= (1e-5 if dtype == "f32" else 1e-2), err


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("d,n_q,n_kv,fb,nf", [
    (72, 384, 4096, 1920, 384), (72, 96, 1024, 512, 96), (72, 384, 1024, 0, 0),
    (72, 200, 1024, 64, 200), (64, 1280, 2304, 256, 1280), (72, 3328, 4096, 2048, 2048)])
def test_attention_split_keys(orch_lib, split, d, n_q, n_kv, fb, nf):
    """With a workspace, query tiles are cut between workgroups (parts of a
    tile from 1 to 8 workgroups, merged by a second kernel); without one,
    every tile stays whole.  Both agree with the oracle."""
    assert orch_lib.attention_workspace_bytes(2, 16, n_q, n_kv, d, 1) > 0
    err = _attention_case(orch_lib, "bf16", 2, 16, d, n_q, n_kv, fb, nf, seed=n_q + d + 1,
                          split=split)
    assert err <= 1e-2, err


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("d,n_q,n_kv,fb,nf", [(72, 384, 1024, 256, 384), (64, 1280, 2304, 256, 1280),
                                             (72, 1280, 4096, 0, 1280), (72, 1664, 4096, 0, 1664)])
@pytest.mark.parametrize("k_ramp,shift,k_spike", [(12.0, 0.0, 0.0), (0.0, 48.0, 0.0), (12.0, 48.0, 0.0),
                                                  (0.0, 0.0, 64.0)])
def test_attention_running_max(orch_lib, split, d, n_q, n_kv, fb, nf, k_ramp, shift, k_spike):
    """The lazy running max: scores growing along the key stream (the max is
    raised and O rescaled mid-stream, also in the pending probabilities of
    the lagging PV product), and a large common score offset (a running max
    of several hundred in log2 units, beyond one bf16 in the d = 72 max
    column).  Sampled query rows at the large shapes."""
    rows = np.r_[np.arange(0, n_q, 37), n_q - 1] if n_q > 1000 else None
    err = _attention_case(orch_lib, "bf16", 2, 16, d, n_q, n_kv, fb, nf, seed=n_q + d + 7, split=split,
                          sample_rows=rows, k_ramp=k_ramp, shift=shift, k_spike=k_spike)
    assert err <= 1e-2, err


def test_attention_full_xl_shape_sampled(orch_lib):
    """DiT-XL/2 1024px, 40% band: 1664 queries x 4096 keys, 16 heads, d = 72."""
    rows = np.r_[np.arange(0, 1664, 97), 1663]
    err = _attention_case(orch_lib, "bf16", 2, 16, 72, 1664, 4096, 0, 1664, seed=5, sample_rows=rows)
    assert err <= 1e-2, err


# ---- conditioning, patch embedding, final layer -----------------------------

def _ctx(orch_lib, cfg):
    blob = generate.make_weight_blob(cfg, 0)
    ctx = orch_lib.DiTStep(cfg, blob)
    hdr, params = oblob.read_blob(blob)
    return ctx, hdr, params


@pytest.mark.parametrize("cfg", [configs.TINY, configs.DIT_S2_256,
                                 configs.scaled(configs.DIT_XL2_512, n_blocks=3)],
                         ids=lambda c: c.name)
def test_conditioning(orch_lib, cfg):
    ctx, hdr, params = _ctx(orch_lib, cfg)
    labels = generate.make_labels(cfg, 0)
    H, L = cfg.hidden, cfg.n_blocks
    out = empty((cfg.cfg_batch, 6 * H * L + 2 * H))
    for t in (0, 500, 999):
        ctx.conditioning(t, labels, out)
        c = dit.conditioning(hdr, params, t, labels)
        blocks, fin = dit.adaln_vectors(hdr, params, c)
        ref = np.concatenate([np.concatenate(blk, axis=1) for blk in blocks] + list(fin), axis=1)
        err = rel_l2(to_host(out), ref)
        assert err <= 1e-5, (t, err)


@pytest.mark.parametrize("cfg,rb,re", [(configs.TINY, 0, 4), (configs.TINY, 3, 8),
                                       (configs.DIT_S2_256, 5, 11)], ids=str)
def test_patch_embed(orch_lib, cfg, rb, re):
    ctx, hdr, params = _ctx(orch_lib, cfg)
    x = generate.make_latent(cfg, 0)
    n_tok = (re - rb) * cfg.R
    out = empty((cfg.cfg_batch, n_tok, cfg.hidden))
    ctx.patch_embed(to_dev(x), rb, re, out)
    ref = dit.patch_embed(hdr, params, x.astype(np.float64), rb, re)
    got = to_host(out)
    for b in range(cfg.cfg_batch):
        assert rel_l2(got[b], ref) <= 1e-6


@pytest.mark.parametrize("cfg,rb,re", [(configs.TINY, 2, 6), (configs.DIT_S2_256, 0, 6),
                                       (configs.scaled(configs.DIT_XL2_512, n_blocks=1), 10, 22)],
                         ids=str)
def test_final_layer(orch_lib, cfg, rb, re):
    ctx, hdr, params = _ctx(orch_lib, cfg)
    rng = np.random.default_rng(rb)
    n_tok = (re - rb) * cfg.R
    H, L, B = cfg.hidden, cfg.n_blocks, cfg.cfg_batch
    h = rng.standard_normal((B, n_tok, H))
    mod = rng.standard_normal((B, 6 * H * L + 2 * H)) * 0.1
    out = empty((B, cfg.out_ch, (re - rb) * cfg.patch, cfg.latent))
    ctx.final_layer(to_dev(h), rb, re, to_dev(mod), out)
    got = to_host(out)
    hr, mr = rounded(h, "f32"), rounded(mod, "f32")
    for b in range(B):
        y = dit.final_layer(hdr, params, hr[b], mr[b, 6 * H * L:6 * H * L + H], mr[b, 6 * H * L + H:])
        ref = dit.unpatchify_rows(hdr, y, re - rb)
        assert rel_l2(got[b], ref) <= (1e-6 if cfg.dtype == "f32" else 1e-2)


# ---- guidance + scheduler update --------------------------------------------

@pytest.mark.parametrize("n", [1, 7, 4096, 26624, (1 << 20) + 3])
@pytest.mark.parametrize("guided,noise", [(False, False), (True, False), (True, True)])
def test_scheduler_update(orch_lib, n, guided, noise):
    rng = np.random.default_rng(n)
    x, ec, eu, z = (rng.standard_normal(n).astype(np.float32) for _ in range(4))
    t, tp = 780, 760
    eta = 0.5 if noise else 0.0
    a, b, c = osched.ddim_coefficients(osched.alpha_bar(), t, tp, eta)
    out = empty((n,))
    orch_lib.scheduler_update(to_dev(x), to_dev(ec), to_dev(eu) if guided else None, 1.5,
                              to_dev(z) if noise else None, a, b, c, out)
    e = dit.guided_eps(np.stack([ec, eu]).astype(np.float64), 1.5) if guided else ec.astype(np.float64)
    ref = osched.scheduler_update(x, e, a, b, c, z if noise else None)
    assert rel_l2(to_host(out), ref) <= 1e-6
