"""Pins of the oracle's DiT band step against library routines, brute force,
closed forms and the invariants of patch parallelism with stale K/V (§II-B,
Algorithm 1)."""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import blob as oblob
from oracle import dit, schedule
from seeded_inputs import configs, generate
from tests._torch_dit import torch_dit_eps

TINY_CFG2 = configs.scaled(configs.TINY, name="tiny_cfg2", cfg_batch=2)


@pytest.fixture(scope="module")
def tiny():
    cfg = TINY_CFG2
    hdr, params = oblob.read_blob(generate.make_weight_blob(cfg, seed=0))
    x = generate.make_latent(cfg, 0).astype(np.float64)
    labels = generate.make_labels(cfg, 0)
    return cfg, hdr, params, x, labels


# ---- elementary functions -------------------------------------------------

def test_gelu_tanh_values():
    x = np.linspace(-6, 6, 101)
    ref = F.gelu(torch.tensor(x), approximate="tanh").numpy()
    np.testing.assert_allclose(dit.gelu_tanh(x), ref, rtol=1e-14, atol=1e-15)
    assert dit.gelu_tanh(np.array(0.0)) == 0.0
    assert dit.gelu_tanh(np.array(30.0)) == pytest.approx(30.0)
    assert abs(dit.gelu_tanh(np.array(-30.0))) < 1e-12


def test_silu_values():
    x = np.linspace(-8, 8, 33)
    np.testing.assert_allclose(dit.silu(x), F.silu(torch.tensor(x)).numpy(), rtol=1e-14)


def test_layer_norm():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((7, 96)) * 3 + 1
    ref = F.layer_norm(torch.tensor(h), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(dit.layer_norm(h), ref, rtol=1e-12, atol=1e-12)
    const = np.full((2, 32), 4.5)
    u = dit.modulate(dit.layer_norm(const), np.full(32, 0.25), np.full(32, 3.0))
    np.testing.assert_allclose(u, 0.25)          # constant row -> LN = 0 -> shift


def test_timestep_embedding_values():
    e0 = dit.timestep_embedding(0, 256)
    np.testing.assert_array_equal(e0, np.r_[np.ones(128), np.zeros(128)])
    e1 = dit.timestep_embedding(1, 256)
    assert e1[0] == pytest.approx(0.5403023058681398, abs=1e-16)
    assert e1[128] == pytest.approx(0.8414709848078965, abs=1e-16)
    # f_127 = 10000^(-127/128)
    assert e1[127] == pytest.approx(math.cos(10000 ** (-127 / 128)), abs=1e-16)


# ---- attention ------------------------------------------------------------

def _attention_bruteforce(q, k, v, heads):
    Nq, H = q.shape
    d = H // heads
    out = np.zeros_like(q)
    for j in range(heads):
        for i in range(Nq):
            s = [sum(q[i, j * d + a] * k[n, j * d + a] for a in range(d)) / math.sqrt(d)
                 for n in range(k.shape[0])]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = sum(w)
            for a in range(d):
                out[i, j * d + a] = sum(w[n] * v[n, j * d + a] for n in range(k.shape[0])) / z
    return out


@pytest.mark.parametrize("nq,nkv,heads,d", [(1, 1, 1, 4), (3, 5, 2, 4), (4, 7, 3, 3), (1, 9, 2, 8)])
def test_attention_bruteforce(nq, nkv, heads, d):
    rng = np.random.default_rng(nq * 100 + nkv)
    H = heads * d
    q, k, v = (rng.standard_normal((n, H)) for n in (nq, nkv, nkv))
    np.testing.assert_allclose(dit.attention(q, k, v, heads), _attention_bruteforce(q, k, v, heads),
                               rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((5, 8))
    v = rng.standard_normal((1, 8))
    k = rng.standard_normal((1, 8))
    np.testing.assert_allclose(dit.attention(q, k, v, 2), np.repeat(v, 5, 0), rtol=1e-14)
    k_eq = np.repeat(rng.standard_normal((1, 8)), 6, 0)
    v6 = rng.standard_normal((6, 8))
    np.testing.assert_allclose(dit.attention(q, k_eq, v6, 2), np.repeat(v6.mean(0, keepdims=True), 5, 0),
                               rtol=1e-12)
    s = rng.standard_normal((4, 9))
    np.testing.assert_allclose(dit.softmax_rows(s), dit.softmax_rows(s + 7.5), rtol=1e-13)


def test_attention_vs_sdpa():
    rng = np.random.default_rng(4)
    heads, d = 4, 16
    q = rng.standard_normal((37, heads * d))
    k = rng.standard_normal((70, heads * d))
    v = rng.standard_normal((70, heads * d))
    tq, tk, tv = (torch.tensor(a).reshape(a.shape[0], heads, d).transpose(0, 1) for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(37, heads * d).numpy()
    np.testing.assert_allclose(dit.attention(q, k, v, heads, q_chunk=16), ref, rtol=1e-12, atol=1e-13)


# ---- patch embedding / unpatchify -----------------------------------------

def test_patch_embed_is_strided_conv(tiny):
    cfg, hdr, params, x, _ = tiny
    H, p, C, R = cfg.hidden, cfg.patch, cfg.in_ch, cfg.R
    ref = F.conv2d(torch.tensor(x)[None], torch.tensor(params["x_embedder.weight"]).reshape(H, C, p, p),
                   torch.tensor(params["x_embedder.bias"]), stride=p)[0]        # [H, R, R]
    ref = ref.reshape(H, R * R).T.numpy() + params["pos_embed"]
    got = dit.patch_embed(hdr, params, x, 2, 6)
    np.testing.assert_allclose(got, ref[2 * R:6 * R], rtol=1e-12, atol=1e-13)


def test_unpatchify_is_pixel_shuffle():
    hdr = {"patch": 2, "grid": 3, "out_ch": 4}
    rng = np.random.default_rng(5)
    y = rng.standard_normal((2 * 3, 16))     # 2 rows of 3 tokens, (dy, dx, c)
    got = dit.unpatchify_rows(hdr, y, 2)
    yy = torch.tensor(y).reshape(2, 3, 2, 2, 4).permute(4, 2, 3, 0, 1).reshape(16, 2, 3)
    ref = F.pixel_shuffle(yy[None], 2)[0].numpy()
    np.testing.assert_array_equal(got, ref)
    # one hand-placed element: token (1, 2), dy=1, dx=0, channel 3
    assert got[3, 1 * 2 + 1, 2 * 2 + 0] == y[1 * 3 + 2, (1 * 2 + 0) * 4 + 3]


def test_blob_roundtrip():
    cfg = configs.TINY
    b = generate.make_weight_blob(cfg, 0)
    hdr, params = oblob.read_blob(b)
    assert hdr["grid"] == 8 and hdr["hidden"] == 128 and hdr["dtype"] == "f32"
    rng = np.random.default_rng([0, configs.STREAM_WEIGHTS])
    w0 = (rng.standard_normal((128, 16)) * 0.02).astype(np.float32)
    np.testing.assert_array_equal(params["x_embedder.weight"], w0)
    cb = configs.scaled(cfg, dtype="bf16")
    hb, pb = oblob.read_blob(generate.make_weight_blob(cb, 0))
    assert hb["dtype"] == "bf16"
    # bf16 storage = round-to-nearest-even of the float32 draw
    np.testing.assert_allclose(pb["x_embedder.weight"], w0, rtol=2 ** -8)
    bits = generate.f32_to_bf16_bits(np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0], np.float32))
    assert list(bits) == [0x3F80, 0x3F82, 0x8000]


# ---- the full-image step against an independent torch DiT -----------------

def test_full_step_matches_torch_dit(tiny):
    cfg, hdr, params, x, labels = tiny
    t = 750
    got = dit.denoiser_band(hdr, params, x, 0, cfg.R, t, labels)["eps"]
    ref = torch_dit_eps(hdr, params, x, t, labels)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_full_step_matches_torch_dit_s2():
    cfg = configs.scaled(configs.DIT_S2_256, dtype="f32", n_blocks=3)
    hdr, params = oblob.read_blob(generate.make_weight_blob(cfg, 1))
    x = generate.make_latent(cfg, 1).astype(np.float64)
    got = dit.denoiser_band(hdr, params, x, 0, cfg.R, 500, [7])["eps"]
    ref = torch_dit_eps(hdr, params, x, 500, [7])
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-11)


# ---- invariants of the band step -------------------------------------------

def test_i1_all_rows_ignores_stale(tiny):
    cfg, hdr, params, x, labels = tiny
    nan_buf = np.full(generate.stale_kv_elems(cfg), np.nan)
    a = dit.patch_step(hdr, params, x, 0, cfg.R, 500, 250, labels, 1.5, nan_buf)
    b = dit.full_step(hdr, params, x, 500, 250, labels, 1.5)
    np.testing.assert_array_equal(a["x_out"], b["x_out"])
    assert np.isfinite(a["x_out"]).all()


def _full_with_kv(hdr, params, x, labels, t=500, tp=250):
    res = dit.full_step(hdr, params, x, t, tp, labels, 1.5, keep_kv=True)
    return res, dit.full_kv_buffer(hdr, res["kv"])


@pytest.mark.parametrize("bands", [[(0, 3), (3, 4), (4, 8)], [(0, 1), (1, 7), (7, 8)], [(0, 8)]])
def test_i2_stitched_bands_equal_full_step(tiny, bands):
    cfg, hdr, params, x, labels = tiny
    full, buf = _full_with_kv(hdr, params, x, labels)
    p = cfg.patch
    stitched = np.zeros_like(full["x_out"])
    eps = np.zeros_like(full["eps"])
    for rb, re in bands:
        r = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, buf)
        stitched[:, rb * p:re * p] = r["x_out"]
        eps[:, :, rb * p:re * p] = r["eps"]
    np.testing.assert_allclose(stitched, full["x_out"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(eps, full["eps"], rtol=1e-12, atol=1e-12)


def test_i3_locality(tiny):
    cfg, hdr, params, x, labels = tiny
    rb, re = 2, 5
    R, p = cfg.R, cfg.patch
    stale = generate.make_stale_kv(cfg, 0).astype(np.float64)
    base = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, stale, keep_kv=True)
    # x outside the band has no effect
    x2 = x.copy()
    x2[:, :rb * p] += 10.0
    x2[:, re * p:] -= 3.0
    np.testing.assert_array_equal(
        dit.patch_step(hdr, params, x2, rb, re, 500, 250, labels, 1.5, stale)["x_out"], base["x_out"])
    # a stale token outside the band does matter; one inside the band does not
    N, H = cfg.n_kv, cfg.hidden
    per = 2 * N * H
    d = cfg.head_dim
    s_out = stale.copy()
    s_out[0 * per + 1 * N * d + 0 * d + 3] = 5.0     # block 0, branch 0, K head 1, token 0
    changed = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, s_out)["x_out"]
    assert np.abs(changed - base["x_out"]).max() > 1e-9
    s_in = stale.copy()
    tok = rb * R + 1
    s_in[0 * per + 1 * N * d + tok * d + 3] = np.nan   # a band token: overwritten by fresh K
    same = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, s_in)["x_out"]
    np.testing.assert_array_equal(same, base["x_out"])
    s_nan = stale.copy()
    s_nan[per + N * H + 2 * d * N + 0] = np.nan         # block 0, branch 1, V, non-band token
    bad = dit.patch_step(hdr, params, x, rb, re, 500, 250, labels, 1.5, s_nan)["x_out"]
    assert np.isnan(bad).any()
    # refresh: band tokens hold fresh K/V, everything else is bitwise unchanged
    newbuf = dit.refreshed_buffer(hdr, stale, base["kv"], rb, re)
    for l, b in itertools.product(range(cfg.n_blocks), range(cfg.cfg_batch)):
        K0, V0 = dit.stale_kv_block(hdr, stale, 2, l, b)
        K1, V1 = dit.stale_kv_block(hdr, newbuf, 2, l, b)
        band = slice(rb * R, re * R)
        np.testing.assert_array_equal(np.delete(K1, band, 0), np.delete(K0, band, 0))
        np.testing.assert_array_equal(np.delete(V1, band, 0), np.delete(V0, band, 0))
        np.testing.assert_array_equal(K1[band], base["kv"][l][b][0])
        np.testing.assert_array_equal(V1[band], base["kv"][l][b][1])


def test_buffer_layout_roundtrip(tiny):
    cfg, hdr, params, x, labels = tiny
    rng = np.random.default_rng(9)
    K = rng.standard_normal((cfg.n_kv, cfg.hidden))
    V = rng.standard_normal((cfg.n_kv, cfg.hidden))
    flat = dit.kv_to_buffer_layout(hdr, K, V)
    N, d = cfg.n_kv, cfg.head_dim
    # hand-placed: K head 2, token 5, dim 7 ; V head 3, dim 1, token 9
    assert flat[2 * N * d + 5 * d + 7] == K[5, 2 * d + 7]
    assert flat[N * cfg.hidden + 3 * d * N + 1 * N + 9] == V[9, 3 * d + 1]
    buf = np.concatenate([flat] * (cfg.n_blocks * 2))
    K2, V2 = dit.stale_kv_block(hdr, buf, 2, 1, 1)
    np.testing.assert_array_equal(K2, K)
    np.testing.assert_array_equal(V2, V)


def test_i4_zero_gates_reduce_to_final_of_embedding(tiny):
    cfg, hdr, params, x, labels = tiny
    H = cfg.hidden
    P = {k: v.copy() for k, v in params.items()}
    for l in range(cfg.n_blocks):
        for g in (2, 5):                      # gate1, gate2 slices of the adaLN output
            P[f"blocks.{l}.adaLN.weight"][g * H:(g + 1) * H] = 0
            P[f"blocks.{l}.adaLN.bias"][g * H:(g + 1) * H] = 0
    P["y_embedder.table"][:] = 0
    eps = dit.denoiser_band(hdr, P, x, 1, 6, 250, labels,
                            generate.make_stale_kv(cfg, 0).astype(np.float64))["eps"]
    # closed form: final layer of the patch embedding, via torch routines
    p, C, R, Co = cfg.patch, cfg.in_ch, cfg.R, cfg.out_ch
    T = {k: torch.tensor(v) for k, v in P.items()}
    h = F.conv2d(torch.tensor(x)[None], T["x_embedder.weight"].reshape(H, C, p, p),
                 T["x_embedder.bias"], stride=p)[0].reshape(H, -1).T + T["pos_embed"]
    half = 128
    fr = torch.exp(-math.log(1e4) * torch.arange(half, dtype=torch.float64) / half)
    te = torch.cat([torch.cos(250 * fr), torch.sin(250 * fr)])
    c = F.linear(F.silu(F.linear(te, T["t_embedder.fc1.weight"], T["t_embedder.fc1.bias"])),
                 T["t_embedder.fc2.weight"], T["t_embedder.fc2.bias"])
    sh, sc = F.linear(F.silu(c), T["final.adaLN.weight"], T["final.adaLN.bias"]).chunk(2)
    y = F.linear(F.layer_norm(h, (H,), eps=1e-6) * (1 + sc) + sh, T["final.linear.weight"],
                 T["final.linear.bias"])
    y = y.reshape(R, R, p, p, Co).permute(4, 2, 3, 0, 1).reshape(Co * p * p, R, R)
    ref = F.pixel_shuffle(y[None], p)[0].numpy()[:, 1 * p:6 * p]
    np.testing.assert_allclose(eps[0], ref, rtol=1e-11, atol=1e-12)
    np.testing.assert_array_equal(eps[0], eps[1])          # zero label table: branches equal
    g1 = dit.guided_eps(eps, 1.5)
    g2 = dit.guided_eps(eps, 7.0)
    np.testing.assert_allclose(g1, g2, rtol=0, atol=1e-15)


def test_guidance_and_update_composition(tiny):
    cfg, hdr, params, x, labels = tiny
    stale = generate.make_stale_kv(cfg, 0)
    r = dit.patch_step(hdr, params, x, 0, 4, 750, 500, labels, 1.5, stale)
    e = r["eps"]
    g = e[1] + 1.5 * (e[0] - e[1])
    A, Bc, C = schedule.ddim_coefficients(schedule.alpha_bar(), 750, 500)
    np.testing.assert_allclose(r["x_out"], A * x[:, :8] - Bc * g, rtol=1e-14, atol=1e-14)


def _branch_order_holds(hdr, params, x, labels, step=dit.patch_step):
    """Guidance at g = 0 is the null-label model alone, at g = 1 the
    class-label model alone (eps_u + g (eps_c - eps_u) with eps_c from the
    class label and eps_u from the null label): checked against single-branch
    runs of the denoiser, which involve no guidance at all."""
    cls, null = int(labels[0]), int(labels[1])
    R = hdr["grid"]
    ok = True
    for g, lab in ((0.0, null), (1.0, cls)):
        two = step(hdr, params, x, 0, R, 500, 250, [cls, null], g)
        one = step(hdr, params, x, 0, R, 500, 250, [lab], 7.0)   # g unused for one branch
        ok &= bool(np.allclose(two["eps_guided"], one["eps_guided"], rtol=1e-12, atol=1e-13))
        ok &= bool(np.allclose(two["x_out"], one["x_out"], rtol=1e-12, atol=1e-13))
    return ok


def test_guidance_branch_order_from_single_branch_runs(tiny):
    cfg, hdr, params, x, labels = tiny
    assert labels[1] == cfg.num_classes and labels[0] != labels[1]
    assert _branch_order_holds(hdr, params, x, labels)
    # and the two single-branch runs differ, so the pin has teeth
    R = cfg.R
    a = dit.patch_step(hdr, params, x, 0, R, 500, 250, [int(labels[0])], 1.0)["eps_guided"]
    b = dit.patch_step(hdr, params, x, 0, R, 500, 250, [int(labels[1])], 1.0)["eps_guided"]
    assert dit.rel_l2(a, b) > 1e-3


def test_sampled_output_rows_equal_the_whole_band(tiny):
    """out_rows restricts the last block and the final layer to some token
    rows; every output row is the same as in the whole-band evaluation."""
    cfg, hdr, params, x, labels = tiny
    stale = generate.make_stale_kv(cfg, 0)
    rb, re = 1, 7
    whole = dit.patch_step(hdr, params, x, rb, re, 750, 500, labels, 1.5, stale)
    rows = [4, 0, 5]
    part = dit.patch_step(hdr, params, x, rb, re, 750, 500, labels, 1.5, stale, out_rows=rows)
    p = cfg.patch
    lat = [r * p + dy for r in rows for dy in range(p)]
    np.testing.assert_allclose(part["eps"], whole["eps"][:, :, lat], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(part["x_out"], whole["x_out"][:, lat], rtol=1e-13, atol=1e-14)
    with pytest.raises(ValueError):
        dit.patch_step(hdr, params, x, rb, re, 750, 500, labels, 1.5, stale, out_rows=[6])
