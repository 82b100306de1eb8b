"""The DiT denoiser on an elastic band of token rows with stale K/V (oracle).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

What one device computes per executed step (Algorithm 1, "one-step inference
on p_i with buffer"; patch parallelism with stale activation reuse, §II-B):
the denoiser eps_theta(x, t) evaluated for the tokens of its band of latent
rows.  Every operation of the DiT is token-local except attention; there the
band's queries attend over the keys/values of the whole image, fresh for the
band's own tokens and taken from the stale buffer for every other token.
Classifier-free guidance combines the two label branches, and the scheduler
update of §I / Lemma 1 produces the band of the next sample.

DiT structure (the paper cites DiT but does not restate it; this is the
reading both sides follow):
  * patch embedding: a p x p, stride-p convolution == a linear map of the
    (channel, dy, dx)-ordered patch vector, plus the fixed position table
    row of the token's global index;
  * conditioning c = MLP(sinusoid_256(t)) + label_table[label], with the
    sinusoid [cos(t f_i), sin(t f_i)], f_i = 10000^(-i/128);
  * adaLN: SiLU(c) -> linear -> six H-vectors per block
    (shift1, scale1, gate1, shift2, scale2, gate2), two for the final layer;
  * block: h += gate1 * Attn(LN(h)(1 + scale1) + shift1)
           h += gate2 * MLP(LN(h)(1 + scale2) + shift2)
    LN without affine, eps 1e-6, biased variance; attention with a biased
    QKV projection, heads split contiguously, softmax(q k^T / sqrt(d)) v,
    then a biased output projection; MLP = fc1 -> GELU (tanh form) -> fc2;
  * final: LN(h)(1 + scale) + shift -> linear to p*p*C_out, unpatchified with
    the output vector ordered (dy, dx, channel).

Stale K/V buffer layout (the interface of the step call): for each block l
and guidance branch b, 2 * N_kv * H elements: first K as [heads][N_kv][d],
then V transposed as [heads][d][N_kv].  The full buffer is [L][B][...].
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import schedule
from .blob import bf16_to_float

LN_EPS = 1e-6


# ---- elementary functions -------------------------------------------------

def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def layer_norm(h, eps: float = LN_EPS):
    """LayerNorm over the last axis: no affine, biased variance."""
    mu = h.mean(axis=-1, keepdims=True)
    var = ((h - mu) ** 2).mean(axis=-1, keepdims=True)
    return (h - mu) / np.sqrt(var + eps)


def modulate(u, shift, scale):
    return u * (1.0 + scale) + shift


def linear(x, W, b):
    """y = x W^T + b with W stored [out][in]."""
    return x @ W.T + b


def timestep_embedding(t: float, dim: int = 256, dtype=np.float64) -> np.ndarray:
    half = dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    a = float(t) * f
    return np.concatenate([np.cos(a), np.sin(a)]).astype(dtype)


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, heads: int, q_chunk: int = 2048):
    """Multi-head attention. q [Nq, H], k/v [Nkv, H] -> [Nq, H].

    Each head j uses columns j*d .. (j+1)*d - 1.  Query rows are processed in
    chunks only to bound memory; every row is computed independently.
    """
    Nq, H = q.shape
    d = H // heads
    scale = 1.0 / math.sqrt(d)
    out = np.empty_like(q)
    for j in range(heads):
        sl = slice(j * d, (j + 1) * d)
        kh = k[:, sl]
        vh = v[:, sl]
        for s in range(0, Nq, q_chunk):
            e = min(Nq, s + q_chunk)
            p = softmax_rows((q[s:e, sl] @ kh.T) * scale)
            out[s:e, sl] = p @ vh
    return out


# ---- model pieces ---------------------------------------------------------

def conditioning(hdr, params, t: int, labels: Sequence[int], dtype=np.float64):
    """c[b] = t_embedder(t) + label_table[labels[b]]  -> [B, H]."""
    e = timestep_embedding(t, hdr["freq_dim"], dtype)
    te = linear(silu(linear(e, params["t_embedder.fc1.weight"], params["t_embedder.fc1.bias"])),
                params["t_embedder.fc2.weight"], params["t_embedder.fc2.bias"])
    table = params["y_embedder.table"]
    return np.stack([te + table[int(lb)] for lb in labels])


def adaln_vectors(hdr, params, c):
    """Per block (shift1, scale1, gate1, shift2, scale2, gate2), each [B, H],
    and the final (shift, scale)."""
    H = hdr["hidden"]
    sc = silu(c)
    blocks = []
    for l in range(hdr["n_blocks"]):
        m = linear(sc, params[f"blocks.{l}.adaLN.weight"], params[f"blocks.{l}.adaLN.bias"])
        blocks.append(tuple(m[:, i * H:(i + 1) * H] for i in range(6)))
    m = linear(sc, params["final.adaLN.weight"], params["final.adaLN.bias"])
    return blocks, (m[:, :H], m[:, H:2 * H])


def patchify_rows(hdr, x_full, row_begin: int, row_end: int):
    """Patch vectors of the band's tokens, [(row_end-row_begin)*R, C*p*p],
    ordered (channel, dy, dx); token order row-major over the band."""
    p, R, C = hdr["patch"], hdr["grid"], hdr["in_ch"]
    rows = []
    for i in range(row_begin, row_end):
        for j in range(R):
            blk = x_full[:, i * p:(i + 1) * p, j * p:(j + 1) * p]   # [C, p, p]
            rows.append(blk.reshape(C * p * p))
    return np.stack(rows)


def patch_embed(hdr, params, x_full, row_begin: int, row_end: int, dtype=np.float64):
    R = hdr["grid"]
    v = patchify_rows(hdr, np.asarray(x_full, dtype=dtype), row_begin, row_end)
    h = linear(v, params["x_embedder.weight"], params["x_embedder.bias"])
    return h + params["pos_embed"][row_begin * R:row_end * R]


def unpatchify_rows(hdr, y, n_rows: int):
    """[n_rows*R, p*p*C_out] ordered (dy, dx, channel) -> [C_out, n_rows*p, R*p]."""
    p, R, Co = hdr["patch"], hdr["grid"], hdr["out_ch"]
    out = np.empty((Co, n_rows * p, R * p), dtype=y.dtype)
    for i in range(n_rows):
        for j in range(R):
            v = y[i * R + j].reshape(p, p, Co)
            for dy in range(p):
                for dx in range(p):
                    out[:, i * p + dy, j * p + dx] = v[dy, dx, :]
    return out


def final_layer(hdr, params, h, shift, scale):
    u = modulate(layer_norm(h), shift, scale)
    return linear(u, params["final.linear.weight"], params["final.linear.bias"])


# ---- stale K/V buffer layout ---------------------------------------------

def _as_float(a, dtype):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_to_float(a).astype(dtype)
    return a.astype(dtype)


def stale_kv_block(hdr, stale_kv, B: int, l: int, b: int, dtype=np.float64):
    """Token-major K and V [N_kv, H] of block l, branch b, read from the buffer."""
    H, heads = hdr["hidden"], hdr["heads"]
    d = H // heads
    N = hdr["grid"] ** 2
    per = 2 * N * H
    base = (l * B + b) * per
    flat = np.asarray(stale_kv).reshape(-1)
    kpart = _as_float(flat[base:base + N * H], dtype).reshape(heads, N, d)
    vpart = _as_float(flat[base + N * H:base + per], dtype).reshape(heads, d, N)
    K = kpart.transpose(1, 0, 2).reshape(N, H)
    V = vpart.transpose(2, 0, 1).reshape(N, H)
    return K, V


def kv_to_buffer_layout(hdr, K, V):
    """Token-major K, V [N, H] -> the buffer's (K [heads][N][d], V [heads][d][N])
    flattened and concatenated."""
    H, heads = hdr["hidden"], hdr["heads"]
    d = H // heads
    N = K.shape[0]
    kpart = K.reshape(N, heads, d).transpose(1, 0, 2).reshape(-1)
    vpart = V.reshape(N, heads, d).transpose(1, 2, 0).reshape(-1)
    return np.concatenate([kpart, vpart])


def assemble_kv(stale, k, v, tok0: int):
    """Keys/values the band attends over: the stale buffer's, with the band's
    own tokens [tok0, tok0 + N_q) replaced by the fresh k, v."""
    K, V = stale[0].copy(), stale[1].copy()
    K[tok0:tok0 + k.shape[0]] = k
    V[tok0:tok0 + v.shape[0]] = v
    return K, V


# ---- the step -------------------------------------------------------------

def denoiser_band(hdr, params, x_full, row_begin: int, row_end: int, t: int,
                  labels: Sequence[int], stale_kv=None, dtype=np.float64,
                  keep_kv: bool = False, keep_h: bool = False,
                  out_rows: Optional[Sequence[int]] = None):
    """eps_theta for the band's tokens, every guidance branch.

    Returns dict with
      eps     [B, C_out, 2r_p, W]  (r_p = band rows * p),
      kv      (if keep_kv) list over blocks of list over branches of the
              band's fresh (K, V), token-major [N_q, H],
      h       (if keep_h) residual stream after patch embedding and after
              every block, list of [B, N_q, H].

    out_rows (optional): band-relative token rows whose outputs are wanted.
    After the last block's QKV projection every token's output depends only
    on its own residual row and on the keys/values, so the last block's
    attention, MLP and the final layer are then evaluated for those rows'
    tokens only (its keys/values still come from every band token); eps
    covers those rows, in the order given: [B, C_out, len(out_rows)*p, W].
    """
    H, heads, L, R = hdr["hidden"], hdr["heads"], hdr["n_blocks"], hdr["grid"]
    B = len(labels)
    n_rows = row_end - row_begin
    Nq = n_rows * R
    tok0 = row_begin * R
    full = row_begin == 0 and row_end == R
    if stale_kv is None and not full:
        raise ValueError("a band of fewer than all rows needs the stale buffer")
    sel = None
    if out_rows is not None:
        if any(r < 0 or r >= n_rows for r in out_rows):
            raise ValueError("out_rows must be band-relative rows")
        sel = np.concatenate([np.arange(r * R, (r + 1) * R) for r in out_rows])

    c = conditioning(hdr, params, t, labels, dtype)
    blocks, (fshift, fscale) = adaln_vectors(hdr, params, c)
    h0 = patch_embed(hdr, params, x_full, row_begin, row_end, dtype)
    h = np.stack([h0.copy() for _ in range(B)])           # [B, Nq, H]
    kv_keep = [] if keep_kv else None
    h_keep = [h.copy()] if keep_h else None

    for l in range(L):
        pre = f"blocks.{l}."
        s1, c1, g1, s2, c2, g2 = blocks[l]
        restrict = sel is not None and l == L - 1
        layer_kv = []
        new_h = []
        for b in range(B):
            u = modulate(layer_norm(h[b]), s1[b], c1[b])
            qkv = linear(u, params[pre + "qkv.weight"], params[pre + "qkv.bias"])
            q, k, v = qkv[:, :H], qkv[:, H:2 * H], qkv[:, 2 * H:]
            if full:
                K, V = k, v
            else:
                K, V = assemble_kv(stale_kv_block(hdr, stale_kv, B, l, b, dtype), k, v, tok0)
            hb = h[b]
            if restrict:                      # only the wanted tokens leave the last block
                q, hb = q[sel], hb[sel]
            o = attention(q, K, V, heads)
            hb = hb + g1[b] * linear(o, params[pre + "proj.weight"], params[pre + "proj.bias"])
            u2 = modulate(layer_norm(hb), s2[b], c2[b])
            m = gelu_tanh(linear(u2, params[pre + "fc1.weight"], params[pre + "fc1.bias"]))
            hb = hb + g2[b] * linear(m, params[pre + "fc2.weight"], params[pre + "fc2.bias"])
            new_h.append(hb)
            if keep_kv:
                layer_kv.append((k, v))
        h = np.stack(new_h)
        if keep_kv:
            kv_keep.append(layer_kv)
        if keep_h:
            h_keep.append(h.copy())

    n_out = n_rows if sel is None else len(out_rows)
    eps = np.stack([unpatchify_rows(hdr, final_layer(hdr, params, h[b], fshift[b], fscale[b]),
                                    n_out) for b in range(B)])
    out = {"eps": eps}
    if keep_kv:
        out["kv"] = kv_keep
    if keep_h:
        out["h"] = h_keep
    return out


def guided_eps(eps, cfg_scale: float):
    """Classifier-free guidance: eps_u + g (eps_c - eps_u) with branch 0 the
    class label and branch 1 the null label; a single branch passes through."""
    if eps.shape[0] == 1:
        return eps[0]
    return eps[1] + cfg_scale * (eps[0] - eps[1])


def patch_step(hdr, params, x_full, row_begin: int, row_end: int, t: int, t_prev: int,
               labels: Sequence[int], cfg_scale: float, stale_kv=None, eta: float = 0.0,
               z=None, T: int = 1000, beta_start: float = 1e-4, beta_end: float = 2e-2,
               dtype=np.float64, keep_kv: bool = False, keep_h: bool = False,
               out_rows: Optional[Sequence[int]] = None) -> Dict:
    """One executed step of one device: eps for the band, guidance, and the
    scheduler update of the band rows (x_out = A x - Bc eps + C z).  With
    out_rows, eps and x_out cover only those band-relative token rows."""
    res = denoiser_band(hdr, params, x_full, row_begin, row_end, t, labels, stale_kv,
                        dtype, keep_kv, keep_h, out_rows)
    ab = schedule.alpha_bar(T, beta_start, beta_end)
    A, Bc, C = schedule.ddim_coefficients(ab, t, t_prev, eta)
    p = hdr["patch"]
    band = range(row_end - row_begin) if out_rows is None else out_rows
    rows = [(row_begin + r) * p + dy for r in band for dy in range(p)]
    x_band = np.asarray(x_full, dtype=np.float64)[:, rows, :]
    z_band = None if z is None else np.asarray(z, dtype=np.float64)[:, rows, :]
    g = guided_eps(res["eps"].astype(np.float64), cfg_scale)
    res["eps_guided"] = g
    res["x_out"] = schedule.scheduler_update(x_band, g, A, Bc, C, z_band)
    res["coeffs"] = (A, Bc, C)
    return res


def full_step(hdr, params, x_full, t: int, t_prev: int, labels, cfg_scale: float, **kw):
    """The unpartitioned step: the band is every row, so nothing is stale."""
    return patch_step(hdr, params, x_full, 0, hdr["grid"], t, t_prev, labels, cfg_scale,
                      None, **kw)


def refreshed_buffer(hdr, stale_kv, kv, row_begin: int, row_end: int, dtype=np.float64):
    """The buffer after a refresh: the band's tokens of every block/branch hold
    the fresh K/V, every other token is unchanged.  Returns float `dtype`."""
    L, R = hdr["n_blocks"], hdr["grid"]
    B = len(kv[0])
    out = []
    tok = slice(row_begin * R, row_end * R)
    for l in range(L):
        for b in range(B):
            K, V = stale_kv_block(hdr, stale_kv, B, l, b, dtype)
            K = K.copy()
            V = V.copy()
            K[tok] = kv[l][b][0]
            V[tok] = kv[l][b][1]
            out.append(kv_to_buffer_layout(hdr, K, V))
    return np.concatenate(out)


def full_kv_buffer(hdr, kv):
    """The buffer holding a full-image step's own K/V (every token fresh)."""
    out = []
    for layer in kv:
        for (K, V) in layer:
            out.append(kv_to_buffer_layout(hdr, K, V))
    return np.concatenate(out)


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))
