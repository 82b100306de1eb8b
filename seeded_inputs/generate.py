"""Seeded synthetic inputs: the weight blob, latents, noise, labels and the
stale K/V buffer.

Nothing here computes any part of the denoising step.  Every random number
comes from ``numpy.random.default_rng([seed, stream])`` so both the CPU
oracle and the GPU path see identical bytes.

Weight blob format (little endian) -- the contract between the two sides:

  header, 256 bytes:
    0   char[8]  magic "ORCHDIT1"
    8   u32      version (1)
    12  u32      dtype   (0 = f32, 1 = bf16 bits)
    16  u32[10]  n_blocks, hidden, heads, mlp_hidden, in_ch, out_ch, patch,
                 grid (token rows R), num_classes, freq_dim
    56  u32      n_tensors
    rest zero
  tensors, in the order of ``tensor_specs``, each starting at the next
  multiple of 256 bytes, row-major, every tensor in the blob dtype.

Linear weights are stored [out][in] (y = W x + b).  The patch-embedding
weight is [H][in_ch * p * p] with the input vector ordered (channel, dy, dx);
the final linear's output vector is ordered (dy, dx, channel).  Each block's
adaLN output is the six H-vectors (shift_msa, scale_msa, gate_msa,
shift_mlp, scale_mlp, gate_mlp); the final adaLN output is (shift, scale).
The label table has num_classes + 1 rows; the last row is the null label.
"""
from __future__ import annotations

import struct
from typing import List, Tuple

import numpy as np

from .configs import (DiTConfig, STREAM_LABELS, STREAM_LATENT, STREAM_NOISE,
                      STREAM_STALE, STREAM_WEIGHTS)

MAGIC = b"ORCHDIT1"
VERSION = 1
HEADER_BYTES = 256
ALIGN = 256
DTYPE_CODE = {"f32": 0, "bf16": 1}
INIT_STD = 0.02


def tensor_specs(cfg: DiTConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    H, F, L = cfg.hidden, cfg.mlp_hidden, cfg.n_blocks
    specs = [
        ("x_embedder.weight", (H, cfg.patch_dim)),
        ("x_embedder.bias", (H,)),
        ("pos_embed", (cfg.n_kv, H)),
        ("t_embedder.fc1.weight", (H, cfg.freq_dim)),
        ("t_embedder.fc1.bias", (H,)),
        ("t_embedder.fc2.weight", (H, H)),
        ("t_embedder.fc2.bias", (H,)),
        ("y_embedder.table", (cfg.num_classes + 1, H)),
    ]
    for l in range(L):
        p = f"blocks.{l}."
        specs += [
            (p + "adaLN.weight", (6 * H, H)), (p + "adaLN.bias", (6 * H,)),
            (p + "qkv.weight", (3 * H, H)), (p + "qkv.bias", (3 * H,)),
            (p + "proj.weight", (H, H)), (p + "proj.bias", (H,)),
            (p + "fc1.weight", (F, H)), (p + "fc1.bias", (F,)),
            (p + "fc2.weight", (H, F)), (p + "fc2.bias", (H,)),
        ]
    specs += [
        ("final.adaLN.weight", (2 * H, H)), ("final.adaLN.bias", (2 * H,)),
        ("final.linear.weight", (cfg.out_patch_dim, H)),
        ("final.linear.bias", (cfg.out_patch_dim,)),
    ]
    return specs


def _elem_bytes(cfg: DiTConfig) -> int:
    return 4 if cfg.dtype == "f32" else 2


def _align(n: int) -> int:
    return (n + ALIGN - 1) // ALIGN * ALIGN


def blob_layout(cfg: DiTConfig):
    """[(name, shape, byte_offset)], total_bytes."""
    off = HEADER_BYTES
    out = []
    eb = _elem_bytes(cfg)
    for name, shape in tensor_specs(cfg):
        out.append((name, shape, off))
        off = _align(off + int(np.prod(shape)) * eb)
    return out, off


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16, returned as uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(a)
    out = rounded.astype(np.uint16)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _encode(values: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(values, dtype=np.float32).view(np.uint8).ravel()
    return f32_to_bf16_bits(values.astype(np.float32)).view(np.uint8).ravel()


def fixed_sincos_pos_embed(H: int, R: int) -> np.ndarray:
    """The fixed (not learned) 2-D sine-cosine position table of a DiT, [R*R, H].

    Token n = i*R + j (row i, column j).  With Q = H/4 and w_k = 10000^(-k/Q):
    channels [0,Q) sin(j w_k), [Q,2Q) cos(j w_k), [2Q,3Q) sin(i w_k),
    [3Q,4Q) cos(i w_k).  It is a parameter table of the model, delivered in
    the blob so that neither side recomputes it.
    """
    assert H % 4 == 0
    Q = H // 4
    w = 1.0 / (10000.0 ** (np.arange(Q, dtype=np.float64) / Q))
    ii, jj = np.meshgrid(np.arange(R, dtype=np.float64), np.arange(R, dtype=np.float64),
                         indexing="ij")
    i = ii.reshape(-1, 1)
    j = jj.reshape(-1, 1)
    return np.concatenate([np.sin(j * w), np.cos(j * w), np.sin(i * w), np.cos(i * w)], axis=1)


def make_weight_blob(cfg: DiTConfig, seed: int = 0) -> np.ndarray:
    """The weight blob (uint8 array).  Every tensor except the fixed position
    table is drawn N(0, 0.02^2) in float64, in blob order, from one stream,
    then stored in the config dtype (RNE)."""
    layout, total = blob_layout(cfg)
    blob = np.zeros(total, dtype=np.uint8)
    hdr = struct.pack("<8sII10II", MAGIC, VERSION, DTYPE_CODE[cfg.dtype],
                      cfg.n_blocks, cfg.hidden, cfg.heads, cfg.mlp_hidden, cfg.in_ch,
                      cfg.out_ch, cfg.patch, cfg.R, cfg.num_classes, cfg.freq_dim,
                      len(layout))
    blob[:len(hdr)] = np.frombuffer(hdr, dtype=np.uint8)
    rng = np.random.default_rng([seed, STREAM_WEIGHTS])
    for name, shape, off in layout:
        if name == "pos_embed":
            vals = fixed_sincos_pos_embed(cfg.hidden, cfg.R)
        else:
            vals = rng.standard_normal(shape) * INIT_STD
        enc = _encode(vals, cfg.dtype)
        blob[off:off + enc.size] = enc
    return blob


def make_latent(cfg: DiTConfig, seed: int = 0) -> np.ndarray:
    """x ~ N(0, 1), float32 [in_ch, latent, latent]."""
    rng = np.random.default_rng([seed, STREAM_LATENT])
    return rng.standard_normal((cfg.in_ch, cfg.latent, cfg.latent)).astype(np.float32)


def make_noise(cfg: DiTConfig, seed: int = 0) -> np.ndarray:
    """z ~ N(0, 1), float32 [in_ch, latent, latent]."""
    rng = np.random.default_rng([seed, STREAM_NOISE])
    return rng.standard_normal((cfg.in_ch, cfg.latent, cfg.latent)).astype(np.float32)


def make_labels(cfg: DiTConfig, seed: int = 0) -> np.ndarray:
    """int32 [cfg_batch]: a class label, then (with guidance) the null label."""
    rng = np.random.default_rng([seed, STREAM_LABELS])
    lab = int(rng.integers(0, cfg.num_classes))
    if cfg.cfg_batch == 1:
        return np.array([lab], dtype=np.int32)
    return np.array([lab, cfg.num_classes], dtype=np.int32)


def make_stale_latent(cfg: DiTConfig, seed: int = 0) -> np.ndarray:
    """float32 [in_ch, latent, latent] ~ N(0, 1), independent of make_latent:
    the sample a model-consistent stale buffer is computed from (its K/V
    under a full-image step), drawn from the stale-buffer stream."""
    rng = np.random.default_rng([seed, STREAM_STALE, 1])
    return rng.standard_normal((cfg.in_ch, cfg.latent, cfg.latent)).astype(np.float32)


def stale_kv_elems(cfg: DiTConfig) -> int:
    return cfg.n_blocks * cfg.cfg_batch * 2 * cfg.n_kv * cfg.hidden


def make_stale_kv(cfg: DiTConfig, seed: int = 0, std: float | None = None) -> np.ndarray:
    """A seeded stale K/V buffer standing in for the other devices' activations.

    Values N(0, std^2) with std = 0.02 * sqrt(H) by default: the spread of a
    linear layer with N(0, 0.02^2) weights applied to unit-variance inputs.
    Returned in the buffer's storage type (float32, or bf16 as uint16 bits),
    flat; its layout is the buffer layout of the step call (the values are
    i.i.d., so the layout does not matter for generation).
    """
    if std is None:
        std = INIT_STD * float(np.sqrt(cfg.hidden))
    rng = np.random.default_rng([seed, STREAM_STALE])
    n = stale_kv_elems(cfg)
    out_dtype = np.float32 if cfg.dtype == "f32" else np.uint16
    out = np.empty(n, dtype=out_dtype)
    chunk = 1 << 24
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        v = (rng.standard_normal(e - s) * std).astype(np.float32)
        out[s:e] = v if cfg.dtype == "f32" else f32_to_bf16_bits(v)
    return out


# ---- convolutional (U-Net) band block --------------------------------------
# Seed streams of its own: parameters, input feature map.
STREAM_UNET_PARAMS = 10
STREAM_UNET_INPUT = 11


def make_unet_params(cfg, seed: int = 0) -> dict:
    """GroupNorm affine (gamma ~ 1 + N(0, 0.02^2), beta ~ N(0, 0.02^2)) fp32,
    conv weight N(0, 0.02^2) as bf16 bits [C_out][3][3][C_in], bias fp32."""
    rng = np.random.default_rng([seed, STREAM_UNET_PARAMS])
    C, Co = cfg.channels, cfg.out_channels
    gamma = (1.0 + rng.standard_normal(C) * INIT_STD).astype(np.float32)
    beta = (rng.standard_normal(C) * INIT_STD).astype(np.float32)
    w = (rng.standard_normal((Co, 3, 3, C)) * INIT_STD).astype(np.float32)
    bias = (rng.standard_normal(Co) * INIT_STD).astype(np.float32)
    return {"gamma": gamma, "beta": beta, "weight_bits": f32_to_bf16_bits(w), "bias": bias}


def make_unet_input(cfg, seed: int = 0) -> np.ndarray:
    """float32 [H][W][C] feature map: N(0, 1) plus a per-channel offset
    N(0, 0.5^2), so the groups' means are not zero."""
    rng = np.random.default_rng([seed, STREAM_UNET_INPUT])
    off = rng.standard_normal(cfg.channels) * 0.5
    x = rng.standard_normal((cfg.height, cfg.width, cfg.channels)) + off
    return x.astype(np.float32)
