"""Workload shapes for the patch-parallel DiT denoising step.

This module holds shapes, seeds and sampler settings only: no arithmetic of
the method.  Both the CPU oracle and the GPU path read their inputs through
``seeded_inputs``; neither imports the other.

Shapes follow the DiT family (a transformer denoiser over p x p latent
patches) that the paper cites as the transformer alternative to U-Nets
(§I, §II-B).  Five workloads, from a tiny fp32 model to DiT-XL/2 at 2048px.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class DiTConfig:
    name: str
    n_blocks: int          # L
    hidden: int            # H
    heads: int
    mlp_hidden: int        # F = 4H
    latent: int            # latent side (latent_h == latent_w)
    num_classes: int       # the null (unconditional) label is index num_classes
    cfg_batch: int         # 1: no guidance; 2: (cond, null) classifier-free guidance
    dtype: str             # "f32" or "bf16": weights, activations and the stale K/V buffer
    steps: int             # DDIM steps M over the T-step DDPM grid
    in_ch: int = 4
    out_ch: int = 4
    patch: int = 2
    freq_dim: int = 256
    T: int = 1000
    beta_start: float = 1e-4
    beta_end: float = 2e-2
    cfg_scale: float = 1.5
    warmup: int = 0        # M_warmup of the tiered schedule (0: plain schedule)
    tiered: bool = False   # slow-tier schedule: stride 2 after the warm-up
    band_rows: Tuple[int, ...] = ()    # default band sizes (token rows)
    share_labels: Tuple[str, ...] = ()

    @property
    def R(self) -> int:
        """Token rows (= token columns) of the latent grid."""
        return self.latent // self.patch

    @property
    def n_kv(self) -> int:
        return self.R * self.R

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def patch_dim(self) -> int:
        return self.in_ch * self.patch * self.patch

    @property
    def out_patch_dim(self) -> int:
        return self.out_ch * self.patch * self.patch

    def n_q(self, rows: int) -> int:
        return rows * self.R


def rows_for_share(share: float, R: int) -> int:
    """Token rows of an elastic band holding `share` of the R rows:
    round half up, at least one row."""
    r = int(share * R + 0.5)
    return max(1, min(R, r))


TINY = DiTConfig(
    name="tiny", n_blocks=2, hidden=128, heads=4, mlp_hidden=512, latent=16,
    num_classes=10, cfg_batch=1, dtype="f32", steps=4,
    band_rows=(4,), share_labels=("rows 0-3",))

DIT_S2_256 = DiTConfig(
    name="dit_s2_256", n_blocks=12, hidden=384, heads=6, mlp_hidden=1536, latent=32,
    num_classes=1000, cfg_batch=1, dtype="bf16", steps=20,
    band_rows=(rows_for_share(0.40, 16),), share_labels=("40%",))

DIT_XL2_512 = DiTConfig(
    name="dit_xl2_512", n_blocks=28, hidden=1152, heads=16, mlp_hidden=4608, latent=64,
    num_classes=1000, cfg_batch=2, dtype="bf16", steps=50,
    band_rows=(12,), share_labels=("12/32 rows",))

DIT_XL2_1024 = DiTConfig(
    name="dit_xl2_1024", n_blocks=28, hidden=1152, heads=16, mlp_hidden=4608, latent=128,
    num_classes=1000, cfg_batch=2, dtype="bf16", steps=50,
    band_rows=tuple(rows_for_share(s, 64) for s in (0.10, 0.25, 0.40, 0.65, 1.00)),
    share_labels=("10%", "25%", "40%", "65%", "100%"))

DIT_XL2_2048 = DiTConfig(
    name="dit_xl2_2048", n_blocks=28, hidden=1152, heads=16, mlp_hidden=4608, latent=256,
    num_classes=1000, cfg_batch=2, dtype="bf16", steps=50, warmup=10, tiered=True,
    band_rows=tuple(rows_for_share(s, 128) for s in (1 / 8, 3 / 8, 5 / 8)),
    share_labels=("1/8", "3/8", "5/8"))

ALL_CONFIGS = (TINY, DIT_S2_256, DIT_XL2_512, DIT_XL2_1024, DIT_XL2_2048)
BY_NAME = {c.name: c for c in ALL_CONFIGS}

# Seed streams: numpy.random.default_rng([seed, stream]).
STREAM_WEIGHTS = 0
STREAM_LATENT = 1
STREAM_NOISE = 2
STREAM_LABELS = 3
STREAM_STALE = 4


def get(name: str) -> DiTConfig:
    return BY_NAME[name]


def scaled(cfg: DiTConfig, **changes) -> DiTConfig:
    """A copy with some fields changed (used for small parity variants)."""
    return dataclasses.replace(cfg, **changes)


def headline_timestep_pair(cfg: DiTConfig) -> Tuple[int, int]:
    """(t, t_prev) of the first step after a 10-step warm-up on the uniform
    grid: 780 -> 760 at M = 50, 780 -> 740 on the stride-2 tier."""
    step = cfg.T // cfg.steps
    m = 10
    t = (cfg.steps - 1 - m) * step
    stride = 2 if cfg.tiered else 1
    t_prev = t - stride * step
    return t, (t_prev if t_prev >= 0 else -1)


def describe(cfg: DiTConfig, rows: Optional[int] = None) -> dict:
    d = {"workload": cfg.name, "blocks": cfg.n_blocks, "hidden": cfg.hidden,
         "heads": cfg.heads, "latent": [cfg.in_ch, cfg.latent, cfg.latent],
         "tokens": cfg.n_kv, "cfg_batch": cfg.cfg_batch}
    if rows is not None:
        d["band_rows"] = rows
        d["n_q"] = cfg.n_q(rows)
    return d


# ---- convolutional (U-Net) band block --------------------------------------

@dataclasses.dataclass(frozen=True)
class UNetConvConfig:
    """GroupNorm -> SiLU -> 3x3 convolution on an H x W feature map with C
    channels (the first half of a U-Net ResNet block)."""
    name: str
    height: int
    width: int
    channels: int
    groups: int
    out_channels: int
    band_rows: Tuple[int, ...] = ()
    share_labels: Tuple[str, ...] = ()


UNET_TINY = UNetConvConfig(name="unet_tiny", height=16, width=16, channels=64, groups=8,
                           out_channels=64, band_rows=(5,), share_labels=("5/16 rows",))

# The first stage of an SDXL-sized U-Net at 1024px: a 128 x 128 latent with
# 320 channels in 32 groups.  The evaluation splits the latent into 32 patch
# units (4 rows each); 18:14 units is its first two-GPU assignment.
UNET_SDXL_1024 = UNetConvConfig(name="unet_sdxl_1024_stage1", height=128, width=128,
                                channels=320, groups=32, out_channels=320,
                                band_rows=(16, 56, 72), share_labels=("1/8", "14/32", "18/32"))

# The deeper stages of the same U-Net at 1024px: 64 x 64 with 640 channels
# and 32 x 32 with 1280 channels, 32 groups each; bands at the same shares of
# the rows (1/8 in the interior, 14/32 at the head, 18/32 at the tail).
UNET_SDXL_1024_S2 = UNetConvConfig(name="unet_sdxl_1024_stage2", height=64, width=64,
                                   channels=640, groups=32, out_channels=640,
                                   band_rows=(8, 28, 36), share_labels=("1/8", "14/32", "18/32"))
UNET_SDXL_1024_S3 = UNetConvConfig(name="unet_sdxl_1024_stage3", height=32, width=32,
                                   channels=1280, groups=32, out_channels=1280,
                                   band_rows=(4, 14, 18), share_labels=("1/8", "14/32", "18/32"))

# A map of 120 x 120 pixels (14400 in all rows, 3120 in a 26-row band: both
# end in a partial 128-pixel tile), 192 -> 320 channels: the convolution takes
# 160-channel tiles for all rows (one round of workgroups) and for the 26-row
# band (its 27 k-tiles split three ways).
UNET_RAGGED_320 = UNetConvConfig(name="unet_ragged_320", height=120, width=120, channels=192, groups=8,
                                 out_channels=320, band_rows=(120, 26), share_labels=("all rows", "26 rows"))

UNET_CONFIGS = (UNET_TINY, UNET_SDXL_1024, UNET_SDXL_1024_S2, UNET_SDXL_1024_S3, UNET_RAGGED_320)
