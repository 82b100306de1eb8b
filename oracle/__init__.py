"""CPU oracle for one device's patch-parallel denoising step.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
numpy implementation of what the GPU path computes, used to check it.  Only
the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never does, and it imports nothing from the
product package.  It shares no code with the GPU path: its own blob reader,
schedule table, sinusoid, GELU, LayerNorm and attention.

Arithmetic is float64 unless a caller passes ``dtype=np.float32`` (used only
to bound the runtime of the largest workloads).

Modules:
  schedule -- noise schedule, DDIM / DPM-Solver-1 coefficients (Lemma 1 and
              the update of §I), timestep grids, the tiered step schedule
              (Algorithm 1, Eq. (2)).
  blob     -- reader of the weight-blob format.
  dit      -- the DiT denoiser on an elastic band of token rows with stale
              K/V for the other rows (§II-B, Algorithm 1), classifier-free
              guidance, and the scheduler update.
  allocator -- device planning: Eq. (2) tiers, Eq. (3) patch mending in
              whole rows, effective speeds from step-time profiles (§V-A).
  sampler  -- full-image and patch-parallel samplers (Algorithm 1 on virtual
              devices).
  unet     -- a U-Net block (GroupNorm -> SiLU -> conv3x3) on a band of rows
              with stale halo rows and stale group statistics (§II-B).

Parity status: the scheduler, attention, LayerNorm, GELU, sinusoid, patch
embedding and unpatchify are pinned by the CPU tests; the DiT block as a
whole is pinned against an independent torch-module DiT on the full image
and by the invariants of the band step (all rows, stitching, locality,
degenerate gates); the U-Net block against torch's GroupNorm and conv2d and
by the same invariants; the planner by the paper's tables.
"""
