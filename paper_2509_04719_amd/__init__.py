"""MI355X (gfx950) patch-parallel DiT denoising step.

One device's share of a patch-parallel denoising step (Algorithm 1 of the
paper): a DiT denoiser on an elastic band of latent token rows whose
attention reads fresh K/V for the band and stale, buffered K/V for every
other row, then classifier-free guidance and the scheduler update of §I with
Lemma 1's coefficient.  The work runs in hand-written HIP kernels behind the
C ABI of include/orch.h (liborch.so); this package holds the kernels'
sources (csrc/), the in-tree build, a ctypes binding and the host-side
sampler schedule.
"""
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))


def lib():
    """The ctypes binding; raises ImportError if liborch.so is not built."""
    from . import _lib
    return _lib
