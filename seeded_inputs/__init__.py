"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds workload shapes and random-input generators only; it computes no part
of the denoising step.
"""
from . import configs, generate  # noqa: F401
from .configs import ALL_CONFIGS, BY_NAME, DiTConfig, get, rows_for_share  # noqa: F401
