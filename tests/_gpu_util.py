"""Helpers of the GPU tests: moving seeded numpy inputs to the device and
comparing results.  Expected values always come from the oracle."""
import numpy as np
import torch

from seeded_inputs import generate

DEV = "cuda:0"


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def to_dev(a: np.ndarray, dtype: str = "f32") -> torch.Tensor:
    """float data -> device tensor of the config dtype (bf16 by RNE)."""
    a = np.ascontiguousarray(a)
    if dtype == "f32":
        return torch.from_numpy(a.astype(np.float32)).to(DEV)
    bits = generate.f32_to_bf16_bits(a.astype(np.float32))
    return torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)


def bits_to_dev(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bits (or float32) -> device tensor."""
    if bits.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.float32)).to(DEV)


def rounded(a: np.ndarray, dtype: str) -> np.ndarray:
    """The float64 values a device tensor of `dtype` holds for `a`."""
    if dtype == "f32":
        return a.astype(np.float32).astype(np.float64)
    return generate.bf16_bits_to_f32(generate.f32_to_bf16_bits(a.astype(np.float32))).astype(np.float64)


def to_host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy().astype(np.float64)


def empty(shape, dtype: str = "f32") -> torch.Tensor:
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    return torch.empty(shape, dtype=td, device=DEV)


def code(dtype: str) -> int:
    return 0 if dtype == "f32" else 1
