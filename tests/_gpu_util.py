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


def max_row_rel_l2(got, ref, p: int) -> float:
    """Largest relative L2 error over token rows.  got/ref [..., C, n*p, W]
    (latent rows of n token rows, p latent rows each): each leading index and
    token row is one group of C*p*W values."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    *lead, C, rows, W = ref.shape
    n = rows // p
    g = got.reshape(-1, C, n, p, W).transpose(0, 2, 1, 3, 4).reshape(-1, C * p * W)
    r = ref.reshape(-1, C, n, p, W).transpose(0, 2, 1, 3, 4).reshape(-1, C * p * W)
    num = np.linalg.norm(g - r, axis=1)
    den = np.maximum(np.linalg.norm(r, axis=1), 1e-300)
    return float((num / den).max())


def model_kv_buffer(hdr, params, cfg, t: int, labels, seed: int = 0, dtype=np.float32):
    """The buffer Algorithm 1's synchronous warm-up leaves: every token's K/V
    of a full-image oracle step at timestep t on an independent seeded
    latent, in the buffer layout and the config's storage type."""
    from oracle import dit
    xs = generate.make_stale_latent(cfg, seed)
    r = dit.denoiser_band(hdr, params, xs, 0, cfg.R, t, labels, None, dtype=dtype, keep_kv=True)
    buf = dit.full_kv_buffer(hdr, r["kv"]).astype(np.float32)
    return buf if cfg.dtype == "f32" else generate.f32_to_bf16_bits(buf)
