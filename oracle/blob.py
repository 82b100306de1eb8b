"""Reader of the weight-blob format (oracle side).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Format: a 256-byte header (magic "ORCHDIT1", u32 version, u32 dtype 0=f32
1=bf16, u32 n_blocks, hidden, heads, mlp_hidden, in_ch, out_ch, patch, grid,
num_classes, freq_dim, n_tensors), then the tensors in a fixed order, each at
the next multiple of 256 bytes, row-major, in the blob dtype.  Linear
weights are [out][in].
"""
from __future__ import annotations

import struct
from typing import Dict

import numpy as np

FIELDS = ("n_blocks", "hidden", "heads", "mlp_hidden", "in_ch", "out_ch", "patch",
          "grid", "num_classes", "freq_dim")


def bf16_to_float(bits: np.ndarray) -> np.ndarray:
    """Exact bfloat16 -> float32 (bf16 is the upper half of a float32)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _shapes(h: Dict[str, int]):
    H, F, L = h["hidden"], h["mlp_hidden"], h["n_blocks"]
    pdim = h["in_ch"] * h["patch"] ** 2
    odim = h["out_ch"] * h["patch"] ** 2
    out = [("x_embedder.weight", (H, pdim)), ("x_embedder.bias", (H,)),
           ("pos_embed", (h["grid"] ** 2, H)),
           ("t_embedder.fc1.weight", (H, h["freq_dim"])), ("t_embedder.fc1.bias", (H,)),
           ("t_embedder.fc2.weight", (H, H)), ("t_embedder.fc2.bias", (H,)),
           ("y_embedder.table", (h["num_classes"] + 1, H))]
    for l in range(L):
        for name, shp in (("adaLN.weight", (6 * H, H)), ("adaLN.bias", (6 * H,)),
                          ("qkv.weight", (3 * H, H)), ("qkv.bias", (3 * H,)),
                          ("proj.weight", (H, H)), ("proj.bias", (H,)),
                          ("fc1.weight", (F, H)), ("fc1.bias", (F,)),
                          ("fc2.weight", (H, F)), ("fc2.bias", (H,))):
            out.append((f"blocks.{l}.{name}", shp))
    out += [("final.adaLN.weight", (2 * H, H)), ("final.adaLN.bias", (2 * H,)),
            ("final.linear.weight", (odim, H)), ("final.linear.bias", (odim,))]
    return out


def read_blob(blob, dtype=np.float64):
    """Parse a blob into (header dict, {name: array in `dtype`})."""
    buf = np.frombuffer(memoryview(blob), dtype=np.uint8)
    magic, version, dcode, *vals = struct.unpack_from("<8sII10II", buf, 0)
    if magic != b"ORCHDIT1" or version != 1:
        raise ValueError("not a version-1 ORCHDIT1 blob")
    hdr = dict(zip(FIELDS, vals[:10]))
    hdr["dtype"] = "f32" if dcode == 0 else "bf16"
    esize = 4 if dcode == 0 else 2
    shapes = _shapes(hdr)
    if vals[10] != len(shapes):
        raise ValueError("tensor count mismatch")
    params = {}
    off = 256
    for name, shp in shapes:
        n = int(np.prod(shp))
        raw = buf[off:off + n * esize]
        if raw.size != n * esize:
            raise ValueError("blob truncated")
        if dcode == 0:
            arr = raw.view(np.float32)
        else:
            arr = bf16_to_float(raw.view(np.uint16))
        params[name] = arr.astype(dtype).reshape(shp)
        off = (off + n * esize + 255) // 256 * 256
    return hdr, params
