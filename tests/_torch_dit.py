"""An independent full-image DiT forward built from torch library routines
(conv2d patch embedding, layer_norm, scaled_dot_product_attention, GELU,
pixel_shuffle), float64 on the CPU.  Used only to pin the oracle's
full-image step; it shares no code with the oracle or the GPU path.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F


def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def torch_dit_eps(hdr, params, x_full, t, labels):
    """eps_theta(x, t) for the whole image, every branch: [B, C_out, Hl, Wl]."""
    P = {k: _t(v) for k, v in params.items()}
    H, heads, L, p, R = hdr["hidden"], hdr["heads"], hdr["n_blocks"], hdr["patch"], hdr["grid"]
    C, Co = hdr["in_ch"], hdr["out_ch"]
    d = H // heads
    x = _t(x_full)[None]                                            # [1, C, Hl, Wl]
    tok = F.conv2d(x, P["x_embedder.weight"].reshape(H, C, p, p), P["x_embedder.bias"],
                   stride=p)                                        # [1, H, R, R]
    tok = tok.flatten(2).transpose(1, 2)[0] + P["pos_embed"]         # [N, H]

    half = hdr["freq_dim"] // 2
    freqs = torch.exp(-math.log(10000.0) * torch.arange(half, dtype=torch.float64) / half)
    arg = float(t) * freqs
    temb = torch.cat([torch.cos(arg), torch.sin(arg)])
    temb = F.linear(F.silu(F.linear(temb, P["t_embedder.fc1.weight"], P["t_embedder.fc1.bias"])),
                    P["t_embedder.fc2.weight"], P["t_embedder.fc2.bias"])
    outs = []
    for lab in labels:
        c = temb + P["y_embedder.table"][int(lab)]
        sc = F.silu(c)
        h = tok.clone()
        for l in range(L):
            pre = f"blocks.{l}."
            mod = F.linear(sc, P[pre + "adaLN.weight"], P[pre + "adaLN.bias"]).chunk(6)
            sh1, sc1, g1, sh2, sc2, g2 = mod
            u = F.layer_norm(h, (H,), eps=1e-6) * (1 + sc1) + sh1
            qkv = F.linear(u, P[pre + "qkv.weight"], P[pre + "qkv.bias"])
            qkv = qkv.reshape(-1, 3, heads, d).permute(1, 2, 0, 3)          # [3, heads, N, d]
            o = F.scaled_dot_product_attention(qkv[0], qkv[1], qkv[2])        # [heads, N, d]
            o = o.permute(1, 0, 2).reshape(-1, H)
            h = h + g1 * F.linear(o, P[pre + "proj.weight"], P[pre + "proj.bias"])
            u = F.layer_norm(h, (H,), eps=1e-6) * (1 + sc2) + sh2
            m = F.gelu(F.linear(u, P[pre + "fc1.weight"], P[pre + "fc1.bias"]), approximate="tanh")
            h = h + g2 * F.linear(m, P[pre + "fc2.weight"], P[pre + "fc2.bias"])
        fsh, fsc = F.linear(sc, P["final.adaLN.weight"], P["final.adaLN.bias"]).chunk(2)
        y = F.linear(F.layer_norm(h, (H,), eps=1e-6) * (1 + fsc) + fsh,
                     P["final.linear.weight"], P["final.linear.bias"])   # [N, p*p*Co] (dy,dx,c)
        # reorder to (c, dy, dx) channels and let pixel_shuffle place them
        y = y.reshape(R, R, p, p, Co).permute(4, 2, 3, 0, 1).reshape(Co * p * p, R, R)
        outs.append(F.pixel_shuffle(y[None], p)[0])
    return torch.stack(outs).numpy()
