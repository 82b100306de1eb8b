"""ctypes binding of liborch.so (argument marshalling only).

Every function here forwards to the C ABI declared in include/orch.h; all
computation happens in the library's HIP kernels.  PyTorch is used only to
hold device memory and to name the current HIP stream.  Importing this
module raises if the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liborch.so")

ORCH_OK, ORCH_EINVAL, ORCH_ENOWEIGHTS, ORCH_EHIP, ORCH_ENOMEM = 0, -1, -2, -3, -4
ORCH_F32, ORCH_BF16 = 0, 1
EPI_STORE, EPI_GELU, EPI_RESIDUAL = 0, 1, 2
DTYPE_CODE = {"f32": ORCH_F32, "bf16": ORCH_BF16}

SYMBOLS = (
    "orch_create", "orch_destroy", "orch_load_dit_weights", "orch_stale_kv_bytes",
    "orch_patch_denoise_step", "orch_scheduler_update", "orch_schedule_coefficients",
    "orch_last_error", "orch_op_layernorm_modulate", "orch_op_linear", "orch_op_qkv_projection",
    "orch_op_attention", "orch_op_conditioning", "orch_op_patch_embed", "orch_op_final_layer",
    "orch_attention_workspace_bytes", "orch_set_kernel_timing", "orch_kernel_times",
    "orch_linear_workspace_bytes",
    "orch_plan_devices", "orch_sample_patch_parallel", "orch_set_work_split",
    "orch_op_attention_noalloc", "orch_speeds_from_profiles", "orch_unet_conv_band",
    "orch_unet_conv_workspace_bytes",
)
KCLASSES = ("conditioning", "patch_embed", "layernorm", "qkv_gemm", "attention", "proj_gemm",
            "fc1_gemm", "fc2_gemm", "final_layer", "update")


class OrchError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"orch error {code}: {msg}")
        self.code = code


class UNetConvShape(C.Structure):
    _fields_ = [("height", C.c_int), ("width", C.c_int), ("channels", C.c_int),
                ("groups", C.c_int), ("out_channels", C.c_int), ("eps", C.c_float)]


class OrchConfig(C.Structure):
    _fields_ = [("n_blocks", C.c_int), ("hidden", C.c_int), ("heads", C.c_int),
                ("mlp_hidden", C.c_int), ("in_ch", C.c_int), ("out_ch", C.c_int),
                ("patch", C.c_int), ("latent", C.c_int), ("num_classes", C.c_int),
                ("freq_dim", C.c_int), ("cfg_batch", C.c_int), ("dtype", C.c_int),
                ("T", C.c_int), ("beta_start", C.c_double), ("beta_end", C.c_double)]


def config_from(cfg) -> OrchConfig:
    """Build the C config from any object with the DiT shape attributes."""
    return OrchConfig(cfg.n_blocks, cfg.hidden, cfg.heads, cfg.mlp_hidden, cfg.in_ch, cfg.out_ch,
                      cfg.patch, cfg.latent, cfg.num_classes, cfg.freq_dim, cfg.cfg_batch,
                      DTYPE_CODE[cfg.dtype], cfg.T, cfg.beta_start, cfg.beta_end)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2509_04719_amd.build`")
    lib = C.CDLL(LIB_PATH)
    vp, i, sz, d, f = C.c_void_p, C.c_int, C.c_size_t, C.c_double, C.c_float
    sig = {
        "orch_create": (i, [C.POINTER(OrchConfig), C.POINTER(vp)]),
        "orch_destroy": (None, [vp]),
        "orch_load_dit_weights": (i, [vp, vp, sz]),
        "orch_stale_kv_bytes": (sz, [vp]),
        "orch_patch_denoise_step": (i, [vp, vp, i, i, i, i, C.POINTER(i), f, vp, i, vp, f, vp, vp,
                                        vp]),
        "orch_scheduler_update": (i, [vp, vp, vp, f, vp, d, d, d, vp, sz, vp]),
        "orch_schedule_coefficients": (i, [C.POINTER(OrchConfig), i, i, d, C.POINTER(d)]),
        "orch_last_error": (C.c_char_p, []),
        "orch_op_layernorm_modulate": (i, [vp, i, i, i, vp, vp, i, vp, i, vp]),
        "orch_op_linear": (i, [vp, i, i, vp, i, vp, i, vp, i, i, vp, vp, sz, i, vp]),
        "orch_linear_workspace_bytes": (sz, [i, i, i, i]),
        "orch_op_qkv_projection": (i, [vp, i, i, i, vp, vp, i, i, vp, vp, sz, i, i, i, vp]),
        "orch_op_attention": (i, [vp, vp, sz, vp, sz, i, i, i, i, i, i, i, vp, vp, sz, i, vp]),
        "orch_attention_workspace_bytes": (sz, [i, i, i, i, i, i]),
        "orch_op_attention_noalloc": (i, [vp, vp, sz, vp, sz, i, i, i, i, i, i, i, vp, i, vp]),
        "orch_set_kernel_timing": (i, [vp, i]),
        "orch_set_work_split": (i, [vp, i]),
        "orch_kernel_times": (i, [vp, C.POINTER(d), C.POINTER(C.c_longlong)]),
        "orch_op_conditioning": (i, [vp, i, C.POINTER(i), vp, vp]),
        "orch_op_patch_embed": (i, [vp, vp, i, i, vp, vp]),
        "orch_op_final_layer": (i, [vp, vp, i, i, vp, vp, vp]),
        "orch_plan_devices": (i, [C.POINTER(d), i, i, i, d, d, i, C.POINTER(i), C.POINTER(i)]),
        "orch_speeds_from_profiles": (i, [i, C.POINTER(i), C.POINTER(i), C.POINTER(d), i,
                                          C.POINTER(d)]),
        "orch_unet_conv_workspace_bytes": (sz, [C.POINTER(UNetConvShape), i]),
        "orch_unet_conv_band": (i, [C.POINTER(UNetConvShape), i, i, vp, vp, vp, vp, vp, vp, vp, i,
                                    vp, vp, sz, vp]),
        "orch_sample_patch_parallel": (i, [vp, vp, i, C.POINTER(i), C.POINTER(i), C.POINTER(i), i, i,
                                           C.POINTER(i), f, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def last_error() -> str:
    return lib.orch_last_error().decode()


def check(rc: int) -> None:
    if rc != ORCH_OK:
        raise OrchError(rc, last_error())


def _ptr(t):
    """Device address of a torch tensor (or None)."""
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def schedule_coefficients(cfg, t: int, t_prev: int, eta: float = 0.0):
    """(a, b, c) of x_prev = a x - b eps + c z, computed by the library (host)."""
    out = (C.c_double * 3)()
    oc = config_from(cfg)
    check(lib.orch_schedule_coefficients(C.byref(oc), t, t_prev, eta, out))
    return out[0], out[1], out[2]


def plan_devices(speeds, m_base, m_warmup, a, b, total_rows):
    """(steps, rows) per device from the library's planner (host only)."""
    n = len(speeds)
    v = (C.c_double * n)(*[float(x) for x in speeds])
    st = (C.c_int * n)()
    rw = (C.c_int * n)()
    check(lib.orch_plan_devices(v, n, m_base, m_warmup, float(a), float(b), total_rows, st, rw))
    return list(st), list(rw)


def speeds_from_profiles(profiles, ref_rows):
    """Effective speeds from per-device [(rows, ms), ...] profiles (host only)."""
    n = len(profiles)
    pts = [pt for prof in profiles for pt in prof]
    npts = (C.c_int * n)(*[len(prof) for prof in profiles])
    rows = (C.c_int * len(pts))(*[int(r) for r, _ in pts])
    ms = (C.c_double * len(pts))(*[float(t) for _, t in pts])
    out = (C.c_double * n)()
    check(lib.orch_speeds_from_profiles(n, npts, rows, ms, int(ref_rows), out))
    return list(out)


class DiTStep:
    """A library context for one DiT config: weights + workspace on the GPU."""

    def __init__(self, cfg, blob=None):
        self.cfg = cfg
        self._c = config_from(cfg)
        h = C.c_void_p()
        check(lib.orch_create(C.byref(self._c), C.byref(h)))
        self.handle = h
        if blob is not None:
            self.load(blob)

    def close(self):
        if getattr(self, "handle", None):
            lib.orch_destroy(self.handle)
            self.handle = None

    def __del__(self):
        self.close()

    def load(self, blob):
        import numpy as np
        b = np.ascontiguousarray(blob, dtype=np.uint8)
        check(lib.orch_load_dit_weights(self.handle, b.ctypes.data_as(C.c_void_p), b.nbytes))

    def stale_kv_bytes(self) -> int:
        return lib.orch_stale_kv_bytes(self.handle)

    def step(self, x_full, row_begin, row_end, t, t_prev, labels, cfg_scale, stale_kv,
             refresh, out_x, out_eps=None, z=None, eta=0.0, stream=None):
        lab = (C.c_int * len(labels))(*[int(v) for v in labels])
        check(lib.orch_patch_denoise_step(self.handle, _ptr(x_full), row_begin, row_end, t, t_prev,
                                          lab, float(cfg_scale), _ptr(stale_kv), int(refresh),
                                          _ptr(z), float(eta), _ptr(out_eps), _ptr(out_x),
                                          _stream(stream)))

    def sample_patch_parallel(self, latent, row_splits, tiers, t_grid, warmup, labels, cfg_scale,
                              kv_a, kv_b, stream=None):
        """Algorithm 1 on virtual devices (bands), in place on `latent`."""
        n = len(tiers)
        sp = (C.c_int * (n + 1))(*[int(v) for v in row_splits])
        tr = (C.c_int * n)(*[int(v) for v in tiers])
        tg = (C.c_int * len(t_grid))(*[int(v) for v in t_grid])
        lab = (C.c_int * len(labels))(*[int(v) for v in labels])
        check(lib.orch_sample_patch_parallel(self.handle, _ptr(latent), n, sp, tr, tg,
                                             len(t_grid) - 1, int(warmup), lab, float(cfg_scale),
                                             _ptr(kv_a), _ptr(kv_b), _stream(stream)))

    def set_work_split(self, enable: bool):
        check(lib.orch_set_work_split(self.handle, int(enable)))

    def set_kernel_timing(self, enable: bool):
        check(lib.orch_set_kernel_timing(self.handle, int(enable)))

    def kernel_times(self):
        """{class: (total_ms, launches)} since the last call (synchronises)."""
        ms = (C.c_double * len(KCLASSES))()
        n = (C.c_longlong * len(KCLASSES))()
        check(lib.orch_kernel_times(self.handle, ms, n))
        return {k: (ms[i], n[i]) for i, k in enumerate(KCLASSES)}

    def conditioning(self, t, labels, out, stream=None):
        lab = (C.c_int * len(labels))(*[int(v) for v in labels])
        check(lib.orch_op_conditioning(self.handle, t, lab, _ptr(out), _stream(stream)))

    def patch_embed(self, x_full, row_begin, row_end, out, stream=None):
        check(lib.orch_op_patch_embed(self.handle, _ptr(x_full), row_begin, row_end, _ptr(out),
                                      _stream(stream)))

    def final_layer(self, h, row_begin, row_end, mod, out_eps, stream=None):
        check(lib.orch_op_final_layer(self.handle, _ptr(h), row_begin, row_end, _ptr(mod),
                                      _ptr(out_eps), _stream(stream)))


def scheduler_update(x, eps_cond, eps_uncond, cfg_scale, z, a, b, c, out, stream=None):
    check(lib.orch_scheduler_update(_ptr(x), _ptr(eps_cond), _ptr(eps_uncond), float(cfg_scale),
                                    _ptr(z), a, b, c, _ptr(out), out.numel(), _stream(stream)))


def layernorm_modulate(x, rows, hidden, rows_per_batch, shift, scale, mod_stride, out, dtype,
                       stream=None):
    check(lib.orch_op_layernorm_modulate(_ptr(x), rows, hidden, rows_per_batch, _ptr(shift),
                                         _ptr(scale), mod_stride, _ptr(out), dtype,
                                         _stream(stream)))


def linear(A, M, K, W, N, bias, epilogue, gate, gate_stride, rows_per_batch, out, dtype,
           stream=None, workspace=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    check(lib.orch_op_linear(_ptr(A), M, K, _ptr(W), N, _ptr(bias), epilogue, _ptr(gate),
                             gate_stride, rows_per_batch, _ptr(out), _ptr(workspace), ws_bytes,
                             dtype, _stream(stream)))


def linear_workspace_bytes(M, N, K, dtype) -> int:
    return lib.orch_linear_workspace_bytes(M, N, K, dtype)


def qkv_projection(A, B, n_tok, K, W, bias, hidden, heads, q_out, kv_out, kv_branch_stride,
                   kv_tokens, tok_offset, dtype, stream=None):
    check(lib.orch_op_qkv_projection(_ptr(A), B, n_tok, K, _ptr(W), _ptr(bias), hidden, heads,
                                     _ptr(q_out), _ptr(kv_out), kv_branch_stride, kv_tokens,
                                     tok_offset, dtype, _stream(stream)))


def attention_workspace_bytes(B, heads, n_q, n_kv, head_dim, dtype) -> int:
    return lib.orch_attention_workspace_bytes(B, heads, n_q, n_kv, head_dim, dtype)


def attention(q, kv_stale, stale_bs, kv_fresh, fresh_bs, fresh_begin, n_fresh, B, heads, n_q,
              n_kv, head_dim, out, dtype, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    check(lib.orch_op_attention(_ptr(q), _ptr(kv_stale), stale_bs, _ptr(kv_fresh), fresh_bs,
                                fresh_begin, n_fresh, B, heads, n_q, n_kv, head_dim, _ptr(out),
                                _ptr(workspace), ws_bytes, dtype, _stream(stream)))


def unet_shape(cfg, eps: float = 1e-5) -> UNetConvShape:
    return UNetConvShape(cfg.height, cfg.width, cfg.channels, cfg.groups, cfg.out_channels, eps)


def unet_conv_workspace_bytes(shape: UNetConvShape, band_rows: int) -> int:
    return lib.orch_unet_conv_workspace_bytes(C.byref(shape), band_rows)


def unet_conv_band(shape: UNetConvShape, row_begin, row_end, x_band, gamma, beta, weight, bias,
                   stale_act, stale_sums, refresh, out, workspace, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size()
    check(lib.orch_unet_conv_band(C.byref(shape), row_begin, row_end, _ptr(x_band), _ptr(gamma),
                                  _ptr(beta), _ptr(weight), _ptr(bias), _ptr(stale_act),
                                  _ptr(stale_sums), int(refresh), _ptr(out), _ptr(workspace),
                                  ws_bytes, _stream(stream)))
