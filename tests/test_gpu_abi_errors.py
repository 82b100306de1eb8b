"""Argument validation of the C ABI: every bad call returns the documented
status, names the problem in orch_last_error(), and writes nothing."""
import ctypes as C

import numpy as np
import pytest
import torch

from seeded_inputs import configs, generate
from tests._gpu_util import DEV, empty, to_dev

pytestmark = pytest.mark.gpu

CFG = configs.TINY


@pytest.fixture(scope="module")
def setup(orch_lib):
    blob = generate.make_weight_blob(CFG, 0)
    ctx = orch_lib.DiTStep(CFG, blob)
    x = to_dev(generate.make_latent(CFG, 0))
    kv = torch.zeros(ctx.stale_kv_bytes() // 4, dtype=torch.float32, device=DEV)
    yield ctx, blob, x, kv
    ctx.close()


def _step(orch_lib, ctx, x, kv, out, rb=0, re=4, t=500, tp=250, labels=(3,), refresh=0,
          eps=None, z=None, eta=0.0):
    lab = (C.c_int * len(labels))(*labels)
    return orch_lib.lib.orch_patch_denoise_step(
        ctx.handle, C.c_void_p(x.data_ptr()) if x is not None else None, rb, re, t, tp, lab, 1.5,
        C.c_void_p(kv.data_ptr()) if kv is not None else None, refresh,
        C.c_void_p(z.data_ptr()) if z is not None else None, eta,
        C.c_void_p(eps.data_ptr()) if eps is not None else None,
        C.c_void_p(out.data_ptr()) if out is not None else None,
        C.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("kw,word", [
    (dict(rb=-1), "band"), (dict(rb=4, re=4), "band"), (dict(re=9), "band"),
    (dict(t=1000), "t_prev"), (dict(t=500, tp=500), "t_prev"), (dict(tp=-2), "t_prev"),
    (dict(labels=(11,)), "label"), (dict(labels=(-1,)), "label"),
    (dict(eta=0.5), "needs z"), (dict(eta=float("nan")), "eta"),
])
def test_step_rejects_and_writes_nothing(orch_lib, setup, kw, word):
    ctx, _, x, kv = setup
    out = torch.full((CFG.in_ch, 8, CFG.latent), 7.0, device=DEV)
    kv_before = kv.clone()
    rc = _step(orch_lib, ctx, x, kv, out, **kw)
    torch.cuda.synchronize()
    assert rc == orch_lib.ORCH_EINVAL
    assert word in orch_lib.last_error()
    assert torch.all(out == 7.0)
    assert torch.equal(kv, kv_before)


def test_null_and_overlap(orch_lib, setup):
    ctx, _, x, kv = setup
    out = empty((CFG.in_ch, 8, CFG.latent))
    assert _step(orch_lib, ctx, None, kv, out) == orch_lib.ORCH_EINVAL
    assert _step(orch_lib, ctx, x, None, out) == orch_lib.ORCH_EINVAL
    assert _step(orch_lib, ctx, x, kv, None) == orch_lib.ORCH_EINVAL
    # inside x_full but not exactly its band
    assert _step(orch_lib, ctx, x, kv, x.view(-1)[4:]) == orch_lib.ORCH_EINVAL
    assert "overlap" in orch_lib.last_error()
    assert _step(orch_lib, ctx, x, kv, x.view(-1)[CFG.latent * 2:], rb=0) == orch_lib.ORCH_EINVAL
    assert "overlap" in orch_lib.last_error()
    assert _step(orch_lib, ctx, x, kv, kv) == orch_lib.ORCH_EINVAL
    ok = _step(orch_lib, ctx, x, kv, out)
    assert ok == orch_lib.ORCH_OK, orch_lib.last_error()


def test_not_loaded_and_bad_blob(orch_lib, setup):
    _, blob, x, kv = setup
    ctx2 = orch_lib.DiTStep(CFG)
    out = empty((CFG.in_ch, 8, CFG.latent))
    assert _step(orch_lib, ctx2, x, kv, out) == orch_lib.ORCH_ENOWEIGHTS
    bad = blob.copy()
    bad[0] = ord("X")
    with pytest.raises(orch_lib.OrchError) as e:
        ctx2.load(bad)
    assert e.value.code == orch_lib.ORCH_EINVAL and "magic" in str(e.value)
    other = generate.make_weight_blob(configs.scaled(CFG, n_blocks=3), 0)
    with pytest.raises(orch_lib.OrchError) as e:
        ctx2.load(other)
    assert "n_blocks" in str(e.value)
    with pytest.raises(orch_lib.OrchError):
        ctx2.load(blob[:1000])
    ctx2.load(blob)
    assert _step(orch_lib, ctx2, x, kv, out) == orch_lib.ORCH_OK
    ctx2.close()


def test_op_argument_checks(orch_lib):
    a = empty((4, 128))
    with pytest.raises(orch_lib.OrchError):
        orch_lib.layernorm_modulate(a, 4, 100, 4, a, a, 128, a, 0)      # hidden % 128
    with pytest.raises(orch_lib.OrchError):
        orch_lib.linear(a, 4, 128, a, 4, a, 7, None, 0, 1, a, 0)        # bad epilogue
    with pytest.raises(orch_lib.OrchError):
        orch_lib.linear(a, 4, 128, a, 4, a, 2, None, 0, 1, a, 0)        # residual without gate
    with pytest.raises(orch_lib.OrchError):
        orch_lib.attention(a, a, 16, None, 0, 0, 4, 1, 1, 4, 64, 32, a, 0)  # fresh without pointer
    with pytest.raises(orch_lib.OrchError):
        orch_lib.scheduler_update(a, a, None, 1.5, None, 1.0, 0.5, 0.3, a)  # c != 0 without z


def test_kernel_timing_counts(orch_lib, setup):
    """Per-kernel timing records every launch of the step by class and does
    not change its result."""
    ctx, _, x, kv = setup
    out0 = empty((CFG.in_ch, 8, CFG.latent))
    out1 = empty((CFG.in_ch, 8, CFG.latent))
    assert _step(orch_lib, ctx, x, kv, out0) == orch_lib.ORCH_OK
    ctx.set_kernel_timing(True)
    for _ in range(3):
        assert _step(orch_lib, ctx, x, kv, out1) == orch_lib.ORCH_OK
    t = ctx.kernel_times()
    ctx.set_kernel_timing(False)
    L = CFG.n_blocks
    want = {"conditioning": 1, "patch_embed": 1, "layernorm": 2 * L + 1, "qkv_gemm": L,
            "attention": L, "proj_gemm": L, "fc1_gemm": L, "fc2_gemm": L, "final_layer": 1,
            "update": 1}
    for k, n in want.items():
        assert t[k][1] == 3 * n, (k, t[k])
        assert t[k][0] > 0.0
    torch.cuda.synchronize()
    assert torch.equal(out0, out1)
    assert all(v == (0.0, 0) for v in ctx.kernel_times().values())


@pytest.mark.parametrize("rb,re", [(0, 4), (3, 8), (2, 5)])
def test_in_place_band_update(orch_lib, setup, rb, re):
    """out_x_patch == the band of x_full: the band is updated in place (in
    x_full's layout), bitwise as the separate output, other rows untouched."""
    ctx, _, x, kv = setup
    p = CFG.patch
    out = empty((CFG.in_ch, (re - rb) * p, CFG.latent))
    assert _step(orch_lib, ctx, x, kv, out, rb=rb, re=re) == orch_lib.ORCH_OK
    xi = x.clone()
    band = xi[:, rb * p:re * p]                     # a view starting at the band of xi
    assert band.data_ptr() == xi.data_ptr() + rb * p * CFG.latent * 4
    assert _step(orch_lib, ctx, xi, kv, band, rb=rb, re=re) == orch_lib.ORCH_OK, \
        orch_lib.last_error()
    torch.cuda.synchronize()
    assert torch.equal(xi[:, rb * p:re * p], out)
    assert torch.equal(xi[:, :rb * p], x[:, :rb * p])
    assert torch.equal(xi[:, re * p:], x[:, re * p:])
