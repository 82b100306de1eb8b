"""The attention entry point that allocates nothing: its output equals the
workspace entry point's on the same inputs (same kernels, same work plan),
bit for bit, on two calls in a row -- the second with a smaller band -- both
of which cut query tiles and so go through the static scratch."""
import ctypes as C

import numpy as np
import pytest
import torch

from seeded_inputs import generate
from tests._gpu_util import DEV

pytestmark = pytest.mark.gpu

BF16 = 1
HEADS, D, N_KV = 16, 72, 4096        # DiT-XL/2 at 1024px
H = HEADS * D


def _bf16(rng, shape, std):
    bits = generate.f32_to_bf16_bits((rng.standard_normal(shape) * std).astype(np.float32))
    return torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)


def _case(orch_lib, n_q, fresh_begin, seed):
    B = 2
    rng = np.random.default_rng([seed, 11])
    q = _bf16(rng, (B, HEADS, n_q, D), 1.0)
    stale = _bf16(rng, (B, 2 * N_KV * H), 0.02 * np.sqrt(H))
    fresh = _bf16(rng, (B, 2 * n_q * H), 0.02 * np.sqrt(H))
    need = orch_lib.attention_workspace_bytes(B, HEADS, n_q, N_KV, D, BF16)
    assert need > 0                                  # the shape cuts query tiles
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    ref = torch.empty((B, n_q, H), dtype=torch.bfloat16, device=DEV)
    orch_lib.attention(q, stale, 2 * N_KV * H, fresh, 2 * n_q * H, fresh_begin, n_q, B, HEADS,
                       n_q, N_KV, D, ref, BF16, workspace=ws)
    got = torch.full((B, n_q, H), float("nan"), dtype=torch.bfloat16, device=DEV)
    s = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = orch_lib.lib.orch_op_attention_noalloc(
        C.c_void_p(q.data_ptr()), C.c_void_p(stale.data_ptr()), 2 * N_KV * H,
        C.c_void_p(fresh.data_ptr()), 2 * n_q * H, fresh_begin, n_q, B, HEADS, n_q, N_KV, D,
        C.c_void_p(got.data_ptr()), BF16, s)
    assert rc == orch_lib.ORCH_OK, orch_lib.last_error()
    torch.cuda.synchronize()
    assert not torch.isnan(got.float()).any()
    assert torch.equal(got, ref)


def test_no_alloc_attention_matches_workspace_entry_point(orch_lib):
    print("\n[no-alloc attention: 1280 queries, then 384]", flush=True)
    _case(orch_lib, 1280, 22 * 64, 0)     # 20-row band of a 64-row grid
    _case(orch_lib, 384, 0, 1)            # 6-row band: smaller, reuses the scratch


def test_no_alloc_attention_rejects_bad_shape(orch_lib):
    rc = orch_lib.lib.orch_op_attention_noalloc(None, None, 0, None, 0, 0, 0, 1, 1, 1, 64, 72,
                                                None, BF16, None)
    assert rc == orch_lib.ORCH_EINVAL and "NULL" in orch_lib.last_error()
