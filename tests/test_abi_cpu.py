"""The C ABI library loads, exports every declared entry point, and its
host-side logic (scheduler coefficients, step schedules) agrees with the
oracle.  No device work: runs without a GPU."""
import os
import re

import numpy as np
import pytest

from oracle import schedule as osched
from paper_2509_04719_amd import schedule as psched
from seeded_inputs import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "orch.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(orch_[a-z_]+)\s*\(", src)))


def test_header_declares_expected_symbols(orch_lib):
    assert _declared_functions() == sorted(orch_lib.SYMBOLS)


def test_library_exports_every_declared_symbol(orch_lib):
    names = _declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(orch_lib.lib, n), n
    out = os.popen(f"nm -D --defined-only {orch_lib.LIB_PATH}").read()
    exported = set(re.findall(r"\bT (orch_\w+)", out))
    assert set(names) <= exported


@pytest.mark.parametrize("pair", osched.step_pairs(1000, 50) + osched.step_pairs(1000, 4)
                         + [(780, 740), (40, -1), (999, 998)])
@pytest.mark.parametrize("eta", [0.0, 0.5, 1.0])
def test_library_schedule_coefficients_match_oracle(orch_lib, pair, eta):
    t, tp = pair
    a, b, c = orch_lib.schedule_coefficients(configs.DIT_XL2_1024, t, tp, eta)
    A, B, Cc = osched.ddim_coefficients(osched.alpha_bar(), t, tp, eta)
    assert a == pytest.approx(A, rel=1e-12)
    assert b == pytest.approx(B, rel=1e-10, abs=1e-14)
    assert c == pytest.approx(Cc, rel=1e-10, abs=1e-14)


@pytest.mark.parametrize("t,tp", [(1000, 500), (-1, -1), (500, 500), (500, 600), (10, -2)])
def test_library_schedule_rejects_bad_pairs(orch_lib, t, tp):
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.schedule_coefficients(configs.TINY, t, tp)
    assert e.value.code == orch_lib.ORCH_EINVAL
    assert "t_prev" in orch_lib.last_error()


def test_product_schedules_match_oracle():
    for M in (4, 20, 50):
        ps = psched.plain_schedule(1000, M)
        assert [(s.t, s.t_prev) for s in ps] == osched.step_pairs(1000, M)
    ts = psched.tiered_schedule(1000, 50, 10)
    assert [(s.m, s.t, s.t_prev, s.refresh) for s in ts] == osched.tiered_schedule(1000, 50, 10)
    assert len(ts) == 30


def test_band_rows_rounding():
    assert [psched.band_rows(s, 64) for s in (0.10, 0.25, 0.40, 0.65, 1.0)] == [6, 16, 26, 42, 64]
    assert [psched.band_rows(s, 128) for s in (1 / 8, 3 / 8, 5 / 8)] == [16, 48, 80]
    assert psched.band_rows(0.40, 16) == 6
    assert configs.DIT_XL2_1024.band_rows == (6, 16, 26, 42, 64)


def test_create_rejects_bad_config_without_gpu_work(orch_lib):
    import ctypes as C
    bad = orch_lib.config_from(configs.scaled(configs.TINY, heads=3))
    h = C.c_void_p()
    rc = orch_lib.lib.orch_create(C.byref(bad), C.byref(h))
    assert rc == orch_lib.ORCH_EINVAL and not h.value
    assert "heads" in orch_lib.last_error()


# ---- device planner (host only: Eq. (2), Eq. (3)) ------------------------

from oracle import allocator as oal  # noqa: E402


def test_library_plan_matches_oracle_exactly(orch_lib):
    rng = np.random.default_rng(7)
    for trial in range(300):
        n = int(rng.integers(1, 9))
        v = list(rng.uniform(0.05, 1.0, n))
        a = float(rng.uniform(0.5, 0.9))
        b = float(rng.uniform(0.05, a - 0.01))
        mb = int(rng.integers(2, 120))
        mw = int(rng.integers(0, mb + 1))
        rows = int(rng.integers(1, 257))
        got = orch_lib.plan_devices(v, mb, mw, a, b, rows)
        want = oal.plan(v, mb, mw, a, b, rows)
        assert got == (want[0], want[1]), (trial, v, a, b, mb, mw, rows)


def test_library_plan_reproduces_quality_tables(orch_lib):
    # two GPUs, 32 units, M_base 100, M_warmup 4, v = 1 - occupancy
    assert orch_lib.plan_devices([1.0, 0.8], 100, 4, 0.75, 0.25, 32) == ([100, 100], [18, 14])
    assert orch_lib.plan_devices([1.0, 0.6], 100, 4, 0.75, 0.25, 32) == ([100, 52], [15, 17])
    assert orch_lib.plan_devices([0.65, 0.55], 100, 4, 0.75, 0.25, 32) == ([100, 100], [17, 15])
    assert orch_lib.plan_devices([0.7, 0.5], 100, 4, 0.75, 0.25, 32) == ([100, 52], [13, 19])
    assert orch_lib.plan_devices([1.0, 0.5], 50, 4, 0.75, 0.25, 32)[0] == [50, 27]
    # Table IV's warm-up of 25 at M_base 100: 25 single steps + 38 double
    assert orch_lib.plan_devices([1.0, 0.5], 100, 25, 0.75, 0.25, 32)[0] == [100, 63]
    # a device whose share rounds to no rows runs no steps
    assert orch_lib.plan_devices([1.0, 1.0, 0.3], 50, 4, 0.75, 0.25, 2) == ([50, 50, 0], [1, 1, 0])


@pytest.mark.parametrize("args,word", [
    (([1.0, -0.5], 50, 4, 0.75, 0.25, 32), "speeds"),
    (([1.0], 50, 60, 0.75, 0.25, 32), "m_warmup"),
    (([1.0], 50, 4, 0.25, 0.75, 32), "0 < b < a < 1"),
    (([1.0], 50, 4, 0.75, 0.25, 0), "total_rows"),
])
def test_library_plan_rejects_bad_arguments(orch_lib, args, word):
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.plan_devices(*args)
    assert e.value.code == orch_lib.ORCH_EINVAL and word in orch_lib.last_error()


@pytest.mark.parametrize("n_q,n_kv,d,want", [
    # DiT-XL/2 1024px, 25% band: 256 query tiles of 64 key tiles on 512
    # workgroups -> 32 units each, every tile cut: 2 * 512 * 128 parts of
    # 72 bf16 + (max, sum)
    (1024, 4096, 72, 2 * 512 * 128 * (72 * 2 + 8)),
    # 20-row band: 320 tiles -> 40 units each (512 workgroups)
    (1280, 4096, 72, 2 * 512 * 128 * (72 * 2 + 8)),
    # 65% band: 672 tiles (two rounds of whole tiles) -> 84 units each
    (2688, 4096, 72, 2 * 512 * 128 * (72 * 2 + 8)),
    (1664, 4096, 72, 0),          # 40% band: 52 units cut against 64 whole, under 12 saved
    (2048, 4096, 72, 0),          # 512 tiles: one whole tile per workgroup
    (4096, 4096, 72, 0),          # 1024 tiles: two whole tiles per workgroup
    (1280, 4096, 80, 0),          # no MFMA path for d = 80
    (1280, 4100, 72, 0),          # keys not a multiple of 64
    (1920, 4096, 72, 0),          # 480 tiles: 60 units cut against 64 whole
])
def test_attention_work_plan_workspace(orch_lib, n_q, n_kv, d, want):
    """Host-side work plan of the attention: when query tiles are cut between
    workgroups, and the workspace their parts take."""
    assert orch_lib.attention_workspace_bytes(2, 16, n_q, n_kv, d, 1) == want
    assert orch_lib.attention_workspace_bytes(2, 16, n_q, n_kv, d, 0) == 0   # fp32: no MFMA path


@pytest.mark.parametrize("M,N,K,want", [
    # DiT-XL/2 at the 10% band (M = 768): fc2 has 54 tiles of 128x128 -> 4
    # k-splits of 18 k-tiles, fp32 partials 4 x 768 x 1152
    (768, 1152, 4608, 4 * 768 * 1152 * 4),
    (768, 1152, 1152, 2 * 768 * 1152 * 4),   # out-proj: 18 k-tiles -> 2 splits of 9
    (2048, 1152, 4608, 0),                    # 144 tiles: a split would take two rounds
    (3328, 1152, 4608, 0),                    # 234 tiles fill the machine
    (768, 3456, 1152, 0),                     # QKV: 162 tiles
    (768, 1152, 4600, 0),                     # K % 64: no MFMA path
])
def test_linear_split_workspace(orch_lib, M, N, K, want):
    """Host-side k-split plan of the projection GEMM."""
    assert orch_lib.linear_workspace_bytes(M, N, K, 1) == want
    assert orch_lib.linear_workspace_bytes(M, N, K, 0) == 0   # fp32: no MFMA path


def test_library_speeds_match_oracle(orch_lib):
    rng = np.random.default_rng(3)
    for trial in range(100):
        n = int(rng.integers(1, 6))
        profs = []
        for _ in range(n):
            k = int(rng.integers(1, 7))
            rows = [int(r) for r in rng.integers(1, 129, k)]
            a, b = rng.uniform(0.0, 3.0), rng.uniform(0.01, 0.5)
            profs.append([(r, a + b * r + rng.uniform(-0.01, 0.01)) for r in rows])
        ref = int(rng.integers(1, 129))
        got = orch_lib.speeds_from_profiles(profs, ref)
        want = [oal.speed_from_profile([r for r, _ in p], [t for _, t in p], ref) for p in profs]
        np.testing.assert_allclose(got, want, rtol=1e-9)


@pytest.mark.parametrize("profs,ref,word", [
    ([[]], 8, "at least one"), ([[(0, 1.0)]], 8, "rows >= 1"), ([[(4, -1.0)]], 8, "times > 0"),
    ([[(4, 1.0)]], 0, "ref_rows"), ([[(4, 10.0), (8, 1.0)]], 64, "not positive"),
])
def test_library_speeds_reject(orch_lib, profs, ref, word):
    with pytest.raises(orch_lib.OrchError) as e:
        orch_lib.speeds_from_profiles(profs, ref)
    assert e.value.code == orch_lib.ORCH_EINVAL and word in orch_lib.last_error()


def _al256(b):
    return (b + 255) // 256 * 256


@pytest.mark.parametrize("H,C,Co,rows,splits", [
    # SDXL-sized stages at 1024px (32 groups): the k-split the launch plan
    # picks per band height (its tile shape is not visible here); the fp32
    # partials of a split take splits x M x C_out x 4 bytes of the workspace
    (128, 320, 320, 16, 3), (128, 320, 320, 56, 2), (128, 320, 320, 72, 1), (128, 320, 320, 128, 1),
    (64, 640, 640, 8, 6), (64, 640, 640, 28, 4), (64, 640, 640, 36, 3), (64, 640, 640, 64, 2),
    (32, 1280, 1280, 4, 16), (32, 1280, 1280, 14, 6), (32, 1280, 1280, 18, 6), (32, 1280, 1280, 32, 4),
])
def test_unet_workspace_follows_launch_plan(orch_lib, H, C, Co, rows, splits):
    """Workspace of the U-Net band block: the band's per-row sums, the
    zero-bordered activation tile [rows + 2][W + 2][C] bf16, and the k-split's
    partial sums; pins the split counts the launch plan chooses."""
    shape = orch_lib.UNetConvShape(H, H, C, 32, Co, 1e-5)
    M = rows * H
    want = _al256(rows * 32 * 8) + _al256((rows + 2) * (H + 2) * C * 2)
    if splits > 1:
        want += _al256(splits * M * Co * 4)
    assert orch_lib.unet_conv_workspace_bytes(shape, rows) == want


def test_unet_rejects_map_beyond_32_bit_offsets(orch_lib):
    """The convolution indexes the activation tile and the weights with 32-bit
    byte offsets; a map whose bf16 tile would reach 2 GiB is refused before
    any launch."""
    import ctypes as C
    shape = orch_lib.UNetConvShape(4096, 4094, 64, 8, 64, 1e-5)   # 4098 x 4096 x 64 x 2 B = 2 GiB
    rc = orch_lib.lib.orch_unet_conv_band(C.byref(shape), 0, 4, None, None, None, None, None, None, None,
                                          0, None, None, C.c_size_t(0), None)
    assert rc == orch_lib.ORCH_EINVAL and "too large" in orch_lib.last_error()
    ok = orch_lib.UNetConvShape(128, 128, 320, 32, 320, 1e-5)
    rc = orch_lib.lib.orch_unet_conv_band(C.byref(ok), 0, 4, None, None, None, None, None, None, None,
                                          0, None, None, C.c_size_t(0), None)
    assert rc == orch_lib.ORCH_EINVAL and "too large" not in orch_lib.last_error()
