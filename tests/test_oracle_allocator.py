"""Pins of the device planner (Eq. (2), Eq. (3)) against the paper's tables."""
import os

import numpy as np
import pytest

from oracle import allocator as al

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_patch_assignment.txt")


def _table1():
    rows = []
    for line in open(GOLDEN):
        if line.strip() and not line.startswith("#"):
            rows.append(tuple(int(x) for x in line.split()))
    return rows


@pytest.mark.parametrize("row", _table1())
def test_table1_assignments(row):
    """Quality table: patch units and reduced tier from occupancies (v = 1 - rho)."""
    o0, o1, p0, p1, red = row
    v = [al.effective_speed(1.0, o0 / 100), al.effective_speed(1.0, o1 / 100)]
    steps, rows = al.plan(v, 100, 4, a=0.75, b=0.25, total_rows=32)
    assert rows == [p0, p1]
    assert steps == [100, 52 if red else 100]


@pytest.mark.parametrize("M_base,expect", [(100, 52), (50, 27)])
def test_table2_step_counts(M_base, expect):
    """Quality table II: a reduced device runs 100:52 and 50:27 steps (M_warmup = 4)."""
    assert al.step_counts([1.0, 0.5], M_base, 4, a=0.75, b=0.25) == [M_base, expect]


def test_thresholds_and_exclusion():
    v = [1.0, 0.9, 0.75, 0.5, 0.25, 0.2]
    steps = al.step_counts(v, 50, 10, a=0.75, b=0.25)
    # a*vmax < v keeps M_base; b*vmax < v <= a*vmax reduced; v <= b*vmax excluded
    assert steps == [50, 50, 30, 30, 0, 0]
    steps, rows = al.plan(v, 50, 10, 0.75, 0.25, 64)
    assert rows[4] == rows[5] == 0 and sum(rows) == 64


def test_reduced_count_equals_executed_schedule():
    """Eq. (2)'s reduced count is the number of steps the reduced tier runs
    (odd M_base - M_warmup included: Table IV's M_warmup = 25 at M_base = 100)."""
    from oracle import schedule
    for mb in range(1, 121):
        for mw in range(0, mb + 1):
            n = len(schedule.tiered_schedule(1000, mb, mw)) if mb <= 1000 else None
            assert al.reduced_steps(mb, mw) == n == schedule.tiered_step_count(mb, mw), (mb, mw)
    assert al.reduced_steps(100, 25) == 63


def test_device_without_rows_has_no_steps():
    """A device kept by Eq. (2) whose Eq. (3) share rounds to 0 rows has no work."""
    v = [1.0, 1.0, 0.3]                      # reduced tier, 0.43 of 2 rows
    assert al.step_counts(v, 50, 4, 0.75, 0.25) == [50, 50, 27]
    assert al.plan(v, 50, 4, 0.75, 0.25, 2) == ([50, 50, 0], [1, 1, 0])
    # equal devices, fewer rows than devices: the last ones get none
    assert al.plan([1.0] * 6, 50, 10, 0.75, 0.25, 4) == ([50] * 4 + [0] * 2, [1] * 4 + [0] * 2)


def test_equal_devices_split_evenly():
    steps, rows = al.plan([0.7] * 4, 50, 10, 0.75, 0.25, 64)
    assert steps == [50] * 4 and rows == [16] * 4


def test_mending_equalises_rate():
    """Eq. (3): (v_i/M_i)/P_i is the same for every device (before rounding)."""
    rng = np.random.default_rng(0)
    v = list(rng.uniform(0.35, 1.0, 7))
    steps = al.step_counts(v, 100, 4, 0.8, 0.25)
    sh = al.patch_shares(v, steps)
    r = [vi / m / s for vi, m, s in zip(v, steps, sh) if m]
    assert np.allclose(r, r[0]) and abs(sum(sh) - 1) < 1e-12


def test_whole_rows_largest_remainder():
    assert al.whole_rows([0.5, 0.5], 5) == [3, 2]          # tie -> lower index
    assert al.whole_rows([0.1, 0.2, 0.7], 10) == [1, 2, 7]
    assert al.whole_rows([1 / 3] * 3, 64) == [22, 21, 21]
    rng = np.random.default_rng(1)
    for _ in range(200):
        s = rng.dirichlet(np.ones(5))
        r = al.whole_rows(list(s), 61)
        assert sum(r) == 61 and all(abs(ri - si * 61) < 1 for ri, si in zip(r, s))


def test_speed_from_profile_pins():
    """Synthetic profiles whose speeds follow from the definition by hand."""
    # exactly linear: t = 2 + 0.5 r  -> at r = 16: 16 / 10
    rows = [4, 8, 16, 32]
    t = [2 + 0.5 * r for r in rows]
    assert abs(al.speed_from_profile(rows, t, 16) - 1.6) < 1e-12
    # no fixed cost: the speed is 1 / beta at any reference height
    assert abs(al.speed_from_profile(rows, [0.25 * r for r in rows], 7) - 4.0) < 1e-12
    # a device k times slower (an occupancy of 1 - 1/k) has 1/k of the speed
    s1 = al.speed_from_profile(rows, t, 16)
    s3 = al.speed_from_profile(rows, [3 * x for x in t], 16)
    assert abs(s1 / s3 - 3.0) < 1e-12
    # the fixed cost makes the speed depend on the reference height
    assert al.speed_from_profile(rows, t, 4) < al.speed_from_profile(rows, t, 32)
    # a single height: alpha = 0
    assert abs(al.speed_from_profile([10, 10], [4.0, 6.0], 3) - 2.0) < 1e-12
    # noise around a line: the least-squares fit recovers it exactly for
    # symmetric residuals
    tn = [x + e for x, e in zip(t, [0.1, -0.1, -0.1, 0.1])]
    r = np.array(rows, float)
    fit = np.polyfit(r, tn, 1)
    assert abs(al.speed_from_profile(rows, tn, 16) - 16 / np.polyval(fit, 16)) < 1e-12


def test_profiled_speeds_reproduce_occupancy_speeds():
    """Profiles of one device scaled by 1/(1 - rho) give speeds proportional
    to 1 - rho, so the plan equals the occupancy plan."""
    rows = [4, 8, 16, 32, 64]
    t = [0.8 + 0.2 * r for r in rows]
    occ = [0.0, 0.4]
    v = [al.speed_from_profile(rows, [x / (1 - o) for x in t], 16) for o in occ]
    assert al.plan(v, 100, 4, 0.75, 0.25, 32) == al.plan([1 - o for o in occ], 100, 4, 0.75, 0.25, 32)
