"""Pins of the oracle's scheduler against closed forms and the paper's tables.

The update of §I and Lemma 1 (Eq. (1)) fix x_prev = A x - Bc eps (+ C z);
Eq. (2) and Table II fix the step count of the reduced tier.
"""
import os

import mpmath
import numpy as np
import pytest

from oracle import schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                out.append(line.split())
    return out


def _mp_coeffs(t, t_prev):
    """Eq. (1) at 50 digits, written from the definitions: abar as a product
    of (1 - beta), lambda = log(alpha/sigma), Bc = sigma_p (e^h - 1); the
    final step (sigma_p = 0) through its limit alpha_p sigma_s/alpha_s."""
    mpmath.mp.dps = 50
    T = 1000
    b0, b1 = mpmath.mpf("1e-4"), mpmath.mpf("2e-2")
    beta = [b0 + (b1 - b0) * i / (T - 1) for i in range(T)]

    def abar(n):
        if n < 0:
            return mpmath.mpf(1)
        p = mpmath.mpf(1)
        for i in range(n + 1):
            p *= 1 - beta[i]
        return p

    a_s, a_p = mpmath.sqrt(abar(t)), mpmath.sqrt(abar(t_prev))
    s_s, s_p = mpmath.sqrt(1 - abar(t)), mpmath.sqrt(1 - abar(t_prev))
    A = a_p / a_s
    if t_prev < 0:
        Bc = a_p * s_s / a_s
    else:
        h = mpmath.log(a_p / s_p) - mpmath.log(a_s / s_s)
        Bc = s_p * mpmath.expm1(h)
    return A, Bc


@pytest.mark.parametrize("row", _rows("scheduler_hand_values.txt"))
def test_p1_hand_values(row):
    t, tp = int(row[0]), int(row[1])
    A_g, B_g = float(row[2]), float(row[3])
    A_mp, B_mp = _mp_coeffs(t, tp)
    assert abs(float(A_mp) - A_g) <= 1e-15 * abs(A_g)
    assert abs(float(B_mp) - B_g) <= 1e-15 * abs(B_g)
    ab = schedule.alpha_bar()
    A, Bc, C = schedule.ddim_coefficients(ab, t, tp)
    assert C == 0.0
    assert abs(A - A_g) <= 1e-13 * abs(A_g)
    assert abs(Bc - B_g) <= 1e-12 * abs(B_g)


def test_p1_update_value():
    # x = 1, eps = 0.5 at 980 -> 960: A - 0.5 Bc
    ab = schedule.alpha_bar()
    A, Bc, C = schedule.ddim_coefficients(ab, 980, 960)
    out = schedule.scheduler_update(np.array([1.0]), np.array([0.5]), A, Bc, C)
    assert abs(out[0] - 1.10840299258051222) < 1e-14


def test_alpha_bar_endpoints():
    ab = schedule.alpha_bar()
    assert ab.shape == (1000,)
    assert ab[0] == pytest.approx(0.9999, rel=1e-15)
    assert ab[999] == pytest.approx(4.0358297653757e-5, rel=1e-12)
    assert np.all(np.diff(ab) < 0)


@pytest.mark.parametrize("pair", schedule.step_pairs(1000, 50)[:-1] + [(750, 500), (999, 0)])
def test_p2_lemma1_equals_rearranged(pair):
    t, tp = pair
    ab = schedule.alpha_bar()
    A1, B1 = schedule.lemma1_coefficients(ab, t, tp)
    A2, B2, _ = schedule.ddim_coefficients(ab, t, tp)
    assert abs(A1 - A2) <= 1e-14 * abs(A2)
    assert abs(B1 - B2) <= 1e-12 * abs(B2)


@pytest.mark.parametrize("pair", [(980, 960), (500, 250), (20, 0), (0, -1), (40, -1), (780, 740)])
def test_p3_forward_marginal(pair):
    """If x_s = alpha_s x0 + sigma_s eps exactly, one step with that eps lands
    on alpha_p x0 + sigma_p eps (and on x0 at the final step)."""
    t, tp = pair
    ab = schedule.alpha_bar()
    a_s, s_s = schedule.alpha_sigma(ab, t)
    a_p, s_p = schedule.alpha_sigma(ab, tp)
    x0 = np.array([0.3, -2.0, 1.7])
    eps = np.array([-1.25, 0.5, 0.0])
    x = a_s * x0 + s_s * eps
    A, Bc, C = schedule.ddim_coefficients(ab, t, tp)
    out = schedule.scheduler_update(x, eps, A, Bc, C)
    np.testing.assert_allclose(out, a_p * x0 + s_p * eps, rtol=0, atol=1e-12)
    if tp == -1:
        np.testing.assert_allclose(out, x0, atol=1e-12)


@pytest.mark.parametrize("t", [1, 10, 500, 999])
def test_eta1_consecutive_is_ddpm_posterior(t):
    """eta = 1 over one grid interval is the DDPM ancestral step: the noise
    scale is the posterior std sqrt(beta_t (1 - abar_{t-1}) / (1 - abar_t))
    and the mean is (x - beta_t / sqrt(1 - abar_t) eps) / sqrt(1 - beta_t)."""
    beta = schedule.betas()
    ab = schedule.alpha_bar()
    A, Bc, C = schedule.ddim_coefficients(ab, t, t - 1, eta=1.0)
    post_var = beta[t] * (1 - ab[t - 1]) / (1 - ab[t])
    assert C * C == pytest.approx(post_var, rel=1e-10)
    assert A == pytest.approx(1 / np.sqrt(1 - beta[t]), rel=1e-13)
    assert Bc == pytest.approx(beta[t] / np.sqrt(1 - ab[t]) / np.sqrt(1 - beta[t]), rel=1e-9)


def test_grid_and_pairs():
    assert schedule.ddim_grid(1000, 4) == [0, 250, 500, 750]
    p = schedule.step_pairs(1000, 50)
    assert p[0] == (980, 960) and p[10] == (780, 760) and p[-2] == (20, 0) and p[-1] == (0, -1)
    assert len(p) == 50
    assert schedule.step_pairs(1000, 4) == [(750, 500), (500, 250), (250, 0), (0, -1)]


@pytest.mark.parametrize("row", _rows("tiered_step_counts.txt"))
def test_p10_table2_step_counts(row):
    mb, mw, mr = map(int, row)
    assert schedule.tiered_step_count(mb, mw) == mr
    assert len(schedule.tiered_schedule(1000, mb, mw)) == mr


def test_p10_tiered_schedule_2048():
    s = schedule.tiered_schedule(1000, 50, 10)
    assert len(s) == 30 == schedule.tiered_step_count(50, 10)
    ms = [m for m, _, _, _ in s]
    assert ms == list(range(10)) + list(range(10, 50, 2))
    assert s[9][1:3] == (800, 780)
    assert s[10][1:3] == (780, 740)          # first stride-2 step
    assert s[-1][1:3] == (20, -1)            # last pair ends the trajectory
    assert all(r for *_, r in s)
    # the executed steps tile the grid with no gap
    for a, b in zip(s, s[1:]):
        assert a[2] == b[1]
