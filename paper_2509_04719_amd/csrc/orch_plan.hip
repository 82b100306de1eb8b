// Device planning of the method, host only: temporal adaptation (Eq. (2),
// tiered step counts with exclusion) and spatial adaptation (Eq. (3), patch
// mending), turned into whole token rows.
#include <cmath>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/orch.h"

namespace orch_detail {
int set_error(int code, const char* msg);
}

int orch_plan_devices(const double* speed, int n, int m_base, int m_warmup, double a, double b,
                      int total_rows, int* steps_out, int* rows_out) {
  using orch_detail::set_error;
  if (!speed || !steps_out || !rows_out) return set_error(ORCH_EINVAL, "NULL argument");
  if (n < 1 || total_rows < 1) return set_error(ORCH_EINVAL, "need n >= 1 and total_rows >= 1");
  if (m_base < 1 || m_warmup < 0 || m_warmup > m_base)
    return set_error(ORCH_EINVAL, "need m_base >= 1 and 0 <= m_warmup <= m_base");
  if (!(0.0 < b && b < a && a < 1.0)) return set_error(ORCH_EINVAL, "need 0 < b < a < 1");
  double vmax = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!(speed[i] > 0.0) || !std::isfinite(speed[i]))
      return set_error(ORCH_EINVAL, "speeds must be finite and > 0");
    vmax = std::max(vmax, speed[i]);
  }
  // Eq. (2): full, reduced or excluded.  The reduced tier runs m_warmup
  // single steps, then the rest of the grid in steps of two intervals (the
  // last one single when m_base - m_warmup is odd): ceil((m_base + m_warmup)/2).
  std::vector<int> steps(n);
  for (int i = 0; i < n; ++i) {
    if (speed[i] > a * vmax) steps[i] = m_base;
    else if (speed[i] > b * vmax) steps[i] = m_warmup + (m_base - m_warmup + 1) / 2;
    else steps[i] = 0;
  }
  // Eq. (3): share of device i = (v_i/M_i) / sum_j (v_j/M_j)
  double tot = 0.0;
  std::vector<double> rate(n, 0.0);
  for (int i = 0; i < n; ++i)
    if (steps[i]) tot += (rate[i] = speed[i] / steps[i]);
  // whole rows by largest remainders (ties to the lower index)
  std::vector<int> rows(n);
  std::vector<double> frac(n);
  int used = 0;
  for (int i = 0; i < n; ++i) {
    const double exact = rate[i] / tot * total_rows;
    rows[i] = (int)std::floor(exact);
    frac[i] = exact - rows[i];
    used += rows[i];
  }
  for (int left = total_rows - used; left > 0; --left) {
    int best = -1;
    for (int i = 0; i < n; ++i)
      if (steps[i] && (best < 0 || frac[i] > frac[best])) best = i;
    ++rows[best];
    frac[best] = -1.0;
  }
  // a device left with no rows has no work
  for (int i = 0; i < n; ++i) {
    steps_out[i] = rows[i] > 0 ? steps[i] : 0;
    rows_out[i] = rows[i];
  }
  return ORCH_OK;
}

// Effective speed of each device from its inference time profile: the
// measured step times t_j at band heights r_j, fitted by least squares as
// t = alpha + beta r (a fixed per-step cost plus a per-row cost), evaluated at
// the reference band height: v = ref_rows / (alpha + beta ref_rows), rows per
// unit of time.  One point (or one distinct height) gives beta = mean t / r.
int orch_speeds_from_profiles(int n, const int* n_points, const int* rows, const double* ms,
                              int ref_rows, double* speed_out) {
  using orch_detail::set_error;
  if (!n_points || !rows || !ms || !speed_out) return set_error(ORCH_EINVAL, "NULL argument");
  if (n < 1 || ref_rows < 1) return set_error(ORCH_EINVAL, "need n >= 1 and ref_rows >= 1");
  int off = 0;
  std::vector<double> v(n);
  for (int i = 0; i < n; ++i) {
    const int k = n_points[i];
    if (k < 1) return set_error(ORCH_EINVAL, "every device needs at least one profile point");
    double sr = 0, st = 0, srr = 0, srt = 0;
    bool distinct = false;
    for (int j = off; j < off + k; ++j) {
      if (rows[j] < 1 || !(ms[j] > 0.0) || !std::isfinite(ms[j]))
        return set_error(ORCH_EINVAL, "profile points need rows >= 1 and finite times > 0");
      distinct |= rows[j] != rows[off];
      sr += rows[j]; st += ms[j]; srr += (double)rows[j] * rows[j]; srt += rows[j] * ms[j];
    }
    double alpha = 0.0, beta;
    if (distinct) {
      beta = (k * srt - sr * st) / (k * srr - sr * sr);
      alpha = (st - beta * sr) / k;
    } else {
      beta = st / sr;
    }
    const double t_ref = alpha + beta * ref_rows;
    if (!(t_ref > 0.0) || !std::isfinite(t_ref))
      return set_error(ORCH_EINVAL, "fitted step time at the reference height is not positive");
    v[i] = ref_rows / t_ref;
    off += k;
  }
  for (int i = 0; i < n; ++i) speed_out[i] = v[i];
  return ORCH_OK;
}
