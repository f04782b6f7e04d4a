// Host side of the calibration: the all-running window of a co-run, the least-squares fit of
// the slowdown factors (Sec. 5.2.2: factors trained on benchmarked co-runs of several shapes
// and combinations) and Algorithm 1 on one vector of stream times.
#include <cmath>
#include <limits>
#include <string>

#include "mist.h"

namespace mist {
__attribute__((visibility("hidden"))) mist_status lib_fail(mist_status code, const std::string& msg);  // sets the thread's error
}

namespace {

int popcount4(int v) { return (v & 1) + (v >> 1 & 1) + (v >> 2 & 1) + (v >> 3 & 1); }

bool finite_nonneg(double x) { return x >= 0.0 && std::isfinite(x); }

}  // namespace

extern "C" {

mist_status mist_corun_reduce(int32_t mask, const double* t, int32_t stride, const int32_t* units, double* mean,
                              int32_t* count) {
  using mist::lib_fail;
  if (!t || !units || !mean || !count) return lib_fail(MIST_E_INVALID, "null argument");
  if (mask < 1 || mask > 15) return lib_fail(MIST_E_INVALID, "mask must be in 1..15");
  double lo = -std::numeric_limits<double>::infinity();
  double hi = std::numeric_limits<double>::infinity();
  for (int j = 0; j < 4; ++j) {
    if (!(mask >> j & 1)) continue;
    if (units[j] < 1) return lib_fail(MIST_E_INVALID, "every member needs a unit");
    if (stride <= units[j]) return lib_fail(MIST_E_INVALID, "stride must exceed every member's unit count");
    const double* tj = t + (int64_t)j * stride;
    for (int i = 0; i < units[j]; ++i)
      if (!(tj[i] <= tj[i + 1]) || !std::isfinite(tj[i]) || !std::isfinite(tj[i + 1]))
        return lib_fail(MIST_E_INVALID, "timestamps must be finite and non-decreasing");
    lo = std::fmax(lo, tj[0]);
    hi = std::fmin(hi, tj[units[j]]);
  }
  for (int j = 0; j < 4; ++j) {
    mean[j] = std::numeric_limits<double>::quiet_NaN();
    count[j] = 0;
    if (!(mask >> j & 1)) continue;
    const double* tj = t + (int64_t)j * stride;
    double sum = 0.0;
    int32_t n = 0;
    for (int i = 0; i < units[j]; ++i) {
      if (tj[i] >= lo && tj[i + 1] <= hi) {
        sum += tj[i + 1] - tj[i];
        ++n;
      }
    }
    if (n) {
      mean[j] = sum / n;
      count[j] = n;
    }
  }
  return MIST_OK;
}

mist_status mist_fit_phi(const mist_corun_sample* s, int64_t n, double* phi) {
  using mist::lib_fail;
  if (!phi || (n > 0 && !s) || n < 0) return lib_fail(MIST_E_INVALID, "bad argument");
  double cs[16][4] = {}, ss[16][4] = {};
  bool seen[16][4] = {};
  for (int64_t i = 0; i < n; ++i) {
    const mist_corun_sample& x = s[i];
    if (x.mask < 1 || x.mask > 15 || x.stream < 0 || x.stream > 3 || !(x.mask >> x.stream & 1))
      return lib_fail(MIST_E_INVALID, "sample " + std::to_string(i) + ": stream not in its mask");
    if (!(x.solo_s > 0.0) || !std::isfinite(x.solo_s) || !(x.corun_s > 0.0) || !std::isfinite(x.corun_s))
      return lib_fail(MIST_E_INVALID, "sample " + std::to_string(i) + ": times must be positive and finite");
    cs[x.mask][x.stream] += x.corun_s * x.solo_s;
    ss[x.mask][x.stream] += x.solo_s * x.solo_s;
    seen[x.mask][x.stream] = true;
  }
  for (int mask = 0; mask < 16; ++mask) {
    for (int j = 0; j < 4; ++j) {
      double v = 1.0;
      if (popcount4(mask) >= 2 && (mask >> j & 1)) {
        if (!seen[mask][j])
          return lib_fail(MIST_E_INVALID, "no sample for stream " + std::to_string(j) + " of mask " +
                                              std::to_string(mask));
        v = std::fmax(1.0, cs[mask][j] / ss[mask][j]);
      }
      phi[mask * 4 + j] = v;
    }
  }
  return MIST_OK;
}

mist_status mist_interference(const double* phi, const double* x, double* out) {
  using mist::lib_fail;
  if (!phi || !x || !out) return lib_fail(MIST_E_INVALID, "null argument");
  for (int j = 0; j < 4; ++j)
    if (!finite_nonneg(x[j])) return lib_fail(MIST_E_INVALID, "stream times must be finite and >= 0");
  for (int mask = 0; mask < 16; ++mask)
    for (int j = 0; j < 4; ++j)
      if (popcount4(mask) >= 2 && (mask >> j & 1) && !(phi[mask * 4 + j] >= 1.0 && std::isfinite(phi[mask * 4 + j])))
        return lib_fail(MIST_E_INVALID, "slowdown factors must be finite and >= 1");
  double X[4] = {x[0], x[1], x[2], x[3]};
  double T = 0.0;
  // While two or more streams still run, the combination of the running streams is scaled by
  // its factors, the smallest scaled time overlaps all of them and is added to the total, and
  // the members keep their scaled leftovers divided by the factor (a multiplication by 1/phi).
  for (;;) {
    int running = 0;
    for (int j = 0; j < 4; ++j)
      if (X[j] > 0.0) running |= 1 << j;
    if (popcount4(running) < 2) break;
    double sc[4];
    double ov = std::numeric_limits<double>::infinity();
    for (int j = 0; j < 4; ++j) {
      if (!(running >> j & 1)) continue;
      sc[j] = X[j] * phi[running * 4 + j];
      ov = std::fmin(ov, sc[j]);
    }
    for (int j = 0; j < 4; ++j)
      if (running >> j & 1) X[j] = (sc[j] - ov) * (1.0 / phi[running * 4 + j]);
    T = T + ov;
  }
  // At most one stream is left.
  *out = T + std::fmax(std::fmax(X[0], X[1]), std::fmax(X[2], X[3]));
  return MIST_OK;
}

}  // extern "C"
