// Host-side part of the C ABI: error state, version, keep count and APC target size.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include "pace_internal.h"

namespace pace {

static thread_local char g_err[512] = "";

pace_status_t set_error(pace_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

pace_status_t check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(PACE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return PACE_OK;
}

}  // namespace pace

extern "C" {

const char* pace_last_error(void) { return pace::g_err; }

int pace_version(void) { return 100; }

int pace_keep_count(double ratio, int n) {
  if (n < 0 || !isfinite(ratio)) return -1;
  double k = ceil(ratio * static_cast<double>(n) - 1e-9);
  if (k < 0) k = 0;
  if (k > n) k = n;
  return static_cast<int>(k);
}

int pace_keep_from_density(double rho, double ratio_lo, double ratio_hi, int n) {
  if (n < 0 || !isfinite(rho) || !(ratio_lo >= 0) || !(ratio_hi >= ratio_lo) || ratio_hi > 1) return -1;
  double r = ratio_lo + (ratio_hi - ratio_lo) * rho;
  r = fmin(fmax(r, ratio_lo), ratio_hi);
  return pace_keep_count(r, n);
}

pace_status_t pace_apc_target_size(double rho, int H, int W, double min_pixels, double max_pixels,
                                   int snap, int* oH, int* oW) {
  PACE_REQUIRE(H > 0 && W > 0 && snap > 0, "pace_apc_target_size: H=%d W=%d snap=%d must be > 0",
               H, W, snap);
  PACE_REQUIRE(oH != nullptr && oW != nullptr, "pace_apc_target_size: null output pointer");
  PACE_REQUIRE(isfinite(rho) && min_pixels >= 0 && max_pixels > 0,
               "pace_apc_target_size: bad rho or pixel budget");
  const double area = static_cast<double>(H) * static_cast<double>(W);
  const double r_cap = fmin(1.0, max_pixels / area);
  const double r_floor = fmin(r_cap, min_pixels / area);
  const double r = fmin(fmax(rho, r_floor), r_cap);
  const double s = sqrt(r);
  auto side = [&](int X) {
    long o = static_cast<long>(floor(X * s / snap + 0.5)) * snap;
    const long hi = static_cast<long>(X / snap) * snap;
    if (o > hi) o = hi;
    const long lo = snap < X ? snap : X;
    if (o < lo) o = lo;
    return static_cast<int>(o);
  };
  *oH = side(H);
  *oW = side(W);
  return PACE_OK;
}

}  // extern "C"
