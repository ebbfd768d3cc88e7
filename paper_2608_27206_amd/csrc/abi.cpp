// Host-side part of the C ABI: error state, version, keep count and APC target size.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

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

bool debug_checks() {
  const char* e = getenv("PACE_DEBUG");
  return e != nullptr && e[0] == '1' && e[1] == '\0';
}

pace_status_t copy_to_host(int32_t* dst, const int32_t* src, int n, hipStream_t stream) {
  if (n <= 0) return PACE_OK;
  if (hipMemcpyAsync(dst, src, static_cast<size_t>(n) * sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
          hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return set_error(PACE_ERR_HIP, "metadata copy to the host failed");
  return PACE_OK;
}

pace_status_t check_offsets(const int32_t* cu, int n, long long total, int max_len, const char* what,
                            hipStream_t stream) {
  if (!debug_checks()) return PACE_OK;
  std::vector<int32_t> h(static_cast<size_t>(n) + 1);
  pace_status_t st = copy_to_host(h.data(), cu, n + 1, stream);
  if (st != PACE_OK) return st;
  if (h[0] != 0) return set_error(PACE_ERR_INVALID_ARG, "%s: offsets[0] = %d, not 0", what, h[0]);
  for (int b = 0; b < n; ++b) {
    const long long len = static_cast<long long>(h[b + 1]) - h[b];
    if (len < 0 || len > max_len)
      return set_error(PACE_ERR_INVALID_ARG, "%s: segment %d has length %lld, outside [0, %d]", what, b,
                       len, max_len);
  }
  if (h[n] > total)
    return set_error(PACE_ERR_INVALID_ARG, "%s: offsets end at %d, past %lld", what, h[n], total);
  return PACE_OK;
}

pace_status_t check_values(const int32_t* v, int n, const int32_t* upper_host, int lo, int vmax,
                           const char* what, hipStream_t stream) {
  if (!debug_checks()) return PACE_OK;
  std::vector<int32_t> h(static_cast<size_t>(n));
  pace_status_t st = copy_to_host(h.data(), v, n, stream);
  if (st != PACE_OK) return st;
  for (int b = 0; b < n; ++b) {
    const int hi = upper_host ? (upper_host[b] < vmax ? upper_host[b] : vmax) : vmax;
    if (h[b] < lo || h[b] > hi)
      return set_error(PACE_ERR_INVALID_ARG, "%s[%d] = %d outside [%d, %d]", what, b, h[b], lo, hi);
  }
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
