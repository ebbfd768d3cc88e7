// APC (Section 3.2, "Condense"): per-patch information density of a uint8 image and
// the bicubic resize by sqrt(r) per side (Appendix implementation details).
//
// Density, five launches (all HBM/L2-bound, fixed reduction orders -> deterministic):
//   apc_patch_pass<0>  per patch-strip tile: ||f_i|| -> 1/||f_i||, and the tile's partial
//                      sum of T_i = f_i/||f_i|| over its patches (one 588-vector per tile)
//   apc_reduce_c       sum of the tile partials per component -> sum_i T_i
//   apc_finalize_c     c = mean T_i, phi = ||c||^2 (equal to Eq. 1's mean pairwise cosine),
//                      rho_g = 1 - phi (Eq. 2), c_hat = c/||c||
//   apc_patch_pass<1>  d_i = ||T_i - c_hat|| (the image is re-read, mostly from L2/MALL)
//   apc_tail           radix select of the n_tail-th largest d, tail mean, rho_d, rho
//
// The per-patch feature is the patch's pixels mapped to x/127.5 - 1 (component order:
// patch row, pixel column, channel).  The order does not change norms or cosines.
#include <math.h>

#include "pace_internal.h"

namespace pace {
namespace {

constexpr int kPatchesPerTile = 16;   // patches of one patch row per workgroup
constexpr int kApcThreads = 256;      // 16 threads per patch
constexpr int kMaxPatch = 16;

struct DensityParams {
  const uint8_t* img;
  int H, W, P;            // image and patch size
  int gh, gw, N;          // patch grid
  int D;                  // 3 * P * P
  int tiles_x;            // tiles per patch row
  int n_tiles;
  int n_tail;
  float alpha, gamma;
  float* inv_norm;        // [N]
  float* partial;         // [n_tiles, D]
  float* csum;            // [D]
  float* chat;            // [D]
  float* stats;           // [8]: phi, rho_g, |c|, ...
  float* d;               // [N]
  float* rho_out;         // [4]
};

// Loads the tile's pixels (P rows x up to 16 patches) into LDS as floats x/127.5 - 1.
__device__ __forceinline__ int load_tile(const DensityParams& p, int tile, float* f, int* py_out,
                                         int* px0_out) {
  const int py = tile / p.tiles_x;
  const int px0 = (tile % p.tiles_x) * kPatchesPerTile;
  const int np = min(kPatchesPerTile, p.gw - px0);
  const int row_bytes = np * p.P * 3;
  const long long rowstride = static_cast<long long>(p.W) * 3;
  const uint8_t* src = p.img + static_cast<long long>(py * p.P) * rowstride + px0 * p.P * 3;
  const int lds_stride = kPatchesPerTile * p.P * 3;
  for (int e = threadIdx.x; e < p.P * row_bytes; e += kApcThreads) {
    const int r = e / row_bytes, cb = e - r * row_bytes;
    f[r * lds_stride + cb] =
        static_cast<float>(src[r * rowstride + cb]) * (1.0f / 127.5f) - 1.0f;
  }
  *py_out = py;
  *px0_out = px0;
  return np;
}

// Feature component e of patch j within the tile (LDS layout [row][tile column byte]).
__device__ __forceinline__ float feat(const float* f, int P, int j, int e) {
  const int r = e / (3 * P), cb = e - r * (3 * P);
  return f[r * (kPatchesPerTile * P * 3) + j * 3 * P + cb];
}

template <int PASS>
__global__ __launch_bounds__(kApcThreads) void apc_patch_pass(const DensityParams p) {
  extern __shared__ float lds[];
  float* f = lds;                                                 // [P][16*P*3] floats
  float* inv = f + p.P * kPatchesPerTile * p.P * 3;               // [16]
  float* chat = inv + kPatchesPerTile;                            // [D] (pass 1)
  const int tile = blockIdx.x;
  int py, px0;
  const int np = load_tile(p, tile, f, &py, &px0);
  if (PASS == 1)
    for (int e = threadIdx.x; e < p.D; e += kApcThreads) chat[e] = p.chat[e];
  __syncthreads();
  const int j = threadIdx.x >> 4, t = threadIdx.x & 15;
  float acc = 0.f;
  if (j < np) {
    if (PASS == 0) {
      for (int e = t; e < p.D; e += 16) { const float x = feat(f, p.P, j, e); acc += x * x; }
    } else {
      const float s = p.inv_norm[py * p.gw + px0 + j];
      for (int e = t; e < p.D; e += 16) {
        const float x = feat(f, p.P, j, e) * s - chat[e];
        acc += x * x;
      }
    }
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if (PASS == 0) {
    if (j < np && t == 0) {
      const float in = 1.0f / sqrtf(acc);
      inv[j] = in;
      p.inv_norm[py * p.gw + px0 + j] = in;
    }
    __syncthreads();
    // tile partial of sum_i T_i, patches added in index order
    for (int e = threadIdx.x; e < p.D; e += kApcThreads) {
      float s = 0.f;
      for (int jj = 0; jj < np; ++jj) s += feat(f, p.P, jj, e) * inv[jj];
      p.partial[static_cast<long long>(tile) * p.D + e] = s;
    }
  } else {
    if (j < np && t == 0) p.d[py * p.gw + px0 + j] = sqrtf(acc);
  }
}

// Sum of the tile partials per component: 64 components per block, 16 interleaved
// slices of the tiles per component, combined in a fixed order.
__global__ __launch_bounds__(1024) void apc_reduce_c(const DensityParams p) {
  __shared__ float part[16][64];
  const int c = threadIdx.x & 63;
  const int e = blockIdx.x * 64 + c;
  const int g = threadIdx.x >> 6;
  float s = 0.f;
  if (e < p.D)
    for (int t = g; t < p.n_tiles; t += 16) s += p.partial[static_cast<long long>(t) * p.D + e];
  part[g][c] = s;
  __syncthreads();
  if (g == 0 && e < p.D) {
    float tot = 0.f;
    for (int i = 0; i < 16; ++i) tot += part[i][c];
    p.csum[e] = tot;
  }
}

__global__ __launch_bounds__(1024) void apc_finalize_c(const DensityParams p) {
  __shared__ float red[16];
  float ss = 0.f;
  const float invN = 1.0f / static_cast<float>(p.N);
  for (int e = threadIdx.x; e < p.D; e += 1024) {
    const float c = p.csum[e] * invN;
    ss += c * c;
  }
  ss = block_reduce<0>(ss, red);
  const float nc = sqrtf(ss);
  const float ic = (nc > 1e-5f) ? 1.0f / nc : 0.f;   // c_hat = 0 when ||c|| is numerically zero
  for (int e = threadIdx.x; e < p.D; e += 1024) p.chat[e] = p.csum[e] * invN * ic;
  if (threadIdx.x == 0) {
    p.stats[0] = ss;          // phi
    p.stats[1] = 1.0f - ss;   // rho_g
    p.stats[2] = nc;
  }
}

__global__ __launch_bounds__(1024) void apc_tail(const DensityParams p) {
  __shared__ uint32_t hist[256 + 8];
  __shared__ float red[16];
  int need = 0;
  // d >= 0, so the raw bit patterns order like the values
  const uint32_t T = block_radix_select(p.N, p.n_tail, [&](int i) { return __float_as_uint(p.d[i]); },
                                        hist, &need);
  float s = 0.f;
  for (int i = threadIdx.x; i < p.N; i += 1024) {
    const float x = p.d[i];
    if (__float_as_uint(x) > T) s += x;
  }
  s = block_reduce<0>(s, red);
  if (threadIdx.x == 0) {
    const float d_top = (s + static_cast<float>(need) * __uint_as_float(T)) / static_cast<float>(p.n_tail);
    const float rho_g = p.stats[1];
    const float rho_d = fminf(d_top / p.gamma, 1.0f);
    p.rho_out[0] = rho_g;
    p.rho_out[1] = rho_d;
    p.rho_out[2] = p.alpha * rho_g + (1.0f - p.alpha) * rho_d;
    p.rho_out[3] = p.stats[0];
  }
}

// ---------------------------------------------------------------- resize
constexpr int kRsTX = 64;    // output columns per workgroup
constexpr int kRsThreads = 256;
constexpr int kRsMaxLds = 64 * 1024;

struct ResizeParams {
  const uint8_t* src;
  uint8_t* dst;
  int H, W, oH, oW;
  int ty;                 // output rows per workgroup
  int tx;                 // output columns per workgroup (<= kRsTX)
  int rows_cap;           // input rows staged per workgroup
  float sx, sy;           // input pixels per output pixel
  float fx, fy;           // kernel stretch (max(1, s))
};

__device__ __forceinline__ float keys_cubic(float x) {
  x = fabsf(x);
  if (x <= 1.f) return (1.5f * x - 2.5f) * x * x + 1.f;              // a = -0.5
  if (x < 2.f) return ((-0.5f * x + 2.5f) * x - 4.f) * x + 2.f;
  return 0.f;
}

// Taps of output coordinate o along an axis of n inputs resized to m outputs.  Input
// pixel i's distance to o's sample point, in kernel units, is
//   ((2i + 1) m - (2o + 1) n) / (2 max(n, m)),
// whose numerator is an exact integer, so the weights carry a single rounding.
struct Taps {
  int lo, hi;        // inclusive tap range (extra taps at |dist| >= 2 weigh 0)
  long long num0;    // numerator at i = lo
  long long step;    // numerator increment per tap (2m)
  float inv_den;     // 1 / (2 max(n, m))
  float inv_sum;     // 1 / sum of the weights
};

__device__ __forceinline__ Taps make_taps(int o, int n, int m) {
  Taps t;
  const long long den = 2ll * (n > m ? n : m);
  // support in input pixels: 2 * max(1, n/m); centre (o + 0.5) n / m
  const float centre = (static_cast<float>(o) + 0.5f) * static_cast<float>(n) / static_cast<float>(m);
  const float support = 2.f * fmaxf(1.f, static_cast<float>(n) / static_cast<float>(m));
  t.lo = max(static_cast<int>(floorf(centre - support - 0.5f)) - 1, 0);
  t.hi = min(static_cast<int>(ceilf(centre + support - 0.5f)) + 1, n - 1);
  t.step = 2ll * m;
  t.num0 = (2ll * t.lo + 1) * m - (2ll * o + 1) * n;
  t.inv_den = 1.f / static_cast<float>(den);
  float sum = 0.f;
  long long num = t.num0;
  for (int i = t.lo; i <= t.hi; ++i, num += t.step) sum += keys_cubic(static_cast<float>(num) * t.inv_den);
  t.inv_sum = 1.f / sum;
  return t;
}

__global__ __launch_bounds__(kRsThreads) void apc_resize(const ResizeParams p) {
  extern __shared__ float hbuf[];   // [rows_cap][tx][3] horizontally filtered rows
  const int ox0 = blockIdx.x * p.tx;
  const int oy0 = blockIdx.y * p.ty;
  const int oy1 = min(p.oH, oy0 + p.ty);
  // input rows needed by this tile's output rows
  const Taps tfirst = make_taps(oy0, p.H, p.oH);
  const Taps tlast = make_taps(oy1 - 1, p.H, p.oH);
  const int ylo = tfirst.lo;
  const int nrows = min(tlast.hi - ylo + 1, p.rows_cap);   // the host sizes rows_cap to fit
  const int ncols = min(p.tx, p.oW - ox0);
  // horizontal pass into LDS
  for (int e = threadIdx.x; e < nrows * ncols; e += kRsThreads) {
    const int r = e / ncols, x = e - r * ncols;
    const Taps t = make_taps(ox0 + x, p.W, p.oW);
    const uint8_t* row = p.src + static_cast<long long>(ylo + r) * p.W * 3;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f;
    long long num = t.num0;
    for (int i = t.lo; i <= t.hi; ++i, num += t.step) {
      const float w = keys_cubic(static_cast<float>(num) * t.inv_den);
      a0 += w * static_cast<float>(row[3 * i + 0]);
      a1 += w * static_cast<float>(row[3 * i + 1]);
      a2 += w * static_cast<float>(row[3 * i + 2]);
    }
    float* h = hbuf + (r * p.tx + x) * 3;
    h[0] = a0 * t.inv_sum; h[1] = a1 * t.inv_sum; h[2] = a2 * t.inv_sum;
  }
  __syncthreads();
  // vertical pass and store
  for (int e = threadIdx.x; e < (oy1 - oy0) * ncols * 3; e += kRsThreads) {
    const int yy = e / (ncols * 3), rem = e - yy * ncols * 3;
    const int x = rem / 3, ch = rem - x * 3;
    const Taps t = make_taps(oy0 + yy, p.H, p.oH);
    float acc = 0.f;
    long long num = t.num0;
    for (int i = t.lo; i <= t.hi; ++i, num += t.step) {
      const int r = i - ylo;
      if (r < 0 || r >= nrows) continue;
      const float w = keys_cubic(static_cast<float>(num) * t.inv_den);
      acc += w * hbuf[(r * p.tx + x) * 3 + ch];
    }
    const float v = floorf(acc * t.inv_sum + 0.5f);
    const int u = static_cast<int>(fminf(fmaxf(v, 0.f), 255.f));
    p.dst[(static_cast<long long>(oy0 + yy) * p.oW + ox0 + x) * 3 + ch] = static_cast<uint8_t>(u);
  }
}

void size_density(Sizer& s, int H, int W, int P) {
  const int gh = H / P, gw = W / P, N = gh * gw, D = 3 * P * P;
  const int tiles = gh * ((gw + kPatchesPerTile - 1) / kPatchesPerTile);
  s.take<float>(N);                              // inv_norm
  s.take<float>(static_cast<size_t>(tiles) * D); // partials
  s.take<float>(D);                              // csum
  s.take<float>(D);                              // chat
  s.take<float>(8);                              // stats
  s.take<float>(N);                              // d (when d_out is null)
}

}  // namespace
}  // namespace pace

using namespace pace;

extern "C" {

size_t pace_apc_density_workspace_size(int H, int W, int patch) {
  if (H <= 0 || W <= 0 || patch <= 0) return 0;
  Sizer s;
  size_density(s, H, W, patch);
  return s.off;
}

pace_status_t pace_apc_density(const uint8_t* img, int H, int W, int patch, double tail_frac,
                               float alpha, float gamma, float* d_out, float* rho_out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(img && rho_out, "pace_apc_density: null device pointer");
  PACE_REQUIRE(patch >= 1 && patch <= kMaxPatch, "pace_apc_density: patch=%d not in [1, %d]", patch,
               kMaxPatch);
  PACE_REQUIRE(H >= patch && W >= patch && H % patch == 0 && W % patch == 0,
               "pace_apc_density: H=%d W=%d must be positive multiples of patch=%d", H, W, patch);
  PACE_REQUIRE(tail_frac > 0 && tail_frac <= 1, "pace_apc_density: tail_frac must be in (0, 1]");
  PACE_REQUIRE(gamma > 0.f, "pace_apc_density: gamma must be > 0");
  const long long N = static_cast<long long>(H / patch) * (W / patch);
  PACE_REQUIRE(N < (1ll << 28), "pace_apc_density: too many patches");
  const size_t need = pace_apc_density_workspace_size(H, W, patch);
  if (workspace == nullptr || workspace_bytes < need)
    return set_error(PACE_ERR_WORKSPACE, "pace_apc_density: workspace %zu < %zu bytes",
                     workspace_bytes, need);
  DensityParams p{};
  p.img = img;
  p.H = H; p.W = W; p.P = patch;
  p.gh = H / patch; p.gw = W / patch; p.N = static_cast<int>(N);
  p.D = 3 * patch * patch;
  p.tiles_x = (p.gw + kPatchesPerTile - 1) / kPatchesPerTile;
  p.n_tiles = p.gh * p.tiles_x;
  int nt = pace_keep_count(tail_frac, p.N);
  p.n_tail = nt < 1 ? 1 : nt;
  p.alpha = alpha; p.gamma = gamma;
  Carver c(workspace, workspace_bytes);
  p.inv_norm = c.take<float>(p.N);
  p.partial = c.take<float>(static_cast<size_t>(p.n_tiles) * p.D);
  p.csum = c.take<float>(p.D);
  p.chat = c.take<float>(p.D);
  p.stats = c.take<float>(8);
  float* dws = c.take<float>(p.N);
  p.d = d_out ? d_out : dws;
  p.rho_out = rho_out;
  const size_t lds = (static_cast<size_t>(patch) * kPatchesPerTile * patch * 3 + kPatchesPerTile +
                      p.D) * sizeof(float);
  hipLaunchKernelGGL(apc_patch_pass<0>, dim3(p.n_tiles), dim3(kApcThreads), lds, stream, p);
  pace_status_t st = check_launch("apc_patch_pass<0>");
  if (st != PACE_OK) return st;
  hipLaunchKernelGGL(apc_reduce_c, dim3((p.D + 63) / 64), dim3(1024), 0, stream, p);
  if ((st = check_launch("apc_reduce_c")) != PACE_OK) return st;
  hipLaunchKernelGGL(apc_finalize_c, dim3(1), dim3(1024), 0, stream, p);
  if ((st = check_launch("apc_finalize_c")) != PACE_OK) return st;
  hipLaunchKernelGGL(apc_patch_pass<1>, dim3(p.n_tiles), dim3(kApcThreads), lds, stream, p);
  if ((st = check_launch("apc_patch_pass<1>")) != PACE_OK) return st;
  hipLaunchKernelGGL(apc_tail, dim3(1), dim3(1024), 0, stream, p);
  return check_launch("apc_tail");
}

pace_status_t pace_apc_downsample(const uint8_t* src, int H, int W, uint8_t* dst, int oH, int oW,
                                  hipStream_t stream) {
  PACE_REQUIRE(src && dst, "pace_apc_downsample: null device pointer");
  PACE_REQUIRE(H >= 1 && W >= 1 && oH >= 1 && oW >= 1 && oH <= H && oW <= W,
               "pace_apc_downsample: sizes %dx%d -> %dx%d must shrink or keep", H, W, oH, oW);
  ResizeParams p{};
  p.src = src; p.dst = dst;
  p.H = H; p.W = W; p.oH = oH; p.oW = oW;
  p.sx = static_cast<float>(static_cast<double>(W) / oW);
  p.sy = static_cast<float>(static_cast<double>(H) / oH);
  p.fx = p.sx > 1.f ? p.sx : 1.f;
  p.fy = p.sy > 1.f ? p.sy : 1.f;
  if (p.fx > 32.f || p.fy > 32.f)
    return set_error(PACE_ERR_UNSUPPORTED, "pace_apc_downsample: shrink factor above 32");
  // rows of input per tile of ty output rows: ty*sy + 4*fy + 5 (generous bound, taps
  // include one extra zero-weight pixel on each side)
  int ty = 16, tx = kRsTX;
  auto rows_for = [&](int t) { return static_cast<int>(ceilf(t * p.sy + 4.f * p.fy)) + 5; };
  auto lds_for = [&](int t, int x) { return static_cast<size_t>(rows_for(t)) * x * 3 * sizeof(float); };
  while (lds_for(ty, tx) > kRsMaxLds) {
    if (ty > 1) ty >>= 1;
    else if (tx > 8) tx >>= 1;
    else return set_error(PACE_ERR_UNSUPPORTED, "pace_apc_downsample: shrink factor too large");
  }
  const size_t lds = lds_for(ty, tx);
  p.ty = ty;
  p.tx = tx;
  p.rows_cap = rows_for(ty);
  dim3 grid((oW + tx - 1) / tx, (oH + ty - 1) / ty);
  hipLaunchKernelGGL(apc_resize, grid, dim3(kRsThreads), lds, stream, p);
  return check_launch("apc_resize");
}

}  // extern "C"
