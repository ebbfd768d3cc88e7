// APC (Section 3.2, "Condense"): per-patch information density of a uint8 image and
// the bicubic resize by sqrt(r) per side (Appendix implementation details).
//
// Density, four launches (all HBM/L2-bound, fixed reduction orders -> deterministic):
//   apc_patch_pass<0>  per patch-strip tile: ||f_i|| -> 1/||f_i|| (from exact integer sums of
//                      the bytes and their squares), and the tile's partial sum of
//                      T_i = f_i/||f_i|| over its patches (one 588-vector per tile)
//   apc_reduce_c       sum of the tile partials per component -> sum_i T_i
//   apc_patch_pass<1>  c = mean T_i, phi = ||c||^2 (equal to Eq. 1's mean pairwise cosine),
//                      rho_g = 1 - phi (Eq. 2) and c_hat = c/||c||, recomputed by every
//                      workgroup from the sums; then d_i = ||T_i - c_hat|| (the image is
//                      re-read, mostly from L2/MALL)
//   apc_tail           the n_tail-th largest d (a value histogram, then the candidates of its
//                      bin ranked), tail mean, rho_d, rho (up to 49,152 distances held in
//                      registers, more re-read from memory)
//
// The per-patch feature is the patch's pixels mapped to x/127.5 - 1 (component order:
// patch row, pixel column, channel).  The order does not change norms or cosines.
#include <math.h>

#include "pace_internal.h"

namespace pace {
namespace {

constexpr int kPatchesPerTile = 64;   // patches of one patch row per workgroup
constexpr int kApcThreads = 256;      // 4 threads per patch for the norms
constexpr int kMaxPatch = 16;

struct DensityParams {
  const uint8_t* img;
  const uint16_t* feat;   // caller-supplied embeddings, bf16 [N, D] (feature entry point)
  const float* featf;     // fp32 [N, D] (pixel-statistic previews)
  int H, W, P;            // image and patch size
  int gh, gw, N;          // patch grid
  int D;                  // 3 * P * P
  int tiles_x;            // tiles per patch row
  int n_tiles;
  int n_tail;
  int row_dwords;         // LDS dwords per staged pixel row
  float alpha, gamma;
  float* inv_norm;        // [N]
  float* partial;         // [n_tiles, D]
  float* csum;            // [D]
  float* chat;            // [D]
  float* stats;           // [8]: phi, rho_g, |c|, ...
  float* d;               // [N]
  float* rho_out;         // [4]
};

// Dword at byte offset a (4-aligned) of a range-checked buffer of `total` bytes.  The plain
// load returns zero for a dword that straddles the end (the range check is per dword), so
// that one dword, the image's last, is assembled from byte loads in a separate fix-up
// after a batch of plain loads (a branch per load would serialise the batch).
__device__ __forceinline__ uint32_t load_dword(__amdgpu_buffer_rsrc_t rs, int a) {
  return __builtin_amdgcn_raw_buffer_load_b32(rs, static_cast<unsigned>(a), 0, 0);
}
__device__ __forceinline__ bool straddles(int a, int total) { return a < total && a + 4 > total; }
__device__ __noinline__ uint32_t load_dword_bytes(__amdgpu_buffer_rsrc_t rs, int a, int total) {
  uint32_t v = 0;
  for (int k = 0; k < 4 && a + k < total; ++k)
    v |= static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b8(rs, static_cast<unsigned>(a + k), 0, 0)) << (8 * k);
  return v;
}

// Stages the tile's pixels (P rows x up to 64 patches) in LDS as bytes, through aligned
// dword loads of a range-checked buffer (reads never leave the image).  Row r of the tile
// starts at byte shift[r] of its LDS row.
__device__ __forceinline__ int stage_tile(const DensityParams& p, int tile, uint32_t* px, int* shift,
                                          int* py_out, int* px0_out) {
  const int py = tile / p.tiles_x;
  const int px0 = (tile % p.tiles_x) * kPatchesPerTile;
  const int np = min(kPatchesPerTile, p.gw - px0);
  const int row_bytes = np * p.P * 3;
  const int total = p.H * p.W * 3;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.img), (short)0, total, 0x00020000);
  const int nd = (row_bytes + 3) / 4 + 1;   // <= 4 * kApcThreads dwords per row
  // eight rows at a time (P <= 16: one or two batches), all of a thread's loads of a batch in
  // flight before its LDS writes
#pragma unroll
  for (int r0 = 0; r0 < kMaxPatch; r0 += 8) {
    if (r0 >= p.P) break;
    uint32_t v[8][4];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = r0 + q;
      const int a0 = ((py * p.P + r) * p.W * 3 + px0 * p.P * 3) & ~3;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int dd = static_cast<int>(threadIdx.x) + u * kApcThreads;
        v[q][u] = (r < p.P && dd < nd) ? load_dword(rs, a0 + 4 * dd) : 0u;
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int a0 = ((py * p.P + r0 + q) * p.W * 3 + px0 * p.P * 3) & ~3;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int a = a0 + 4 * (static_cast<int>(threadIdx.x) + u * kApcThreads);
        if (r0 + q < p.P && straddles(a, total)) v[q][u] = load_dword_bytes(rs, a, total);
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int r = r0 + q;
      if (r < p.P) {
        const int b0 = (py * p.P + r) * p.W * 3 + px0 * p.P * 3;
        if (threadIdx.x == 0) shift[r] = b0 - (b0 & ~3);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int dd = static_cast<int>(threadIdx.x) + u * kApcThreads;
          if (dd < nd) px[r * p.row_dwords + dd] = v[q][u];
        }
      }
    }
  }
  *py_out = py;
  *px0_out = px0;
  return np;
}

// Feature value of a staged byte: x/127.5 - 1.
__device__ __forceinline__ float feat_of(uint8_t b) { return static_cast<float>(b) * (1.0f / 127.5f) - 1.0f; }

// Feature component e = (patch row r, byte cb within the patch row: pixel column, channel)
// of a tile's patches; patch j of the tile starts at byte j * 3P of each staged row.
template <int PASS>
__global__ __launch_bounds__(kApcThreads) void apc_patch_pass(const DensityParams p) {
  extern __shared__ __align__(16) uint32_t lds[];
  uint32_t* px = lds;                                             // [P][row_dwords]
  float* inv = reinterpret_cast<float*>(px + p.P * p.row_dwords);  // [64]
  float* chat = inv + kPatchesPerTile;   // pass 1: c_hat as [P][cstride] (+12 floats of slack)
  const int pb = 3 * p.P;                // bytes of one patch row
  const int cstride = (pb + 3) & ~3;
  __shared__ int shift[kMaxPatch];
  __shared__ float red[kApcThreads / 64];
  const int tile = blockIdx.x;
  // pass 1: the component sums of sum_i T_i (D <= 3 * 16^2, three per thread), requested
  // before the tile so that their loads fly with the tile's
  constexpr int kCPer = (3 * kMaxPatch * kMaxPatch + kApcThreads - 1) / kApcThreads;
  float cs[kCPer];
  if (PASS == 1) {
#pragma unroll
    for (int k = 0; k < kCPer; ++k) {
      const int e = static_cast<int>(threadIdx.x) + k * kApcThreads;
      cs[k] = e < p.D ? p.csum[e] : 0.f;
    }
  }
  const int j = threadIdx.x >> 2, t = threadIdx.x & 3;
  float s_inv = 0.f;   // pass 1: 1/||f|| of the thread's patch, requested before the tile
  if (PASS == 1) {
    const int px0_ = (tile % p.tiles_x) * kPatchesPerTile;
    if (j < min(kPatchesPerTile, p.gw - px0_)) s_inv = p.inv_norm[(tile / p.tiles_x) * p.gw + px0_ + j];
  }
  int py, px0;
  const int np = stage_tile(p, tile, px, shift, &py, &px0);
  if (PASS == 1) {
    // c = mean_i T_i and phi = ||c||^2 (equal to Eq. 1's mean pairwise cosine), summed by
    // every workgroup in the same fixed order, so that all get the same c_hat
    const float invN = 1.0f / static_cast<float>(p.N);
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < kCPer; ++k) {
      const int e = static_cast<int>(threadIdx.x) + k * kApcThreads;
      const float c = cs[k] * invN;
      if (e < p.D) chat[(e / pb) * cstride + e % pb] = c;
      ss += c * c;
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  }
  __syncthreads();
  if (PASS == 1) {
    float ss = red[0];
#pragma unroll
    for (int i = 1; i < kApcThreads / 64; ++i) ss += red[i];
    const float nc = sqrtf(ss);
    const float ic = (nc > 1e-5f) ? 1.0f / nc : 0.f;   // c_hat = 0 when ||c|| is numerically zero
#pragma unroll
    for (int k = 0; k < kCPer; ++k) {
      const int e = static_cast<int>(threadIdx.x) + k * kApcThreads;
      if (e < p.D) chat[(e / pb) * cstride + e % pb] *= ic;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      p.stats[0] = ss;          // phi
      p.stats[1] = 1.0f - ss;   // rho_g (Eq. 2)
      p.stats[2] = nc;
    }
    __syncthreads();
  }
  const uint8_t* pxb = reinterpret_cast<const uint8_t*>(px);
  const int rb = p.row_dwords * 4;
  // Thread t of patch j takes bytes [12t, 12t + nb) of each of the patch's rows (nb <= 12, as a
  // patch row has at most 48 bytes): four dword reads cover them, realigned with alignbyte, so a
  // row costs a few LDS reads instead of one per byte.  The row's first byte sits at byte
  // (row start & 3) of its staged LDS row.
  const int c0 = 12 * t;
  const int nb = min(12, pb - c0);
  auto row_bytes = [&](int r, uint32_t x[3]) __attribute__((always_inline)) {
    const int b0 = (py * p.P + r) * p.W * 3 + px0 * pb;
    const int o = r * rb + (b0 & 3) + j * pb + c0;
    const uint32_t* wp = px + (o >> 2);
    const uint32_t w0 = wp[0], w1 = wp[1], w2 = wp[2], w3 = wp[3];
    const int al = o & 3;
    x[0] = __builtin_amdgcn_alignbyte(w1, w0, al);
    x[1] = __builtin_amdgcn_alignbyte(w2, w1, al);
    x[2] = __builtin_amdgcn_alignbyte(w3, w2, al);
  };
  if (PASS == 0) {
    // ||f||^2 = sum (b/127.5 - 1)^2 = (4 sum b^2 - 1020 sum b + 65025 D) / 65025, from exact
    // integer sums of b^2 and b (packed-byte dot products; bytes past nb masked off)
    uint32_t sq = 0u, sm = 0u;
    if (j < np && nb > 0) {
      uint32_t keep[3];
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const int v = min(max(nb - 4 * k, 0), 4);
        keep[k] = v >= 4 ? 0xffffffffu : ((1u << (8 * v)) - 1u);
      }
#pragma unroll 2
      for (int r = 0; r < p.P; ++r) {
        uint32_t x[3];
        row_bytes(r, x);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          const uint32_t w = x[k] & keep[k];
          sq = __builtin_amdgcn_udot4(w, w, sq, false);
          sm = __builtin_amdgcn_udot4(w, 0x01010101u, sm, false);
        }
      }
    }
    sq += __shfl_xor(sq, 1, 64);
    sq += __shfl_xor(sq, 2, 64);
    sm += __shfl_xor(sm, 1, 64);
    sm += __shfl_xor(sm, 2, 64);
    if (j < np && t == 0) {
      const int num = 4 * static_cast<int>(sq) - 1020 * static_cast<int>(sm) + 65025 * p.D;
      const float in = 255.0f / sqrtf(static_cast<float>(num));
      inv[j] = in;
      p.inv_norm[py * p.gw + px0 + j] = in;
    }
    __syncthreads();
    // tile partial of sum_i T_i, patches added in index order
    for (int e = threadIdx.x; e < p.D; e += kApcThreads) {
      const int r = e / pb, cb = e - r * pb;
      const uint8_t* col = pxb + r * rb + shift[r] + cb;
      float sum = 0.f;
#pragma unroll 8
      for (int jj = 0; jj < np; ++jj) sum += feat_of(col[jj * pb]) * inv[jj];
      p.partial[static_cast<long long>(tile) * p.D + e] = sum;
    }
  } else {
    // d_i^2 = sum_e (f_e s - c_hat_e)^2 over the thread's bytes of every row, in row order
    float acc = 0.f;
    if (j < np && nb > 0) {
#pragma unroll 2
      for (int r = 0; r < p.P; ++r) {
        uint32_t x[3];
        row_bytes(r, x);
        // 12 values from the thread's first column (the ones past nb, read from the next row or
        // the slack, are not used)
        const float4* cr = reinterpret_cast<const float4*>(chat + r * cstride + c0);
        const float4 ca = cr[0], cb = cr[1], cc = cr[2];
        const float cv[12] = {ca.x, ca.y, ca.z, ca.w, cb.x, cb.y, cb.z, cb.w, cc.x, cc.y, cc.z, cc.w};
#pragma unroll
        for (int i = 0; i < 12; ++i) {
          const float y = feat_of(static_cast<uint8_t>(x[i >> 2] >> (8 * (i & 3)))) * s_inv - cv[i];
          acc += (i < nb) ? y * y : 0.f;
        }
      }
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    if (j < np && t == 0) p.d[py * p.gw + px0 + j] = sqrtf(acc);
  }
}

// ---------------------------------------------------------------- caller-supplied embeddings
// Density of bf16 embeddings x [N, D] (the first vision block's output in the paper's
// preview): T_i = x_i / max(||x_i||, 1e-12).  Two passes over the matrix:
//   apc_feat_pass<0>  per block of 64 rows: each wave takes 16 rows, values spread over its
//                     lanes, for 1/||x_i||; then each thread sums its columns (8-column chunks
//                     when rows are 16-byte vectors) of x_i / ||x_i|| over the block's rows
//                     (L2-resident) -> the block partial
//   apc_feat_pass<1>  one wave per row: d_i = ||x_i / ||x_i|| - c_hat||
// The partials then go through apc_reduce_c, apc_finalize_c (c, phi and c_hat once, as pass 1
// here has a small workgroup per row) and apc_tail.
constexpr int kFeatRows = 64;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

struct FeatAdd { __device__ float operator()(float a, float b) const { return a + b; } };

// Element access: kFeatBf16Vec reads bf16 rows as 16-byte chunks of 8 values (D a multiple of
// 8, aligned rows); kFeatBf16 and kFeatF32 read value by value.
constexpr int kFeatBf16 = 0, kFeatBf16Vec = 1, kFeatF32 = 2;

template <int PASS, int MODE>
__global__ __launch_bounds__(256) void apc_feat_pass(const DensityParams p) {
  constexpr bool VEC = MODE == kFeatBf16Vec;
  __shared__ float inv[kFeatRows];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nchunk = p.D / 8;
  auto at = [&](long long idx) -> float {
    if constexpr (MODE == kFeatF32) return p.featf[idx];
    else return __uint_as_float(static_cast<uint32_t>(p.feat[idx]) << 16);
  };
  if (PASS == 0) {
    const int r0 = blockIdx.x * kFeatRows;
    for (int rr = w; rr < kFeatRows; rr += 4) {
      const int i = r0 + rr;
      float ss = 0.f;
      if (i < p.N) {
        if constexpr (VEC) {
          const uint4* row = reinterpret_cast<const uint4*>(p.feat + static_cast<long long>(i) * p.D);
          for (int c = lane; c < nchunk; c += 64) {
            const uint4 v = row[c];
            const float a[8] = {bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y),
                                bf16_lo(v.z), bf16_hi(v.z), bf16_lo(v.w), bf16_hi(v.w)};
#pragma unroll
            for (int k = 0; k < 8; ++k) ss += a[k] * a[k];
          }
        } else {
          for (int e = lane; e < p.D; e += 64) {
            const float a = at(static_cast<long long>(i) * p.D + e);
            ss += a * a;
          }
        }
      }
      ss = wave_reduce_dpp(ss, FeatAdd{});
      if (lane == 0) {
        const float in = (i < p.N) ? 1.0f / fmaxf(sqrtf(ss), 1e-12f) : 0.f;
        inv[rr] = in;
        if (i < p.N) p.inv_norm[i] = in;
      }
    }
    __syncthreads();
    // block partial of sum_i T_i, rows added in index order
    const int nrows = min(kFeatRows, p.N - r0);
    float* part = p.partial + static_cast<long long>(blockIdx.x) * p.D;
    if constexpr (VEC) {
      for (int c = threadIdx.x; c < nchunk; c += 256) {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        const uint4* col = reinterpret_cast<const uint4*>(p.feat + static_cast<long long>(r0) * p.D) + c;
#pragma unroll 4
        for (int rr = 0; rr < nrows; ++rr) {
          const uint4 v = col[static_cast<long long>(rr) * nchunk];
          const float s = inv[rr];
          acc[0] += bf16_lo(v.x) * s; acc[1] += bf16_hi(v.x) * s;
          acc[2] += bf16_lo(v.y) * s; acc[3] += bf16_hi(v.y) * s;
          acc[4] += bf16_lo(v.z) * s; acc[5] += bf16_hi(v.z) * s;
          acc[6] += bf16_lo(v.w) * s; acc[7] += bf16_hi(v.w) * s;
        }
        float4* out = reinterpret_cast<float4*>(part + c * 8);
        out[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        out[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
      }
    } else {
      for (int e = threadIdx.x; e < p.D; e += 256) {
        float acc = 0.f;
#pragma unroll 4
        for (int rr = 0; rr < nrows; ++rr) acc += at(static_cast<long long>(r0 + rr) * p.D + e) * inv[rr];
        part[e] = acc;
      }
    }
  } else {
    const int i = blockIdx.x * 4 + w;
    if (i >= p.N) return;
    const float s = p.inv_norm[i];
    float acc = 0.f;
    if constexpr (VEC) {
      const uint4* row = reinterpret_cast<const uint4*>(p.feat + static_cast<long long>(i) * p.D);
      const float4* ch = reinterpret_cast<const float4*>(p.chat);
      for (int c = lane; c < nchunk; c += 64) {
        const uint4 v = row[c];
        const float4 c0 = ch[2 * c], c1 = ch[2 * c + 1];
        const float a[8] = {bf16_lo(v.x) * s - c0.x, bf16_hi(v.x) * s - c0.y, bf16_lo(v.y) * s - c0.z,
                            bf16_hi(v.y) * s - c0.w, bf16_lo(v.z) * s - c1.x, bf16_hi(v.z) * s - c1.y,
                            bf16_lo(v.w) * s - c1.z, bf16_hi(v.w) * s - c1.w};
#pragma unroll
        for (int k = 0; k < 8; ++k) acc += a[k] * a[k];
      }
    } else {
      for (int e = lane; e < p.D; e += 64) {
        const float a = at(static_cast<long long>(i) * p.D + e) * s - p.chat[e];
        acc += a * a;
      }
    }
    acc = wave_reduce_dpp(acc, FeatAdd{});
    if (lane == 0) p.d[i] = sqrtf(acc);
  }
}

// ---------------------------------------------------------------- pixel-statistic previews
// Training-free preview vectors per patch (the preview ablation of Section 4), one wave per
// patch, written as fp32 rows of out [N, dim]:
//   kind 0  RGB statistics: channel means and population std of x/255           dim 6
//   kind 1  colour entropy terms -p_k ln p_k over 64 colours (4 levels/channel)  dim 64
//   kind 2  Sobel magnitude of the grey image summed per orientation octant,
//           / (255 P^2)                                                          dim 8
//   kind 3  4-neighbour Laplacian of the grey image / 255                        dim P^2
// Grey is held as the exact integer 1000 x grey = 299 R + 587 G + 114 B, so gradients, the
// Laplacian and the octant decisions are exact integer arithmetic; neighbours cross patch
// borders and the image edge is clamped.
constexpr int kPixMaxPatch = 16;
constexpr int kPixMaxPix = kPixMaxPatch * kPixMaxPatch / 64;   // pixels per lane

struct PixelParams {
  const uint8_t* img;
  int H, W, P, gw, N, kind, dim;
  float* out;
};

__host__ __device__ inline int pixel_feature_dim(int kind, int P) {
  return kind == 0 ? 6 : kind == 1 ? 64 : kind == 2 ? 8 : P * P;
}

// Octant 0..7 of the angle of (gx, gy), 45-degree sectors counter-clockwise from +x (y down
// the rows), decided by integer comparisons; (0, 0) is octant 0.
__device__ __forceinline__ int sobel_octant(int gx, int gy) {
  const int ax = abs(gx), ay = abs(gy);
  if (gx > 0 && gy >= 0) return ay < ax ? 0 : 1;
  if (gx <= 0 && gy > 0) return ax <= ay ? 2 : 3;
  if (gx < 0 && gy <= 0) return ay < ax ? 4 : 5;
  if (gx >= 0 && gy < 0) return ax <= ay ? 6 : 7;
  return 0;
}

__global__ __launch_bounds__(64) void apc_pixel_features(const PixelParams p) {
  __shared__ int grey[(kPixMaxPatch + 2) * (kPixMaxPatch + 2)];
  __shared__ int hist[64];
  const int i = blockIdx.x;
  const int lane = threadIdx.x;
  const int P = p.P, P2 = P * P;
  const int y0 = (i / p.gw) * P, x0 = (i % p.gw) * P;
  float* out = p.out + static_cast<long long>(i) * p.dim;
  auto pixel = [&](int y, int x) -> const uint8_t* { return p.img + (static_cast<long long>(y) * p.W + x) * 3; };

  if (p.kind <= 1) {
    uint32_t px[kPixMaxPix];
#pragma unroll
    for (int k = 0; k < kPixMaxPix; ++k) {
      const int t = lane + 64 * k;
      px[k] = 0;
      if (t < P2) {
        const uint8_t* q = pixel(y0 + t / P, x0 + t % P);
        px[k] = q[0] | (q[1] << 8) | (q[2] << 16);
      }
    }
    if (p.kind == 0) {
      float s[3] = {0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < kPixMaxPix; ++k)
        if (lane + 64 * k < P2)
#pragma unroll
          for (int c = 0; c < 3; ++c) s[c] += static_cast<float>((px[k] >> (8 * c)) & 255u);
      float mean[3], v[3] = {0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 3; ++c) mean[c] = wave_reduce_dpp(s[c], FeatAdd{}) / static_cast<float>(P2);
#pragma unroll
      for (int k = 0; k < kPixMaxPix; ++k)
        if (lane + 64 * k < P2)
#pragma unroll
          for (int c = 0; c < 3; ++c) {
            const float dv = static_cast<float>((px[k] >> (8 * c)) & 255u) - mean[c];
            v[c] += dv * dv;
          }
#pragma unroll
      for (int c = 0; c < 3; ++c) v[c] = wave_reduce_dpp(v[c], FeatAdd{});
      if (lane < 6) {
        const int c = lane % 3;
        const float m = c == 0 ? mean[0] : c == 1 ? mean[1] : mean[2];
        const float vv = c == 0 ? v[0] : c == 1 ? v[1] : v[2];
        out[lane] = lane < 3 ? m / 255.f : sqrtf(vv / static_cast<float>(P2)) / 255.f;
      }
    } else {
      hist[lane] = 0;
      __syncthreads();
#pragma unroll
      for (int k = 0; k < kPixMaxPix; ++k)
        if (lane + 64 * k < P2) {
          const uint32_t u = px[k];
          const int colour = ((u & 255u) >> 6) * 16 + (((u >> 8) & 255u) >> 6) * 4 + (((u >> 16) & 255u) >> 6);
          atomicAdd(&hist[colour], 1);
        }
      __syncthreads();
      const int cnt = hist[lane];
      const float pk = static_cast<float>(cnt) / static_cast<float>(P2);
      out[lane] = cnt > 0 ? -pk * logf(pk) : 0.f;
    }
    return;
  }

  const int G = P + 2;
  for (int t = lane; t < G * G; t += 64) {
    const int y = min(max(y0 - 1 + t / G, 0), p.H - 1);
    const int x = min(max(x0 - 1 + t % G, 0), p.W - 1);
    const uint8_t* q = pixel(y, x);
    grey[t] = 299 * q[0] + 587 * q[1] + 114 * q[2];
  }
  __syncthreads();
  auto g = [&](int r, int c) { return grey[(r + 1) * G + (c + 1)]; };   // patch coordinates
  if (p.kind == 3) {
    for (int t = lane; t < P2; t += 64) {
      const int r = t / P, c = t % P;
      const int lap = 4 * g(r, c) - g(r - 1, c) - g(r + 1, c) - g(r, c - 1) - g(r, c + 1);
      out[t] = static_cast<float>(lap) / 255000.f;
    }
    return;
  }
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int t = lane; t < P2; t += 64) {
    const int r = t / P, c = t % P;
    const int gx = (g(r - 1, c + 1) + 2 * g(r, c + 1) + g(r + 1, c + 1)) -
                   (g(r - 1, c - 1) + 2 * g(r, c - 1) + g(r + 1, c - 1));
    const int gy = (g(r + 1, c - 1) + 2 * g(r + 1, c) + g(r + 1, c + 1)) -
                   (g(r - 1, c - 1) + 2 * g(r - 1, c) + g(r - 1, c + 1));
    const float mag = static_cast<float>(sqrt(static_cast<double>(gx) * gx + static_cast<double>(gy) * gy));
    const int o = sobel_octant(gx, gy);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += (o == k) ? mag : 0.f;
  }
  const float scale = 1.f / (1000.f * 255.f * static_cast<float>(P2));
  float mine = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float tot = wave_reduce_dpp(acc[k], FeatAdd{});
    if (lane == k) mine = tot * scale;
  }
  if (lane < 8) out[lane] = mine;
}

// Sum of the tile partials per component: 64 components per block, 16 interleaved
// slices of the tiles per component, combined in a fixed order.
__global__ __launch_bounds__(1024) void apc_reduce_c(const DensityParams p) {
  __shared__ float part[16][64];
  const int c = threadIdx.x & 63;
  const int e = blockIdx.x * 64 + c;
  const int g = threadIdx.x >> 6;
  float s = 0.f;
  if (e < p.D) {
    // eight tiles' loads in flight, added in tile order
    for (int t0 = g; t0 < p.n_tiles; t0 += 16 * 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = t0 + 16 * u;
        v[u] = t < p.n_tiles ? p.partial[static_cast<long long>(t) * p.D + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
  }
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

constexpr int kTailR = 48;       // most distances per thread held in registers: up to 49,152 patches
constexpr int kTailBins = 4096;  // value bins over [0, 2], the range of d
constexpr int kTailCand = 256;   // candidates ranked by direct comparison

struct TailAdd { __device__ float operator()(float a, float b) const { return a + b; } };

// Sum of the n_tail largest distances, then rho_d and rho.  d >= 0, so the raw bit patterns
// order like the values.  With the distances in registers (thread t holds patches
// j * 1024 + t, j < R; R = 4, 16, 32, 44 or 48, the fewest that hold the patch count, so that
// smaller images do not walk 48 slots per thread): a histogram of floor(d * 2048) (monotone
// in d, clamped), the bin b* that
// holds the n_tail-th largest value, the threshold T (the need-th largest key in bin b*,
// by direct comparison among the bin's few candidates, or a radix select when it holds
// many ties), and sum = (sum of d > T) + need_eq * T, reduced in a fixed order.
template <int R>
__global__ __launch_bounds__(1024) void apc_tail(const DensityParams p) {
  __shared__ __align__(16) uint32_t hist[kTailBins];
  __shared__ uint32_t rhist[4 * 256];
  __shared__ uint32_t cand_key[kTailCand];
  __shared__ int cand_idx[kTailCand];
  __shared__ __align__(16) uint32_t wt[16];
  __shared__ uint32_t misc[8];   // 0: b*, 1: need, 2: candidates, 3: T, 4: need_eq, 5-6: radix
  __shared__ float red[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  uint32_t T;
  int need_eq;
  float s = 0.f;
  if (p.N <= 1024 * R) {
    // Slots past N read as +0 (range-checked loads), the smallest possible distance.  They
    // are counted into bin 0 at once, not one contended atomic each, and take part in every
    // later step as ordinary zeros: as n_tail <= N, the top n_tail values, T and the sum are
    // those of the N distances (a tie at 0 adds 0), and no step needs a per-slot range test.
    const uint32_t pad = static_cast<uint32_t>(1024 * R - p.N);
    for (int i = tid; i < kTailBins; i += 1024) hist[i] = i == 0 ? pad : 0u;
    rhist[tid] = 0u;
    if (tid < 8) misc[tid] = 0u;
    uint32_t key[R];
    const auto rd = range_rsrc(p.d, static_cast<unsigned>(p.N) * 4u);
#pragma unroll
    for (int j = 0; j < R; ++j)
      key[j] = __float_as_uint(rload_f32(rd, static_cast<unsigned>(j * 1024 + tid) * 4u));
    __syncthreads();
    const int jfull = p.N >> 10;
    const bool rem_live = tid < (p.N & 1023);
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int bin = static_cast<int>(fminf(__uint_as_float(key[j]) * 2048.f, static_cast<float>(kTailBins - 1)));
      if (j < jfull || (j == jfull && rem_live)) atomicAdd(&hist[bin], 1u);
    }
    __syncthreads();
    // thread t covers bins 4095 - 4t down to 4092 - 4t (descending)
    {
      const int bhi = kTailBins - 1 - 4 * tid;
      const uint4 h4 = *reinterpret_cast<const uint4*>(&hist[bhi - 3]);
      const uint32_t cs[4] = {h4.w, h4.z, h4.y, h4.x};
      const uint32_t tot = cs[0] + cs[1] + cs[2] + cs[3];
      const uint32_t incl = wave_incl_scan(tot);
      if (lane == 63) wt[w] = incl;
      __syncthreads();
      uint32_t before = incl - tot;
      for (int i = 0; i < w; ++i) before += wt[i];
      const uint32_t K = static_cast<uint32_t>(p.n_tail);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (before < K && before + cs[q] >= K) { misc[0] = bhi - q; misc[1] = K - before; }
        before += cs[q];
      }
    }
    __syncthreads();
    const int bstar = static_cast<int>(misc[0]);
    const int need = static_cast<int>(misc[1]);   // 1 <= need <= count of bin b*
    // d * 2048 is exact, so bin b* holds exactly the keys in [b*/2048, (b*+1)/2048), the
    // last bin everything from 4095/2048 up
    const uint32_t lo = __float_as_uint(static_cast<float>(bstar) * (1.f / 2048.f));
    const uint32_t span = (bstar == kTailBins - 1) ? 0xffffffffu - lo
                          : __float_as_uint(static_cast<float>(bstar + 1) * (1.f / 2048.f)) - lo;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      if (key[j] - lo < span) {
        const uint32_t slot = atomicAdd(&misc[2], 1u);
        if (slot < static_cast<uint32_t>(kTailCand)) { cand_key[slot] = key[j]; cand_idx[slot] = j * 1024 + tid; }
      }
    }
    __syncthreads();
    const uint32_t ncand = misc[2];
    if (ncand <= 64u) {
      // one wave ranks up to 64 candidates, one per lane, the others' keys read by lane index
      if (w == 0) {
        const bool mine = lane < static_cast<int>(ncand);
        const uint32_t kt = mine ? cand_key[lane] : 0u;
        const int it = mine ? cand_idx[lane] : 0;
        int rank = 0, greater = 0;
        for (uint32_t u = 0; u < ncand; ++u) {
          const uint32_t ku = __builtin_amdgcn_readlane(kt, u);
          const int iu = __builtin_amdgcn_readlane(it, u);
          rank += (ku > kt || (ku == kt && iu < it)) ? 1 : 0;
          greater += ku > kt ? 1 : 0;
        }
        if (mine && rank == need - 1) { misc[3] = kt; misc[4] = static_cast<uint32_t>(need - greater); }
      }
    } else if (ncand <= static_cast<uint32_t>(kTailCand)) {
      if (tid < static_cast<int>(ncand)) {
        const uint32_t kt = cand_key[tid];
        const int it = cand_idx[tid];
        int rank = 0, greater = 0;
#pragma unroll 8
        for (uint32_t u = 0; u < ncand; ++u) {
          const uint32_t ku = cand_key[u];
          rank += (ku > kt || (ku == kt && cand_idx[u] < it)) ? 1 : 0;
          greater += ku > kt ? 1 : 0;
        }
        if (rank == need - 1) { misc[3] = kt; misc[4] = static_cast<uint32_t>(need - greater); }
      }
    } else {
      // many equal distances in one bin: radix select over the candidates' keys (+1, so
      // that every candidate ranks above the others' 0)
      uint32_t ck[R];
#pragma unroll
      for (int j = 0; j < R; ++j) ck[j] = (key[j] - lo < span) ? key[j] + 1u : 0u;
      int ne = 0;
      const uint32_t T1 = radix_select_prezeroed<R, true>(ck, 1024 * R, need, rhist, &misc[5], &ne);
      if (tid == 0) { misc[3] = T1 - 1u; misc[4] = static_cast<uint32_t>(ne); }
    }
    __syncthreads();
    T = misc[3];
    need_eq = static_cast<int>(misc[4]);
#pragma unroll
    for (int j = 0; j < R; ++j)
      if (key[j] > T) s += __uint_as_float(key[j]);
  } else {
    int need = 0;
    T = block_radix_select(p.N, p.n_tail, [&](int i) { return __float_as_uint(p.d[i]); }, rhist, &need);
    need_eq = need;
    for (int i = tid; i < p.N; i += 1024) {
      const float x = p.d[i];
      if (__float_as_uint(x) > T) s += x;
    }
  }
  s = wave_reduce_dpp(s, TailAdd{});
  if (lane == 0) red[w] = s;
  __syncthreads();
  if (tid == 0) {
    float tot = 0.f;
    for (int i = 0; i < 16; ++i) tot += red[i];
    const float d_top = (tot + static_cast<float>(need_eq) * __uint_as_float(T)) / static_cast<float>(p.n_tail);
    const float rho_g = p.stats[1];
    const float rho_d = fminf(d_top / p.gamma, 1.0f);
    p.rho_out[0] = rho_g;
    p.rho_out[1] = rho_d;
    p.rho_out[2] = p.alpha * rho_g + (1.0f - p.alpha) * rho_d;
  }
}

// The tail kernel for p.N distances: the fewest registers per thread that hold them all, or
// the largest form (which re-reads them from memory beyond 49,152).
void launch_tail(const DensityParams& p, hipStream_t stream) {
  if (p.N <= 1024 * 4) hipLaunchKernelGGL(apc_tail<4>, dim3(1), dim3(1024), 0, stream, p);
  else if (p.N <= 1024 * 16) hipLaunchKernelGGL(apc_tail<16>, dim3(1), dim3(1024), 0, stream, p);
  else if (p.N <= 1024 * 32) hipLaunchKernelGGL(apc_tail<32>, dim3(1), dim3(1024), 0, stream, p);
  else if (p.N <= 1024 * 44) hipLaunchKernelGGL(apc_tail<44>, dim3(1), dim3(1024), 0, stream, p);
  else hipLaunchKernelGGL(apc_tail<kTailR>, dim3(1), dim3(1024), 0, stream, p);
}

// ---------------------------------------------------------------- resize
// One workgroup per output tile of ty x tx pixels.  It computes the tile's column and row
// tap weights once (LDS), stages the input region it needs (range-checked dword loads,
// so reads never leave the image), runs the horizontal pass into LDS in fp32 and the
// vertical pass straight to the output.  Shrinks beyond 32x per side, whose spans do not fit
// a staged tile, take apc_resize_direct (one workgroup per output pixel).
constexpr int kRsThreads = 256;
constexpr int kRsMaxLds = 64 * 1024;

struct ResizeParams {
  const uint8_t* src;
  uint8_t* dst;
  int H, W, oH, oW;
  int ty, tx;             // output rows / columns per workgroup
  float rx, ry;           // W / oW and H / oH (register path: per-axis constants set on the host)
  float invdx, invdy;     // 1 / (2 max(W, oW)) and 1 / (2 max(H, oH))
  int ntx, nty;           // tap slots per output column / row (upper bound of the tap count)
  int rows_cap;           // input rows staged per workgroup
  int cols_cap;           // input columns staged per workgroup
  int row_dwords;         // LDS dwords per staged input row
  // LDS carve (in 4-byte words)
  int o_wx, o_wy, o_lox, o_loy, o_pix, o_h;
};

__device__ __forceinline__ float keys_cubic(float x) {
  x = fabsf(x);
  if (x <= 1.f) return (1.5f * x - 2.5f) * x * x + 1.f;              // a = -0.5
  if (x < 2.f) return ((-0.5f * x + 2.5f) * x - 4.f) * x + 2.f;
  return 0.f;
}

// Taps of output coordinate o along an axis of n inputs resized to m outputs: input i's
// distance to o's sample point in kernel units is ((2i+1) m - (2o+1) n) / (2 max(n, m)); its
// numerator is an exact integer, so every weight carries a single rounding.  Writes
// normalised weights for inputs lo .. lo+count-1, the span from the first to the last
// nonzero weight within `slots` candidates (zero past the image or the support), and
// returns lo (count in *count).
__device__ __forceinline__ int make_taps(int o, int n, int m, int slots, float* w, int* count) {
  const float centre = (static_cast<float>(o) + 0.5f) * static_cast<float>(n) / static_cast<float>(m);
  const float support = 2.f * fmaxf(1.f, static_cast<float>(n) / static_cast<float>(m));
  const int lo = max(static_cast<int>(floorf(centre - support - 0.5f)) - 1, 0);
  const float inv_den = 1.f / static_cast<float>(2ll * (n > m ? n : m));
  long long num = (2ll * lo + 1) * m - (2ll * o + 1) * n;
  float sum = 0.f;
  for (int j = 0; j < slots; ++j, num += 2ll * m) {
    const float wt = (lo + j < n) ? keys_cubic(static_cast<float>(num) * inv_den) : 0.f;
    w[j] = wt;
    sum += wt;
  }
  const float inv = 1.f / sum;
  int j0 = 0, j1 = slots - 1;
  while (j0 < j1 && w[j0] == 0.f) ++j0;
  while (j1 > j0 && w[j1] == 0.f) --j1;
  for (int j = j0; j <= j1; ++j) w[j - j0] = w[j] * inv;
  for (int j = j1 - j0 + 1; j < slots; ++j) w[j] = 0.f;
  *count = j1 - j0 + 1;
  return lo + j0;
}

// make_taps spread over a row of 16 lanes, lane j holding candidate j (slots <= 16): every
// lane of the row evaluates one weight, the row's sum comes from a butterfly (every lane ends
// with the same bits) and the first and last nonzero candidates from a ballot.  The same
// weights, lo and count as make_taps up to the order of the normalising sum.  All 64 lanes
// of the wave must call it together (`valid` false for rows of 16 with no coordinate); the
// distance numerator is formed in 32 bits when 2 n m fits, which makes the same float.
constexpr int kRegTaps = 16;
// keys_cubic without branches (both pieces evaluated, then selected): the same values
__device__ __forceinline__ float keys_cubic_sel(float x) {
  x = fabsf(x);
  const float a = (1.5f * x - 2.5f) * x * x + 1.f;
  const float b = ((-0.5f * x + 2.5f) * x - 4.f) * x + 2.f;
  return x <= 1.f ? a : (x < 2.f ? b : 0.f);
}
// ratio = n / m and inv_den = 1 / (2 max(n, m)) come from the host.  The first candidate lo may
// sit one sample off the one make_taps finds (the centre rounds differently), but the 16
// candidates still cover the support, whose weights come from the same exact numerators.
__device__ __forceinline__ void make_taps_row16(int o, bool valid, int n, int m, int slots, float ratio,
                                                float inv_den, float* w_out, int* lo_out, int* count_out) {
  const int lane = threadIdx.x & 63, j = lane & 15;
  const float centre = (static_cast<float>(o) + 0.5f) * ratio;
  const float support = 2.f * fmaxf(1.f, ratio);
  const int lo = max(static_cast<int>(floorf(centre - support - 0.5f)) - 1, 0);
  float wt = 0.f;
  if (valid && j < slots && lo + j < n) {
    float num;
    if (2ll * n * m < (1ll << 31))
      num = static_cast<float>((2 * (lo + j) + 1) * m - (2 * o + 1) * n);
    else
      num = static_cast<float>((2ll * (lo + j) + 1) * m - (2ll * o + 1) * n);
    wt = keys_cubic_sel(num * inv_den);
  }
  float sum = wt;
  sum += dpp_f32<kDppQuadXor1>(sum);
  sum += dpp_f32<kDppQuadXor2>(sum);
  sum += dpp_f32<kDppRowHalfMirror>(sum);
  sum += dpp_f32<kDppRowMirror>(sum);
  const uint32_t bits = static_cast<uint32_t>(__ballot(wt != 0.f) >> (lane & 48)) & 0xffffu;
  if (!valid) return;
  const int j1 = bits ? 31 - __builtin_clz(bits) : 0;
  const int j0 = bits ? __builtin_ctz(bits) : 0;
  const int cnt = j1 - j0 + 1;
  const float inv = 1.f / sum;
  if (j >= j0 && j <= j1) w_out[j - j0] = wt * inv;
  if (j >= cnt && j < slots) w_out[j] = 0.f;
  if (j == 0) { *lo_out = lo + j0; *count_out = cnt; }
}

// The resize with taps of at most kRegTaps per axis (shrinks up to 3x per side) and
// tx dividing the block: the horizontal pass keeps one output column per thread, its
// weights in registers, and reads each staged row's bytes as aligned dwords; the vertical
// pass keeps one (column, channel) and half of the tile's rows per thread.  NT bounds the
// nonzero horizontal taps: the stretched kernel is nonzero on an open interval of width 4s,
// which holds at most ceil(4s) + 1 sample points (the extra one when rounding leaves a
// near-zero weight at an end), so the NT-tap loop runs unpredicated, the weights past a
// column's count being zero (adding 0 * x leaves every sum bit for bit as it was).  Same
// arithmetic, in the same order, as apc_resize.
template <int NT>
__global__ __launch_bounds__(kRsThreads) void apc_resize_reg(const ResizeParams p) {
  constexpr int ND = (3 * NT + 3) / 4 + 1;   // dwords covering 3 NT bytes at any byte shift
  extern __shared__ float sm[];
  float* wx = sm + p.o_wx;                      // [tx][ntx], ntx a multiple of 4
  float* wy = sm + p.o_wy;                      // [ty][nty]
  int* lox = reinterpret_cast<int*>(sm + p.o_lox);
  int* loy = reinterpret_cast<int*>(sm + p.o_loy);
  int* cnx = lox + p.tx;
  int* cny = loy + p.ty;
  uint32_t* pix = reinterpret_cast<uint32_t*>(sm + p.o_pix);
  float* hb = sm + p.o_h;
  __shared__ int shift[256];
  const int tid = threadIdx.x;
  const int ox0 = blockIdx.x * p.tx, oy0 = blockIdx.y * p.ty;
  const int ncols = min(p.tx, p.oW - ox0), nrows = min(p.ty, p.oH - oy0);
  // taps: 16 lanes per output coordinate, the tile's columns first, then its rows
  for (int b = 0; b < (p.tx + p.ty) * 16; b += kRsThreads) {
    const int item = (b + tid) >> 4;
    if (item < p.tx)
      make_taps_row16(ox0 + item, item < ncols, p.W, p.oW, p.ntx, p.rx, p.invdx, wx + item * p.ntx, &lox[item],
                      &cnx[item]);
    else {
      const int r = min(item - p.tx, p.ty - 1);
      make_taps_row16(oy0 + r, item - p.tx < nrows, p.H, p.oH, p.nty, p.ry, p.invdy, wy + r * p.nty, &loy[r],
                      &cny[r]);
    }
  }
  __syncthreads();
  const int xlo = lox[0], ylo = loy[0];
  const int xin = lox[ncols - 1] + cnx[ncols - 1] - xlo;
  const int yin = loy[nrows - 1] + cny[nrows - 1] - ylo;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.src), (short)0, p.H * p.W * 3, 0x00020000);
  const int nd = (xin * 3 + 3) / 4 + 1;
  const int total = p.H * p.W * 3;
  for (int r = tid; r < yin; r += kRsThreads) {
    const int b0 = (ylo + r) * p.W * 3 + xlo * 3;
    shift[r] = b0 - (b0 & ~3);
  }
  // staging: wave w takes rows w, w + 4, ..., lane l dwords l, l + 64, ...; eight loads in
  // flight per lane before their LDS writes
  {
    const int w = tid >> 6, l = tid & 63;
    for (int r0 = w; r0 < yin; r0 += 8 * (kRsThreads / 64)) {
      for (int d = l; d - l < nd; d += 64) {
        uint32_t v[8];
        int addr[8];
        bool ok[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int r = r0 + u * (kRsThreads / 64);
          ok[u] = r < yin && d < nd;
          addr[u] = (((ylo + r) * p.W + xlo) * 3 & ~3) + 4 * d;
          v[u] = ok[u] ? load_dword(rs, addr[u]) : 0u;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (ok[u] && straddles(addr[u], total)) v[u] = load_dword_bytes(rs, addr[u], total);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (ok[u]) pix[(r0 + u * (kRsThreads / 64)) * p.row_dwords + d] = v[u];
      }
    }
  }
  __syncthreads();
  // horizontal pass: thread -> output column c, staged rows g, g + G, ...
  {
    const int c = tid % p.tx, g = tid / p.tx, G = kRsThreads / p.tx;
    if (c < ncols) {
      float wr[kRegTaps];
#pragma unroll
      for (int q = 0; q < kRegTaps / 4; ++q) {
        const float4 f = (4 * q < p.ntx) ? *reinterpret_cast<const float4*>(wx + c * p.ntx + 4 * q)
                                         : make_float4(0.f, 0.f, 0.f, 0.f);
        wr[4 * q] = f.x; wr[4 * q + 1] = f.y; wr[4 * q + 2] = f.z; wr[4 * q + 3] = f.w;
      }
      const int xoff = (lox[c] - xlo) * 3;
      for (int r = g; r < yin; r += G) {
        const int off = shift[r] + xoff;                       // byte offset in the staged row
        const uint32_t* dp = pix + r * p.row_dwords + (off >> 2);
        const uint32_t sh = static_cast<uint32_t>(off & 3);
        uint32_t d[ND];
#pragma unroll
        for (int k = 0; k < ND; ++k) d[k] = dp[k];
        uint32_t e[ND - 1];
#pragma unroll
        for (int k = 0; k < ND - 1; ++k) e[k] = __builtin_amdgcn_alignbyte(d[k + 1], d[k], sh);
        float a0 = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int b = 3 * j;
          a0 += wr[j] * static_cast<float>((e[b >> 2] >> (8 * (b & 3))) & 255u);
          a1 += wr[j] * static_cast<float>((e[(b + 1) >> 2] >> (8 * ((b + 1) & 3))) & 255u);
          a2 += wr[j] * static_cast<float>((e[(b + 2) >> 2] >> (8 * ((b + 2) & 3))) & 255u);
        }
        float* h = hb + (r * p.tx + c) * 3;
        h[0] = a0; h[1] = a1; h[2] = a2;
      }
    }
  }
  __syncthreads();
  // vertical pass: thread -> (column, channel), half of the tile's output rows
  if (tid < 6 * ncols) {
    const int half = tid >= 3 * ncols ? 1 : 0;
    const int cc = tid - half * 3 * ncols;
    const int c = cc / 3, ch = cc - 3 * c;
    const int rmid = (nrows + 1) / 2;
    for (int r = half * rmid; r < (half ? nrows : rmid); ++r) {
      const float* w = wy + r * p.nty;
      const int base = loy[r] - ylo;
      const int nt = cny[r];
      float acc = 0.f;
#pragma unroll 4
      for (int j = 0; j < nt; ++j) acc += w[j] * hb[((base + j) * p.tx + c) * 3 + ch];
      const float v = floorf(acc + 0.5f);
      const int u = static_cast<int>(fminf(fmaxf(v, 0.f), 255.f));
      p.dst[(static_cast<long long>(oy0 + r) * p.oW + ox0 + c) * 3 + ch] = static_cast<uint8_t>(u);
    }
  }
}

// Shrinks too strong for a staged tile (beyond 32x per side): one workgroup per output pixel,
// straight from memory.  Thread t takes the input columns x = lo_x + t, lo_x + t + 256, ...
// of the pixel's span (consecutive threads read consecutive pixels); for every input row y of
// the span it adds w_x * x[y][x] over its columns (float64) and then w_y times that into its
// sums.  The weights are make_taps' (the same exact integer distance numerators, fp32 cubic),
// normalised at the end by their sums; the workgroup's sums are reduced in a fixed order.
__device__ __forceinline__ void direct_span(int o, int n, int m, int* lo, int* cnt) {
  const double centre = (static_cast<double>(o) + 0.5) * n / m;
  const double support = 2.0 * fmax(1.0, static_cast<double>(n) / m);
  *lo = max(static_cast<int>(floor(centre - support - 0.5)) - 1, 0);
  *cnt = min(n, static_cast<int>(ceil(centre + support + 0.5)) + 2) - *lo;
}
__device__ __forceinline__ float direct_weight(int i, int o, int n, int m, float inv_den) {
  const long long num = (2ll * i + 1) * m - (2ll * o + 1) * n;
  return keys_cubic(static_cast<float>(num) * inv_den);
}

__global__ __launch_bounds__(kRsThreads) void apc_resize_direct(const ResizeParams p) {
  __shared__ double red[4][kRsThreads / 64];
  const int ox = static_cast<int>(blockIdx.x % static_cast<unsigned>(p.oW));
  const int oy = static_cast<int>(blockIdx.x / static_cast<unsigned>(p.oW));
  const int tid = threadIdx.x;
  int lox, nx, loy, ny;
  direct_span(ox, p.W, p.oW, &lox, &nx);
  direct_span(oy, p.H, p.oH, &loy, &ny);
  const float idx = p.invdx, idy = p.invdy;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, swx = 0.0, swy = 0.0;
  for (int j = tid; j < nx; j += kRsThreads) swx += direct_weight(lox + j, ox, p.W, p.oW, idx);
  for (int yi = 0; yi < ny; ++yi) {
    const int y = loy + yi;
    const float wy = direct_weight(y, oy, p.H, p.oH, idy);
    if (tid == 0) swy += wy;
    if (wy == 0.f) continue;   // the same for every thread
    const uint8_t* row = p.src + static_cast<long long>(y) * p.W * 3;
    double h0 = 0.0, h1 = 0.0, h2 = 0.0;
    for (int j = tid; j < nx; j += kRsThreads) {
      const int x = lox + j;
      const double wx = direct_weight(x, ox, p.W, p.oW, idx);
      h0 += wx * row[3 * x];
      h1 += wx * row[3 * x + 1];
      h2 += wx * row[3 * x + 2];
    }
    a0 += wy * h0;
    a1 += wy * h1;
    a2 += wy * h2;
  }
  double v[4] = {a0, a1, a2, swx};
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v[k] += __shfl_xor(v[k], o, 64);
  if ((tid & 63) == 0)
#pragma unroll
    for (int k = 0; k < 4; ++k) red[k][tid >> 6] = v[k];
  __syncthreads();
  if (tid == 0) {
    double t[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      t[k] = red[k][0];
#pragma unroll
      for (int wv = 1; wv < kRsThreads / 64; ++wv) t[k] += red[k][wv];
    }
    const double norm = 1.0 / (t[3] * swy);
    uint8_t* dst = p.dst + (static_cast<long long>(oy) * p.oW + ox) * 3;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const double val = floor(t[c] * norm + 0.5);
      dst[c] = static_cast<uint8_t>(fmin(fmax(val, 0.0), 255.0));
    }
  }
}

__global__ __launch_bounds__(kRsThreads) void apc_resize(const ResizeParams p) {
  extern __shared__ float sm[];
  float* wx = sm + p.o_wx;                      // [tx][ntx]
  float* wy = sm + p.o_wy;                      // [ty][nty]
  int* lox = reinterpret_cast<int*>(sm + p.o_lox);   // [tx]: first tap, then [tx]: tap count
  int* loy = reinterpret_cast<int*>(sm + p.o_loy);   // [ty]: first tap, then [ty]: tap count
  int* cnx = lox + p.tx;
  int* cny = loy + p.ty;
  uint32_t* pix = reinterpret_cast<uint32_t*>(sm + p.o_pix);   // [rows_cap][row_dwords]
  float* hb = sm + p.o_h;                       // [rows_cap][tx][3]
  __shared__ int shift[256];                    // byte shift of each staged row
  const int ox0 = blockIdx.x * p.tx, oy0 = blockIdx.y * p.ty;
  const int ncols = min(p.tx, p.oW - ox0), nrows = min(p.ty, p.oH - oy0);
  for (int c = threadIdx.x; c < ncols; c += kRsThreads)
    lox[c] = make_taps(ox0 + c, p.W, p.oW, p.ntx, wx + c * p.ntx, &cnx[c]);
  for (int r = threadIdx.x; r < nrows; r += kRsThreads)
    loy[r] = make_taps(oy0 + r, p.H, p.oH, p.nty, wy + r * p.nty, &cny[r]);
  __syncthreads();
  const int xlo = lox[0], ylo = loy[0];
  const int xin = lox[ncols - 1] + cnx[ncols - 1] - xlo;      // staged input columns
  const int yin = loy[nrows - 1] + cny[nrows - 1] - ylo;      // staged input rows
  // stage input rows ylo .. ylo+yin-1, bytes [xlo*3, (xlo+xin)*3) of each, as aligned dwords
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.src), (short)0, p.H * p.W * 3, 0x00020000);
  const int nd = (xin * 3 + 3) / 4 + 1;
  const int total = p.H * p.W * 3;
  for (int r = threadIdx.x; r < yin; r += kRsThreads) {
    const int b0 = (ylo + r) * p.W * 3 + xlo * 3;
    shift[r] = b0 - (b0 & ~3);
  }
  // eight loads in flight per thread before their LDS writes
  for (int e0 = threadIdx.x; e0 < yin * nd; e0 += 8 * kRsThreads) {
    uint32_t v[8];
    int slot[8], addr[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + u * kRsThreads;
      const int r = e / nd, d = e - r * nd;
      const int a0 = ((ylo + r) * p.W * 3 + xlo * 3) & ~3;
      slot[u] = (e < yin * nd) ? r * p.row_dwords + d : -1;
      addr[u] = a0 + 4 * d;
      v[u] = (e < yin * nd) ? load_dword(rs, addr[u]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (slot[u] >= 0 && straddles(addr[u], total)) v[u] = load_dword_bytes(rs, addr[u], total);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (slot[u] >= 0) pix[slot[u]] = v[u];
  }
  __syncthreads();
  const uint8_t* pixb = reinterpret_cast<const uint8_t*>(pix);
  // horizontal pass: staged rows x output columns x 3 channels
  for (int e = threadIdx.x; e < yin * ncols; e += kRsThreads) {
    const int r = e / ncols, c = e - r * ncols;
    const uint8_t* row = pixb + r * p.row_dwords * 4 + shift[r] + (lox[c] - xlo) * 3;
    const float* w = wx + c * p.ntx;
    const int nt = cnx[c];
    float a0 = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll 4
    for (int j = 0; j < nt; ++j) {
      const float wt = w[j];
      a0 += wt * static_cast<float>(row[3 * j + 0]);
      a1 += wt * static_cast<float>(row[3 * j + 1]);
      a2 += wt * static_cast<float>(row[3 * j + 2]);
    }
    float* h = hb + (r * p.tx + c) * 3;
    h[0] = a0; h[1] = a1; h[2] = a2;
  }
  __syncthreads();
  // vertical pass and store
  for (int e = threadIdx.x; e < nrows * ncols * 3; e += kRsThreads) {
    const int r = e / (ncols * 3), rem = e - r * ncols * 3;
    const int c = rem / 3, ch = rem - c * 3;
    const float* w = wy + r * p.nty;
    const int base = loy[r] - ylo;
    const int nt = cny[r];
    float acc = 0.f;
#pragma unroll 4
    for (int j = 0; j < nt; ++j) acc += w[j] * hb[((base + j) * p.tx + c) * 3 + ch];
    const float v = floorf(acc + 0.5f);
    const int u = static_cast<int>(fminf(fmaxf(v, 0.f), 255.f));
    p.dst[(static_cast<long long>(oy0 + r) * p.oW + ox0 + c) * 3 + ch] = static_cast<uint8_t>(u);
  }
}

void size_density(Sizer& s, int H, int W, int P) {
  const int gh = H / P, gw = W / P, N = gh * gw, D = 3 * P * P;
  const int tiles = gh * ((gw + kPatchesPerTile - 1) / kPatchesPerTile);
  s.take<float>(N);                              // inv_norm
  s.take<float>(static_cast<size_t>(tiles) * D); // partials
  s.take<float>(D);                              // csum
  s.take<float>(8);                              // stats
  s.take<float>(N);                              // d (when d_out is null)
}

// The density steps over a feature matrix: pass 0 (norms and block partials), the partial
// reduction, c and phi, pass 1 (distances) and the tail.
pace_status_t launch_feature_density(const DensityParams& p, int mode, hipStream_t stream) {
  const dim3 g0(p.n_tiles), g1((p.N + 3) / 4), blk(256);
  if (mode == kFeatBf16Vec) hipLaunchKernelGGL((apc_feat_pass<0, kFeatBf16Vec>), g0, blk, 0, stream, p);
  else if (mode == kFeatBf16) hipLaunchKernelGGL((apc_feat_pass<0, kFeatBf16>), g0, blk, 0, stream, p);
  else hipLaunchKernelGGL((apc_feat_pass<0, kFeatF32>), g0, blk, 0, stream, p);
  pace_status_t st = check_launch("apc_feat_pass<0>");
  if (st != PACE_OK) return st;
  hipLaunchKernelGGL(apc_reduce_c, dim3((p.D + 63) / 64), dim3(1024), 0, stream, p);
  if ((st = check_launch("apc_reduce_c")) != PACE_OK) return st;
  hipLaunchKernelGGL(apc_finalize_c, dim3(1), dim3(1024), 0, stream, p);
  if ((st = check_launch("apc_finalize_c")) != PACE_OK) return st;
  if (mode == kFeatBf16Vec) hipLaunchKernelGGL((apc_feat_pass<1, kFeatBf16Vec>), g1, blk, 0, stream, p);
  else if (mode == kFeatBf16) hipLaunchKernelGGL((apc_feat_pass<1, kFeatBf16>), g1, blk, 0, stream, p);
  else hipLaunchKernelGGL((apc_feat_pass<1, kFeatF32>), g1, blk, 0, stream, p);
  if ((st = check_launch("apc_feat_pass<1>")) != PACE_OK) return st;
  launch_tail(p, stream);
  return check_launch("apc_tail");
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
  PACE_REQUIRE(N < (1ll << 28) && static_cast<long long>(H) * W * 3 < (1ll << 31),
               "pace_apc_density: image too large");
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
  p.row_dwords = ((kPatchesPerTile * patch * 3 + 3) / 4 + 2 + 3) & ~3;
  int nt = pace_keep_count(tail_frac, p.N);
  p.n_tail = nt < 1 ? 1 : nt;
  p.alpha = alpha; p.gamma = gamma;
  Carver c(workspace, workspace_bytes);
  p.inv_norm = c.take<float>(p.N);
  p.partial = c.take<float>(static_cast<size_t>(p.n_tiles) * p.D);
  p.csum = c.take<float>(p.D);
  p.stats = c.take<float>(8);
  float* dws = c.take<float>(p.N);
  p.d = d_out ? d_out : dws;
  p.rho_out = rho_out;
  const size_t lds = (static_cast<size_t>(patch) * p.row_dwords + kPatchesPerTile +
                      static_cast<size_t>(patch) * ((3 * patch + 3) & ~3) + 12) * sizeof(float);
  hipLaunchKernelGGL(apc_patch_pass<0>, dim3(p.n_tiles), dim3(kApcThreads), lds, stream, p);
  pace_status_t st = check_launch("apc_patch_pass<0>");
  if (st != PACE_OK) return st;
  hipLaunchKernelGGL(apc_reduce_c, dim3((p.D + 63) / 64), dim3(1024), 0, stream, p);
  if ((st = check_launch("apc_reduce_c")) != PACE_OK) return st;
  hipLaunchKernelGGL(apc_patch_pass<1>, dim3(p.n_tiles), dim3(kApcThreads), lds, stream, p);
  if ((st = check_launch("apc_patch_pass<1>")) != PACE_OK) return st;
  launch_tail(p, stream);
  return check_launch("apc_tail");
}

size_t pace_apc_density_features_workspace_size(int N, int D) {
  if (N <= 0 || D <= 0) return 0;
  Sizer s;
  const int blocks = (N + kFeatRows - 1) / kFeatRows;
  s.take<float>(N);                                  // inv_norm
  s.take<float>(static_cast<size_t>(blocks) * D);    // partials
  s.take<float>(D);                                  // csum
  s.take<float>(D);                                  // chat
  s.take<float>(8);                                  // stats
  s.take<float>(N);                                  // d (when d_out is null)
  return s.off;
}

pace_status_t pace_apc_density_features(const uint16_t* feat, int N, int D, double tail_frac,
                                        float alpha, float gamma, float* d_out, float* rho_out,
                                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(feat && rho_out, "pace_apc_density_features: null device pointer");
  PACE_REQUIRE((reinterpret_cast<uintptr_t>(feat) & 1u) == 0, "pace_apc_density_features: feat must be 2-byte aligned");
  PACE_REQUIRE(N >= 1 && D >= 1, "pace_apc_density_features: N=%d and D=%d must be >= 1", N, D);
  PACE_REQUIRE(static_cast<long long>(N) * D < (1ll << 40) && D <= (1 << 20),
               "pace_apc_density_features: matrix too large");
  PACE_REQUIRE(tail_frac > 0 && tail_frac <= 1, "pace_apc_density_features: tail_frac must be in (0, 1]");
  PACE_REQUIRE(gamma > 0.f, "pace_apc_density_features: gamma must be > 0");
  const size_t need = pace_apc_density_features_workspace_size(N, D);
  if (workspace == nullptr || workspace_bytes < need)
    return set_error(PACE_ERR_WORKSPACE, "pace_apc_density_features: workspace %zu < %zu bytes",
                     workspace_bytes, need);
  DensityParams p{};
  p.feat = feat;
  p.N = N;
  p.D = D;
  p.n_tiles = (N + kFeatRows - 1) / kFeatRows;
  int nt = pace_keep_count(tail_frac, p.N);
  p.n_tail = nt < 1 ? 1 : nt;
  p.alpha = alpha; p.gamma = gamma;
  Carver c(workspace, workspace_bytes);
  p.inv_norm = c.take<float>(N);
  p.partial = c.take<float>(static_cast<size_t>(p.n_tiles) * D);
  p.csum = c.take<float>(D);
  p.chat = c.take<float>(D);
  p.stats = c.take<float>(8);
  float* dws = c.take<float>(N);
  p.d = d_out ? d_out : dws;
  p.rho_out = rho_out;
  const int mode = (D % 8 == 0 && aligned16(feat)) ? kFeatBf16Vec : kFeatBf16;
  return launch_feature_density(p, mode, stream);
}

size_t pace_apc_pixel_density_workspace_size(int H, int W, int patch, int kind) {
  if (H <= 0 || W <= 0 || patch <= 0 || kind < 0 || kind > 3) return 0;
  const int N = (H / patch) * (W / patch);
  const int D = pixel_feature_dim(kind, patch);
  if (N <= 0) return 0;
  Sizer s;
  s.take<float>(static_cast<size_t>(N) * D);          // the preview vectors
  return align_up(s.off, 256) + pace_apc_density_features_workspace_size(N, D);
}

pace_status_t pace_apc_pixel_features(const uint8_t* img, int H, int W, int patch, int kind,
                                      float* out, hipStream_t stream) {
  PACE_REQUIRE(img && out, "pace_apc_pixel_features: null device pointer");
  PACE_REQUIRE(kind >= 0 && kind <= 3, "pace_apc_pixel_features: kind=%d not in [0, 3]", kind);
  PACE_REQUIRE(patch >= 1 && patch <= kPixMaxPatch, "pace_apc_pixel_features: patch=%d not in [1, %d]",
               patch, kPixMaxPatch);
  PACE_REQUIRE(H >= patch && W >= patch && H % patch == 0 && W % patch == 0,
               "pace_apc_pixel_features: H=%d W=%d must be positive multiples of patch=%d", H, W, patch);
  PACE_REQUIRE(static_cast<long long>(H) * W * 3 < (1ll << 31), "pace_apc_pixel_features: image too large");
  PixelParams q{};
  q.img = img;
  q.H = H; q.W = W; q.P = patch;
  q.gw = W / patch;
  q.N = (H / patch) * q.gw;
  q.kind = kind;
  q.dim = pixel_feature_dim(kind, patch);
  q.out = out;
  hipLaunchKernelGGL(apc_pixel_features, dim3(q.N), dim3(64), 0, stream, q);
  return check_launch("apc_pixel_features");
}

pace_status_t pace_apc_pixel_density(const uint8_t* img, int H, int W, int patch, int kind,
                                     double tail_frac, float alpha, float gamma, float* d_out,
                                     float* rho_out, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
  PACE_REQUIRE(img && rho_out, "pace_apc_pixel_density: null device pointer");
  PACE_REQUIRE(tail_frac > 0 && tail_frac <= 1, "pace_apc_pixel_density: tail_frac must be in (0, 1]");
  PACE_REQUIRE(gamma > 0.f, "pace_apc_pixel_density: gamma must be > 0");
  PACE_REQUIRE(kind >= 0 && kind <= 3, "pace_apc_pixel_density: kind=%d not in [0, 3]", kind);
  PACE_REQUIRE(patch >= 1 && patch <= kPixMaxPatch && H >= patch && W >= patch && H % patch == 0 &&
                   W % patch == 0,
               "pace_apc_pixel_density: H=%d W=%d must be positive multiples of patch=%d <= %d", H, W,
               patch, kPixMaxPatch);
  const size_t need = pace_apc_pixel_density_workspace_size(H, W, patch, kind);
  if (workspace == nullptr || workspace_bytes < need)
    return set_error(PACE_ERR_WORKSPACE, "pace_apc_pixel_density: workspace %zu < %zu bytes",
                     workspace_bytes, need);
  const int N = (H / patch) * (W / patch);
  const int D = pixel_feature_dim(kind, patch);
  Carver c(workspace, workspace_bytes);
  float* feats = c.take<float>(static_cast<size_t>(N) * D);
  pace_status_t st = pace_apc_pixel_features(img, H, W, patch, kind, feats, stream);
  if (st != PACE_OK) return st;
  DensityParams p{};
  p.featf = feats;
  p.N = N;
  p.D = D;
  p.n_tiles = (N + kFeatRows - 1) / kFeatRows;
  const int nt = pace_keep_count(tail_frac, p.N);
  p.n_tail = nt < 1 ? 1 : nt;
  p.alpha = alpha; p.gamma = gamma;
  p.inv_norm = c.take<float>(N);
  p.partial = c.take<float>(static_cast<size_t>(p.n_tiles) * D);
  p.csum = c.take<float>(D);
  p.chat = c.take<float>(D);
  p.stats = c.take<float>(8);
  float* dws = c.take<float>(N);
  p.d = d_out ? d_out : dws;
  p.rho_out = rho_out;
  return launch_feature_density(p, kFeatF32, stream);
}

pace_status_t pace_apc_downsample(const uint8_t* src, int H, int W, uint8_t* dst, int oH, int oW,
                                  hipStream_t stream) {
  PACE_REQUIRE(src && dst, "pace_apc_downsample: null device pointer");
  PACE_REQUIRE(H >= 1 && W >= 1 && oH >= 1 && oW >= 1 && oH <= H && oW <= W,
               "pace_apc_downsample: sizes %dx%d -> %dx%d must shrink or keep", H, W, oH, oW);
  PACE_REQUIRE(static_cast<long long>(H) * W * 3 < (1ll << 31), "pace_apc_downsample: image too large");
  const double sx = static_cast<double>(W) / oW, sy = static_cast<double>(H) / oH;
  ResizeParams p{};
  p.src = src; p.dst = dst;
  p.H = H; p.W = W; p.oH = oH; p.oW = oW;
  p.rx = static_cast<float>(W) / static_cast<float>(oW);
  p.ry = static_cast<float>(H) / static_cast<float>(oH);
  p.invdx = 1.f / static_cast<float>(2ll * (W > oW ? W : oW));
  p.invdy = 1.f / static_cast<float>(2ll * (H > oH ? H : oH));
  if (sx > 32.0 || sy > 32.0) {
    // a staged tile's input span grows with the shrink factor: per output pixel from memory
    hipLaunchKernelGGL(apc_resize_direct, dim3(static_cast<unsigned>(oW) * oH), dim3(kRsThreads), 0, stream, p);
    return check_launch("apc_resize_direct");
  }
  // taps of one output pixel span at most 4*s + 4 inputs (the support plus one zero-weight
  // guard tap on each side)
  p.ntx = static_cast<int>(ceil(4.0 * (sx > 1 ? sx : 1))) + 4;
  p.nty = static_cast<int>(ceil(4.0 * (sy > 1 ? sy : 1))) + 4;
  // 16 x 32 output pixels per workgroup: small enough LDS for three or more workgroups per CU
  // (the image latency of one is hidden by the others), large enough to amortise the taps' halo
  int ty = 16, tx = 32;
  auto plan = [&](int t_y, int t_x, ResizeParams& q) {
    q.ty = t_y; q.tx = t_x;
    q.rows_cap = static_cast<int>(ceil((t_y - 1) * sy)) + q.nty + 1;
    q.cols_cap = static_cast<int>(ceil((t_x - 1) * sx)) + q.ntx + 1;
    q.row_dwords = (q.cols_cap * 3 + 3) / 4 + 2;
    int off = 0;
    q.o_wx = off; off += t_x * q.ntx;
    q.o_wy = off; off += t_y * q.nty;
    q.o_lox = off; off += 2 * t_x;
    q.o_loy = off; off += 2 * t_y;
    q.o_pix = off; off += q.rows_cap * q.row_dwords;
    q.o_h = off; off += q.rows_cap * t_x * 3;
    return static_cast<size_t>(off) * 4;
  };
  size_t lds = plan(ty, tx, p);
  while (lds > kRsMaxLds || p.rows_cap > 256) {
    if (ty > 1) ty >>= 1;
    else if (tx > 1) tx >>= 1;
    else {
      hipLaunchKernelGGL(apc_resize_direct, dim3(static_cast<unsigned>(oW) * oH), dim3(kRsThreads), 0, stream, p);
      return check_launch("apc_resize_direct");
    }
    lds = plan(ty, tx, p);
  }
  dim3 grid((oW + tx - 1) / tx, (oH + ty - 1) / ty);
  const int ntx4 = (p.ntx + 3) / 4 * 4;
  // nonzero horizontal taps per output column: at most ceil(4 sx) + 1 (see apc_resize_reg)
  const int nz = static_cast<int>(ceil(4.0 * (sx > 1 ? sx : 1))) + 1;
  if (ntx4 <= kRegTaps && p.nty <= kRegTaps && kRsThreads % tx == 0 &&
      6 * tx <= kRsThreads && (tx == 32 || tx == 16)) {
    ResizeParams q = p;
    q.ntx = ntx4;
    const size_t lds_q = plan(ty, tx, q);
    if (lds_q <= kRsMaxLds) {
      // ntx4 <= 16 caps ceil(4 sx) at 12, so nz <= 13
      if (nz <= 5) hipLaunchKernelGGL(apc_resize_reg<5>, grid, dim3(kRsThreads), lds_q, stream, q);
      else if (nz <= 9) hipLaunchKernelGGL(apc_resize_reg<9>, grid, dim3(kRsThreads), lds_q, stream, q);
      else hipLaunchKernelGGL(apc_resize_reg<13>, grid, dim3(kRsThreads), lds_q, stream, q);
      return check_launch("apc_resize_reg");
    }
  }
  hipLaunchKernelGGL(apc_resize, grid, dim3(kRsThreads), lds, stream, p);
  return check_launch("apc_resize");
}

}  // extern "C"
