// DDAE (Section 3.3, "Extract"): token maps, min-max normalisation, std confidences,
// softmax(sigma / tau) fusion, top-K ranking and the gather of the kept rows.
//
// Two launches per call when every image has at most 16,384 tokens:
//   ddae_token_maps      grid-wide, one wave of 64 tokens (one per lane) per workgroup,
//                        workgroups never straddle two images: head sums (and the 2x2
//                        merge + permutation for S_vis) -> raw S_vis, S_llm per LLM
//                        visual token (HBM-bound read of the masses), plus each
//                        workgroup's min, max and float64 sum and sum of squares of
//                        both maps
//   ddae_select_gather   a few workgroups per image, each running the same deterministic
//                        selection: the image's statistics from those partials (min-max
//                        ranges; the std of a min-max map is std(raw) / range), the fused
//                        scores in registers (R per thread), top-K by a value-range
//                        histogram and the ranked candidates of its threshold bin (a radix
//                        select when that bin holds many ties), lower-index ties, the
//                        ascending positions of the kept tokens; then each workgroup copies
//                        its own slice of the kept hidden rows.  Repeating the selection
//                        in every workgroup costs L2 reads, not latency, and saves a
//                        launch between the selection and the gather.
// Larger images take the general path: ddae_select (one workgroup per image, maps read
// from memory in every pass) and gather_rows.
#include <math.h>

#include <mutex>
#include <vector>

#include "pace_internal.h"

namespace pace {
namespace {

// Statistics of one map workgroup's tokens.
struct MapPartial {
  float vmin, vmax, lmin, lmax;
  double sv, sv2, sl, sl2;
};

struct SelectParams {
  const float* vis_mass;
  const int32_t* vis_perm;
  const float* llm_mass;
  const float* scores_in;  // given scores (top-K only) or null
  float* vraw;
  float* lraw;
  float* scores;
  float* fuse;
  int32_t* idx;
  long long vis_stride;    // elements per head row of vis_mass (= nv_total * merge)
  int Hv, merge, Hl;
  int B, nv_total;
  int mode;
  float tau, w_llm_fixed;
  int cu_nv[PACE_MAX_SEGMENTS + 1];
  int cu_keep[PACE_MAX_SEGMENTS + 1];
  // map workgroups of image b: [cu_mwg[b], cu_mwg[b+1]); select workgroups likewise
  int cu_mwg[PACE_MAX_SEGMENTS + 1];
  int cu_swg[PACE_MAX_SEGMENTS + 1];
  MapPartial* part;
  const uint4* hidden;
  uint4* out;
  int words_per_row;
  int rows_per_wg;
};

// Largest b < B with cu[b] <= x (cu nondecreasing, cu[0] = 0 <= x).
__device__ __forceinline__ int find_image(const int* cu, int B, int x) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

struct MinOp { __device__ float operator()(float a, float b) const { return fminf(a, b); } };
struct MaxOp { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
struct AddOpD { __device__ double operator()(double a, double b) const { return a + b; } };

constexpr int kMapTokens = 64;    // tokens per map workgroup: one wave, one token per lane
constexpr int kMapHeadsL = 32;    // LLM heads whose loads are in flight together
constexpr int kMapHeadsV = 16;    // vision heads likewise

// One token per lane: every load of a head reads that head's row over 64 consecutive tokens
// (LLM masses) or their permuted 2x2 groups (vision masses), all heads' loads in flight
// together.  Each sum over heads keeps four interleaved partial sums (head 4u + r into sum r,
// u increasing), combined as (s0 + s1) + (s2 + s3).  Then the workgroup's partial
// statistics (wave reductions in a fixed order).
__global__ __launch_bounds__(kMapTokens) void ddae_token_maps(const SelectParams p) {
  // XCD-contiguous logical order: the workgroups of neighbouring raster runs, which read the
  // two halves of the same cache lines of window-ordered vision masses, share an L2
  const int lb = remap_block_id(blockIdx.x, gridDim.x);
  const int b = __builtin_amdgcn_readfirstlane(find_image(p.cu_mwg, p.B, lb));
  const int n0 = p.cu_nv[b];
  const int n = p.cu_nv[b + 1] - n0;
  const int li = (lb - p.cu_mwg[b]) * kMapTokens + static_cast<int>(threadIdx.x);
  const bool valid = li < n;
  const int ii = n0 + (valid ? li : 0);
  // the permutation entry first (the vision loads depend on it), then the LLM masses
  const int local = p.vis_perm ? p.vis_perm[ii] : (ii - n0);
  float l4[4] = {0.f, 0.f, 0.f, 0.f};
  for (int h0 = 0; h0 < p.Hl; h0 += kMapHeadsL) {
    float lm[kMapHeadsL];
    // heads past the last re-read the last one (no predicated loads); they are not added
#pragma unroll
    for (int u = 0; u < kMapHeadsL; ++u)
      lm[u] = p.llm_mass[static_cast<long long>(min(h0 + u, p.Hl - 1)) * p.nv_total + ii];
#pragma unroll
    for (int u = 0; u < kMapHeadsL; ++u)
      if (h0 + u < p.Hl) l4[u & 3] += lm[u];
  }
  const long long patch0 = static_cast<long long>(n0 + local) * p.merge;
  float v4[4] = {0.f, 0.f, 0.f, 0.f};
  if (p.merge == 4) {
    for (int h0 = 0; h0 < p.Hv; h0 += kMapHeadsV) {
      float4 m[kMapHeadsV];
#pragma unroll
      for (int u = 0; u < kMapHeadsV; ++u)
        m[u] = *reinterpret_cast<const float4*>(p.vis_mass + min(h0 + u, p.Hv - 1) * p.vis_stride + patch0);
#pragma unroll
      for (int u = 0; u < kMapHeadsV; ++u)
        if (h0 + u < p.Hv) v4[u & 3] += (m[u].x + m[u].y) + (m[u].z + m[u].w);
    }
  } else {
    for (int h = 0; h < p.Hv; ++h) {
      const float* row = p.vis_mass + h * p.vis_stride + patch0;
      for (int t = 0; t < p.merge; ++t) v4[h & 3] += row[t];
    }
  }
  const float v = (v4[0] + v4[1]) + (v4[2] + v4[3]);
  const float l = (l4[0] + l4[1]) + (l4[2] + l4[3]);
  if (valid) {
    p.vraw[ii] = v;
    p.lraw[ii] = l;
  }
  if (p.part == nullptr) return;
  const float vmin = wave_reduce_dpp(valid ? v : INFINITY, MinOp{});
  const float vmax = wave_reduce_dpp(valid ? v : -INFINITY, MaxOp{});
  const float lmin = wave_reduce_dpp(valid ? l : INFINITY, MinOp{});
  const float lmax = wave_reduce_dpp(valid ? l : -INFINITY, MaxOp{});
  const double dv = valid ? static_cast<double>(v) : 0.0, dl = valid ? static_cast<double>(l) : 0.0;
  const double sv = wave_reduce_dpp(dv, AddOpD{}), sv2 = wave_reduce_dpp(dv * dv, AddOpD{});
  const double sl = wave_reduce_dpp(dl, AddOpD{}), sl2 = wave_reduce_dpp(dl * dl, AddOpD{});
  if (threadIdx.x == 0) {
    MapPartial r;
    r.vmin = vmin; r.vmax = vmax; r.lmin = lmin; r.lmax = lmax;
    r.sv = sv; r.sv2 = sv2; r.sl = sl; r.sl2 = sl2;
    p.part[lb] = r;
  }
}

constexpr int kSelThreads = 1024;
constexpr int kSelR = 16;   // scores per thread kept in registers: images up to 16,384 tokens

// Block-wide combinations of two or four per-thread values in one exchange (fixed wave
// order, deterministic).  `red` holds 4 floats per wave.
__device__ __forceinline__ void block_minmax2(float& a_min, float& a_max, float& b_min, float& b_max,
                                              float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  a_min = wave_min(a_min); a_max = wave_max(a_max);
  b_min = wave_min(b_min); b_max = wave_max(b_max);
  __syncthreads();
  if (lane == 0) { red[4 * w] = a_min; red[4 * w + 1] = a_max; red[4 * w + 2] = b_min; red[4 * w + 3] = b_max; }
  __syncthreads();
  a_min = red[0]; a_max = red[1]; b_min = red[2]; b_max = red[3];
  for (int i = 1; i < nw; ++i) {
    a_min = fminf(a_min, red[4 * i]); a_max = fmaxf(a_max, red[4 * i + 1]);
    b_min = fminf(b_min, red[4 * i + 2]); b_max = fmaxf(b_max, red[4 * i + 3]);
  }
}
__device__ __forceinline__ void block_sum2(float& a, float& b, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  __syncthreads();
  if (lane == 0) { red[4 * w] = a; red[4 * w + 1] = b; }
  __syncthreads();
  a = red[0]; b = red[1];
  for (int i = 1; i < nw; ++i) { a += red[4 * i]; b += red[4 * i + 1]; }
}

// One image whose tokens fit in registers (n <= kSelThreads * kSelR): every map is read
// once; thread t owns tokens t * kSelR + j.  Same steps and outputs as the general path.
__device__ void select_in_registers(const SelectParams& p, int b, float* red, uint32_t* hist, int* cnt) {
  const int n0 = p.cu_nv[b];
  const int n = p.cu_nv[b + 1] - n0;
  const int K = p.cu_keep[b + 1] - p.cu_keep[b];
  const int out0 = p.cu_keep[b];
  const int tid = threadIdx.x;
  const int base = tid * kSelR;
  float sc[kSelR];
  if (p.scores_in == nullptr) {
    const float* vr = p.vraw + n0;
    const float* lr = p.lraw + n0;
    float a[kSelR], c[kSelR];
    float vmin = INFINITY, vmax = -INFINITY, lmin = INFINITY, lmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < kSelR; ++j) {
      const bool ok = base + j < n;
      a[j] = ok ? vr[base + j] : 0.f;
      c[j] = ok ? lr[base + j] : 0.f;
      if (ok) {
        vmin = fminf(vmin, a[j]); vmax = fmaxf(vmax, a[j]);
        lmin = fminf(lmin, c[j]); lmax = fmaxf(lmax, c[j]);
      }
    }
    block_minmax2(vmin, vmax, lmin, lmax, red);
    const float vrange = vmax - vmin, lrange = lmax - lmin;
    // min-max normalised maps (a constant map normalises to zeros)
    float sum_v = 0.f, sum_l = 0.f;
#pragma unroll
    for (int j = 0; j < kSelR; ++j) {
      a[j] = vrange > 0.f ? (a[j] - vmin) / vrange : 0.f;
      c[j] = lrange > 0.f ? (c[j] - lmin) / lrange : 0.f;
      if (base + j < n) { sum_v += a[j]; sum_l += c[j]; }
    }
    block_sum2(sum_v, sum_l, red);
    const float mean_v = sum_v / n, mean_l = sum_l / n;
    float var_v = 0.f, var_l = 0.f;
#pragma unroll
    for (int j = 0; j < kSelR; ++j) {
      if (base + j < n) {
        const float da = a[j] - mean_v, dc = c[j] - mean_l;
        var_v += da * da; var_l += dc * dc;
      }
    }
    block_sum2(var_v, var_l, red);
    const float sig_v = sqrtf(var_v / n), sig_l = sqrtf(var_l / n);   // population std
    float w_l, w_v;
    if (p.mode == 0) {
      w_l = 1.f / (1.f + expf((sig_v - sig_l) / p.tau));   // softmax over two entries
      w_v = 1.f - w_l;
    } else {
      w_l = p.w_llm_fixed;
      w_v = 1.f - p.w_llm_fixed;
    }
    if (tid == 0 && p.fuse) {
      p.fuse[4 * b + 0] = sig_l; p.fuse[4 * b + 1] = sig_v;
      p.fuse[4 * b + 2] = w_l;   p.fuse[4 * b + 3] = w_v;
    }
    float* S = p.scores + n0;
#pragma unroll
    for (int j = 0; j < kSelR; ++j) {
      sc[j] = w_l * c[j] + w_v * a[j];
      if (base + j < n) S[base + j] = sc[j];
    }
  } else {
    const float* S = p.scores_in + n0;
#pragma unroll
    for (int j = 0; j < kSelR; ++j) sc[j] = (base + j < n) ? S[base + j] : 0.f;
  }

  if (K <= 0) return;
  int32_t* idx = p.idx + out0;
  if (K >= n) {
    for (int i = tid; i < n; i += kSelThreads) idx[i] = n0 + i;
    return;
  }
  uint32_t key[kSelR];
#pragma unroll
  for (int j = 0; j < kSelR; ++j) key[j] = float_key(sc[j]);
  int need = 0;
  const uint32_t T = block_radix_select_regs<kSelR>(key, n, K, hist, &need);
  // ascending compaction: keep key > T, plus the `need` lowest-index keys == T
  int n_eq = 0;
#pragma unroll
  for (int j = 0; j < kSelR; ++j) n_eq += (base + j < n && key[j] == T) ? 1 : 0;
  int tot = 0;
  int eq_rank = block_exclusive_sum(n_eq, cnt, &tot);
  bool keep[kSelR];
  int n_keep = 0;
#pragma unroll
  for (int j = 0; j < kSelR; ++j) {
    const bool ok = base + j < n;
    const bool eq = ok && key[j] == T;
    keep[j] = (ok && key[j] > T) || (eq && eq_rank < need);
    eq_rank += eq ? 1 : 0;
    n_keep += keep[j] ? 1 : 0;
  }
  int pos = block_exclusive_sum(n_keep, cnt, &tot);
#pragma unroll
  for (int j = 0; j < kSelR; ++j) {
    if (keep[j]) {
      if (pos < K) idx[pos] = n0 + base + j;
      ++pos;
    }
  }
}

__global__ __launch_bounds__(kSelThreads) void ddae_select(const SelectParams p) {
  __shared__ float red[4 * (kSelThreads / 64)];
  __shared__ uint32_t hist[256 + 8];
  __shared__ int cnt[kSelThreads / 64];
  const int b = blockIdx.x;
  const int n0 = p.cu_nv[b];
  const int n = p.cu_nv[b + 1] - n0;
  if (n <= kSelThreads * kSelR) {
    select_in_registers(p, b, red, hist, cnt);
    return;
  }
  const int K = p.cu_keep[b + 1] - p.cu_keep[b];
  const int out0 = p.cu_keep[b];
  float* S = p.scores + n0;
  const int tid = threadIdx.x;

  if (p.scores_in == nullptr) {
    const float* vr = p.vraw + n0;
    const float* lr = p.lraw + n0;
    float vmin = INFINITY, vmax = -INFINITY, lmin = INFINITY, lmax = -INFINITY;
    for (int i = tid; i < n; i += kSelThreads) {
      const float a = vr[i], c = lr[i];
      vmin = fminf(vmin, a); vmax = fmaxf(vmax, a);
      lmin = fminf(lmin, c); lmax = fmaxf(lmax, c);
    }
    vmin = block_reduce<2>(vmin, red); vmax = block_reduce<1>(vmax, red);
    lmin = block_reduce<2>(lmin, red); lmax = block_reduce<1>(lmax, red);
    const float vrange = vmax - vmin, lrange = lmax - lmin;
    // min-max normalised maps (a constant map normalises to zeros)
    auto sv = [&](int i) { return vrange > 0.f ? (vr[i] - vmin) / vrange : 0.f; };
    auto sl = [&](int i) { return lrange > 0.f ? (lr[i] - lmin) / lrange : 0.f; };
    float sum_v = 0.f, sum_l = 0.f;
    for (int i = tid; i < n; i += kSelThreads) { sum_v += sv(i); sum_l += sl(i); }
    sum_v = block_reduce<0>(sum_v, red);
    sum_l = block_reduce<0>(sum_l, red);
    const float mean_v = sum_v / n, mean_l = sum_l / n;
    float var_v = 0.f, var_l = 0.f;
    for (int i = tid; i < n; i += kSelThreads) {
      const float a = sv(i) - mean_v, c = sl(i) - mean_l;
      var_v += a * a; var_l += c * c;
    }
    var_v = block_reduce<0>(var_v, red);
    var_l = block_reduce<0>(var_l, red);
    const float sig_v = sqrtf(var_v / n), sig_l = sqrtf(var_l / n);   // population std
    float w_l, w_v;
    if (p.mode == 0) {
      // softmax([sigma_llm, sigma_vis] / tau) over two entries
      w_l = 1.f / (1.f + expf((sig_v - sig_l) / p.tau));
      w_v = 1.f - w_l;
    } else {
      w_l = p.w_llm_fixed;
      w_v = 1.f - p.w_llm_fixed;
    }
    if (tid == 0 && p.fuse) {
      p.fuse[4 * b + 0] = sig_l; p.fuse[4 * b + 1] = sig_v;
      p.fuse[4 * b + 2] = w_l;   p.fuse[4 * b + 3] = w_v;
    }
    for (int i = tid; i < n; i += kSelThreads) S[i] = w_l * sl(i) + w_v * sv(i);
    __syncthreads();
  } else {
    S = const_cast<float*>(p.scores_in) + n0;
  }

  if (K <= 0) return;
  int32_t* idx = p.idx + out0;
  if (K >= n) {
    for (int i = tid; i < n; i += kSelThreads) idx[i] = n0 + i;
    return;
  }
  // radix select of the K-th largest score (S is re-read from L2 each pass)
  int need = 0;
  const uint32_t T = block_radix_select(n, K, [&](int i) { return float_key(S[i]); }, hist, &need);
  // ascending compaction: keep key > T, plus the `need` lowest-index keys == T
  int eq_base = 0, out_base = 0;
  for (int c0 = 0; c0 < n; c0 += kSelThreads) {
    const int i = c0 + tid;
    const uint32_t key = (i < n) ? float_key(S[i]) : 0u;
    const bool gt = (i < n) && key > T;
    const bool eq = (i < n) && key == T;
    int eq_tot = 0;
    const int eq_rank = eq_base + block_exclusive_count(eq, cnt, &eq_tot);
    const bool keep = gt || (eq && eq_rank < need);
    int keep_tot = 0;
    const int pos = out_base + block_exclusive_count(keep, cnt, &keep_tot);
    if (keep && pos < K) idx[pos] = n0 + i;
    eq_base += eq_tot;
    out_base += keep_tot;
  }
}

// Exclusive prefix sum of per-thread counts over the block in thread order, and the block
// total.  `wt` is LDS scratch of one word per wave that no other live step uses.  One barrier.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* wt, uint32_t* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const uint32_t incl = wave_incl_scan(v);
  if (lane == 63) wt[w] = incl;
  __syncthreads();
  uint32_t before = 0, tot = 0;
  for (int i0 = 0; i0 < nw; i0 += 4) {   // wt is 16-byte aligned and nw a multiple of 4
    const uint4 c4 = *reinterpret_cast<const uint4*>(&wt[i0]);
    const uint32_t c[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      before += (i0 + q < w) ? c[q] : 0u;
      tot += c[q];
    }
  }
  *total = tot;
  return before + incl - v;
}

constexpr int kValBins = 4096;   // value-range bins of the first selection pass
constexpr int kCandMax = 256;    // candidates ranked by direct comparison

// Selection + gather for images of up to kSelThreads * R tokens (R = 4, 8, 12 or 16 scores
// per thread, the fewest that hold the largest image of the call).  Image b owns select
// workgroups [cu_swg[b], cu_swg[b+1]); each one computes the image's whole selection (same
// inputs, same fixed-order arithmetic, hence the same result in every workgroup), the first
// one writes idx, the scores and the fusion statistics, and workgroup g of the image copies
// kept rows [g * rows_per_wg, (g + 1) * rows_per_wg).
//
// The selection finds the threshold pair (T_key, T_idx): token i is kept iff
// key_i > T_key, or key_i == T_key and i <= T_idx (ties to the lower index).  Steps:
//   1. scores from coalesced loads, transposed through LDS so that thread t holds tokens
//      R t .. R t + R - 1 (the compaction then needs a single block scan);
//   2. a histogram of floor((S - S_min) * 4096 / (S_max - S_min)), a map that is monotone
//      in S also in fp32, and the bin b* that holds the K-th largest score;
//   3. the tokens of bin b* (few, unless scores tie heavily): ranked by direct comparison
//      when at most kCandMax (up to 64 by one wave, a lane each), else by a radix select on
//      their keys;
//   4. ascending compaction: position = number of kept tokens before it.
template <int R>
__global__ __launch_bounds__(kSelThreads) void ddae_select_gather(const SelectParams p) {
  constexpr int kSPad = R + 4;   // LDS floats per thread's row of R scores (+4: 16-byte rows, banks)
  __shared__ __align__(16) uint32_t hist[kValBins];
  __shared__ uint32_t rhist[4 * 256];
  __shared__ __align__(16) float sbuf[kSelThreads * kSPad];
  __shared__ uint32_t cand_key[kCandMax];
  __shared__ int cand_idx[kCandMax];
  __shared__ __align__(16) uint32_t wt[4][kSelThreads / 64];
  __shared__ float wmm[2][kSelThreads / 64];
  __shared__ uint32_t misc[8];   // 0: b*, 1: need, 2: candidates, 3: T_key, 4: T_idx, 5-6: radix
  __shared__ float st_f[4];
  __shared__ double st_d[4];
  extern __shared__ int rows_lds[];   // rows_per_wg source rows of this workgroup's slice
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int b = __builtin_amdgcn_readfirstlane(find_image(p.cu_swg, p.B, blockIdx.x));
  const int gi = blockIdx.x - p.cu_swg[b];
  const bool lead = gi == 0;
  const int n0 = p.cu_nv[b];
  const int n = p.cu_nv[b + 1] - n0;
  const int K = p.cu_keep[b + 1] - p.cu_keep[b];
  const int out0 = p.cu_keep[b];
  const int r0 = gi * p.rows_per_wg;
  const int r1 = min(K, r0 + p.rows_per_wg);
  for (int i = tid; i < kValBins; i += kSelThreads) hist[i] = 0u;
  rhist[tid] = 0u;
  if (tid < 8) misc[tid] = 0u;
  for (int i = tid; i < p.rows_per_wg; i += kSelThreads) rows_lds[i] = -1;

  // ---- 1. scores (strided, coalesced) -> LDS -> blocked registers.  Every load is issued
  // first (they do not depend on the statistics), and the lead's score stores come last:
  // loads and stores share one in-order completion counter, so a store issued between
  // loads would make each later wait cover it too.
  const bool maps = p.scores_in == nullptr;
  // an image of up to 16,384 tokens has at most 256 map workgroups: wave 0 loads four
  // partials per lane, before anything else
  static_assert(kSelThreads * R <= 4 * 64 * kMapTokens, "partials per lane");
  MapPartial r[4];
  const int q0 = p.cu_mwg[b] + lane, q1 = p.cu_mwg[b + 1];
  if (maps && w == 0) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (q0 + 64 * u < q1) r[u] = p.part[q0 + 64 * u];
  }
  float a[R], c[R];
  {
    const auto ra = range_rsrc(maps ? p.vraw + n0 : p.scores_in + n0, static_cast<unsigned>(n) * 4u);
#pragma unroll
    for (int j = 0; j < R; ++j) a[j] = rload_f32(ra, static_cast<unsigned>(j * kSelThreads + tid) * 4u);
    if (maps) {
      const auto rl = range_rsrc(p.lraw + n0, static_cast<unsigned>(n) * 4u);
#pragma unroll
      for (int j = 0; j < R; ++j) c[j] = rload_f32(rl, static_cast<unsigned>(j * kSelThreads + tid) * 4u);
    }
  }
  float smin_l = INFINITY, smax_l = -INFINITY;
  if (maps) {
    // image statistics from the map workgroups' partials, in a fixed order (wave 0)
    if (w == 0) {
      float vmin = INFINITY, vmax = -INFINITY, lmin = INFINITY, lmax = -INFINITY;
      double sv = 0.0, sv2 = 0.0, sl = 0.0, sl2 = 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (q0 + 64 * u < q1) {
          vmin = fminf(vmin, r[u].vmin); vmax = fmaxf(vmax, r[u].vmax);
          lmin = fminf(lmin, r[u].lmin); lmax = fmaxf(lmax, r[u].lmax);
          sv += r[u].sv; sv2 += r[u].sv2; sl += r[u].sl; sl2 += r[u].sl2;
        }
      }
      vmin = wave_reduce_dpp(vmin, MinOp{}); vmax = wave_reduce_dpp(vmax, MaxOp{});
      lmin = wave_reduce_dpp(lmin, MinOp{}); lmax = wave_reduce_dpp(lmax, MaxOp{});
      sv = wave_reduce_dpp(sv, AddOpD{}); sv2 = wave_reduce_dpp(sv2, AddOpD{});
      sl = wave_reduce_dpp(sl, AddOpD{}); sl2 = wave_reduce_dpp(sl2, AddOpD{});
      if (lane == 0) {
        // population std of a min-max normalised map = std(raw map) / range (0 for a
        // constant map, which normalises to zeros)
        const double dn = static_cast<double>(n);
        const double vr = static_cast<double>(vmax) - vmin, lr = static_cast<double>(lmax) - lmin;
        const double mv = sv / dn, ml = sl / dn;
        const double sig_v = vr > 0.0 ? sqrt(fmax(sv2 / dn - mv * mv, 0.0)) / vr : 0.0;
        const double sig_l = lr > 0.0 ? sqrt(fmax(sl2 / dn - ml * ml, 0.0)) / lr : 0.0;
        double w_l;
        if (p.mode == 0)   // softmax of two entries
          w_l = 1.0 / (1.0 + static_cast<double>(expf(static_cast<float>((sig_v - sig_l) / p.tau))));
        else
          w_l = p.w_llm_fixed;
        st_f[0] = vmin; st_f[1] = vmax; st_f[2] = lmin; st_f[3] = lmax;
        st_d[0] = sig_l; st_d[1] = sig_v; st_d[2] = w_l; st_d[3] = 1.0 - w_l;
      }
    }
    __syncthreads();
    // (x - min) * (1 / range): a multiply per token instead of an IEEE division
    const float vmin = st_f[0], vrange = st_f[1] - st_f[0];
    const float lmin = st_f[2], lrange = st_f[3] - st_f[2];
    const float vinv = vrange > 0.f ? 1.f / vrange : 0.f, linv = lrange > 0.f ? 1.f / lrange : 0.f;
    const float w_l = static_cast<float>(st_d[2]), w_v = static_cast<float>(st_d[3]);
#pragma unroll
    for (int j = 0; j < R; ++j) a[j] = w_l * ((c[j] - lmin) * linv) + w_v * ((a[j] - vmin) * vinv);
  }
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int i = j * kSelThreads + tid;
    if (i < n) {
      sbuf[(i / R) * kSPad + i % R] = a[j];
      smin_l = fminf(smin_l, a[j]);
      smax_l = fmaxf(smax_l, a[j]);
    }
  }
  if (maps && lead) {
    const auto rs = range_rsrc(p.scores + n0, static_cast<unsigned>(n) * 4u);
#pragma unroll
    for (int j = 0; j < R; ++j)
      rstore_b32(rs, static_cast<unsigned>(j * kSelThreads + tid) * 4u, __float_as_uint(a[j]));
    if (tid == 0 && p.fuse) {
      p.fuse[4 * b + 0] = static_cast<float>(st_d[0]); p.fuse[4 * b + 1] = static_cast<float>(st_d[1]);
      p.fuse[4 * b + 2] = static_cast<float>(st_d[2]); p.fuse[4 * b + 3] = static_cast<float>(st_d[3]);
    }
  }
  smin_l = wave_reduce_dpp(smin_l, MinOp{});
  smax_l = wave_reduce_dpp(smax_l, MaxOp{});
  if (lane == 0) { wmm[0][w] = smin_l; wmm[1][w] = smax_l; }
  __syncthreads();
  if (K <= 0) return;

  const int base = tid * R;
  uint32_t key[R];
  {
    float s[R];
#pragma unroll
    for (int q = 0; q < R / 4; ++q) {
      const float4 f = *reinterpret_cast<const float4*>(&sbuf[tid * kSPad + 4 * q]);
      s[4 * q] = f.x; s[4 * q + 1] = f.y; s[4 * q + 2] = f.z; s[4 * q + 3] = f.w;
    }
#pragma unroll
    for (int j = 0; j < R; ++j) key[j] = float_key(s[j]);
    if (K < n) {
      float smin = wmm[0][0], smax = wmm[1][0];
      for (int i = 1; i < kSelThreads / 64; ++i) { smin = fminf(smin, wmm[0][i]); smax = fmaxf(smax, wmm[1][i]); }
      // ---- 2. value-range histogram (monotone non-decreasing bin map, clamped)
      const float cscale = smax > smin ? fminf(static_cast<float>(kValBins) / (smax - smin), 3.4e38f) : 0.f;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const int bin = static_cast<int>(fminf((s[j] - smin) * cscale, static_cast<float>(kValBins - 1)));
        // equal scores would all hit one LDS address: the all-equal case is counted below
        if (base + j < n && cscale > 0.f) atomicAdd(&hist[bin], 1u);
        key[j] = (base + j < n) ? key[j] : 0u;
        s[j] = static_cast<float>(bin);   // keep the bin (exact small integer)
      }
      if (cscale == 0.f && tid == 0) hist[0] = static_cast<uint32_t>(n);
      __syncthreads();
      // thread t covers bins 4095 - 4t down to 4092 - 4t (descending)
      const int bhi = kValBins - 1 - 4 * tid;
      const uint4 h4 = *reinterpret_cast<const uint4*>(&hist[bhi - 3]);
      const uint32_t c0 = h4.w, c1 = h4.z, c2 = h4.y, c3 = h4.x;
      uint32_t tot_all = 0;
      uint32_t before = block_excl_scan(c0 + c1 + c2 + c3, wt[0], &tot_all);
      const uint32_t cs[4] = {c0, c1, c2, c3};
      const uint32_t uK = static_cast<uint32_t>(K);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (before < uK && before + cs[q] >= uK) { misc[0] = bhi - q; misc[1] = uK - before; }
        before += cs[q];
      }
      __syncthreads();
      const int bstar = static_cast<int>(misc[0]);
      const int need = static_cast<int>(misc[1]);   // 1 <= need <= count of bin b*
      // ---- 3. candidates: the tokens of bin b*
#pragma unroll
      for (int j = 0; j < R; ++j) {
        if (base + j < n && static_cast<int>(s[j]) == bstar) {
          const uint32_t slot = atomicAdd(&misc[2], 1u);
          if (slot < static_cast<uint32_t>(kCandMax)) { cand_key[slot] = key[j]; cand_idx[slot] = base + j; }
        }
      }
      __syncthreads();
      const uint32_t ncand = misc[2];
      if (ncand <= 64u) {
        // one wave ranks up to 64 candidates, one per lane, the others' keys read by lane
        // index; rank = candidates ahead in (key descending, index ascending) order
        if (w == 0) {
          const bool mine = lane < static_cast<int>(ncand);
          const uint32_t kt = mine ? cand_key[lane] : 0u;
          const int it = mine ? cand_idx[lane] : 0;
          int rank = 0;
          for (uint32_t u = 0; u < ncand; ++u) {
            const uint32_t ku = __builtin_amdgcn_readlane(kt, u);
            const int iu = __builtin_amdgcn_readlane(it, u);
            rank += (ku > kt || (ku == kt && iu < it)) ? 1 : 0;
          }
          if (mine && rank == need - 1) { misc[3] = kt; misc[4] = static_cast<uint32_t>(it); }
        }
      } else if (ncand <= static_cast<uint32_t>(kCandMax)) {
        // rank = candidates ahead in (key descending, index ascending) order
        if (tid < static_cast<int>(ncand)) {
          const uint32_t kt = cand_key[tid];
          const int it = cand_idx[tid];
          int rank = 0;
#pragma unroll 8
          for (uint32_t u = 0; u < ncand; ++u) {
            const uint32_t ku = cand_key[u];
            rank += (ku > kt || (ku == kt && cand_idx[u] < it)) ? 1 : 0;
          }
          if (rank == need - 1) { misc[3] = kt; misc[4] = static_cast<uint32_t>(it); }
        }
      } else {
        // many ties in one bin: radix select over the candidates' keys, then the lowest
        // indices among the keys equal to the threshold
        uint32_t ck[R];
#pragma unroll
        for (int j = 0; j < R; ++j) ck[j] = (base + j < n && static_cast<int>(s[j]) == bstar) ? key[j] : 0u;
        // keys of non-candidates are 0: below every candidate key only if no candidate key
        // is 0, so they are excluded by count instead (the radix ranks the top `need` of
        // all ck, and every candidate outranks a non-candidate unless keys are 0, i.e. -NaN)
        int need_eq = 0;
        const uint32_t T = radix_select_prezeroed<R, false>(ck, n, need, rhist, &misc[5], &need_eq);
        uint32_t eqc = 0;
#pragma unroll
        for (int j = 0; j < R; ++j) eqc += (base + j < n && static_cast<int>(s[j]) == bstar && key[j] == T) ? 1u : 0u;
        uint32_t tot_eq = 0;
        uint32_t eq_before = block_excl_scan(eqc, wt[1], &tot_eq);
#pragma unroll
        for (int j = 0; j < R; ++j) {
          if (base + j < n && static_cast<int>(s[j]) == bstar && key[j] == T) {
            if (eq_before == static_cast<uint32_t>(need_eq - 1)) { misc[3] = T; misc[4] = static_cast<uint32_t>(base + j); }
            ++eq_before;
          }
        }
      }
      __syncthreads();
      const uint32_t tkey = misc[3];
      const int tidx = static_cast<int>(misc[4]);
#pragma unroll
      for (int j = 0; j < R; ++j)
        key[j] = (base + j < n && (key[j] > tkey || (key[j] == tkey && base + j <= tidx))) ? 1u : 0u;
    } else {
#pragma unroll
      for (int j = 0; j < R; ++j) key[j] = (base + j < n) ? 1u : 0u;   // every token kept
    }
  }
  // ---- 4. ascending compaction (key[j] is now the keep flag)
  uint32_t kc = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) kc += key[j];
  uint32_t tot_keep = 0;
  uint32_t pos = block_excl_scan(kc, wt[2], &tot_keep);
  if (lead) {   // the kept indices (one workgroup stores them; the others only need their slice)
    const auto ri = range_rsrc(p.idx + out0, static_cast<unsigned>(K) * 4u);
    uint32_t ps = pos;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      rstore_b32(ri, key[j] ? ps * 4u : kNoStore, static_cast<uint32_t>(n0 + base + j));
      ps += key[j];
    }
  }
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if (key[j] && static_cast<int>(pos) >= r0 && static_cast<int>(pos) < r1) rows_lds[pos - r0] = n0 + base + j;
    pos += key[j];
  }
  if (p.hidden == nullptr || r1 <= r0) return;
  __syncthreads();
  // this workgroup's slice of the gather, in 16-byte words
  const int W = p.words_per_row;
  const int total = (r1 - r0) * W;
  for (int e = tid; e < total; e += kSelThreads) {
    const int r = e / W, wd = e - r * W;
    const int src = rows_lds[r];
    if (src >= 0 && src < p.nv_total)   // always true; never read outside hidden
      p.out[static_cast<long long>(out0 + r0 + r) * W + wd] = p.hidden[static_cast<long long>(src) * W + wd];
  }
}

// out[r, :] = hidden[idx[r], :] in 16-byte words; one row per block-row.
__global__ __launch_bounds__(256) void gather_rows(const uint4* __restrict__ hidden,
                                                   const int32_t* __restrict__ idx,
                                                   uint4* __restrict__ out, int rows,
                                                   int words_per_row, int src_rows) {
  const int r = blockIdx.x;
  if (r >= rows) return;
  const int sr = idx[r];
  if (sr < 0 || sr >= src_rows) return;   // never read outside hidden
  const long long src = static_cast<long long>(sr) * words_per_row;
  const long long dst = static_cast<long long>(r) * words_per_row;
  for (int w = threadIdx.x; w < words_per_row; w += 256) {
    out[dst + w] = hidden[src + w];
  }
}

pace_status_t run_select(SelectParams& p, const void* hidden, size_t row_bytes, void* out,
                         hipStream_t stream, bool need_maps) {
  int nmax = 0;
  p.cu_mwg[0] = 0;
  for (int b = 0; b < p.B; ++b) {
    const int n = p.cu_nv[b + 1] - p.cu_nv[b];
    nmax = n > nmax ? n : nmax;
    p.cu_mwg[b + 1] = p.cu_mwg[b] + (n + kMapTokens - 1) / kMapTokens;
  }
  const bool fused = nmax <= kSelThreads * kSelR;
  if (!fused) p.part = nullptr;
  if (need_maps && p.nv_total > 0) {
    hipLaunchKernelGGL(ddae_token_maps, dim3(p.cu_mwg[p.B]), dim3(kMapTokens), 0, stream, p);
    pace_status_t st = check_launch("ddae_token_maps");
    if (st != PACE_OK) return st;
  }
  // kept rows of this launch: [cu_keep[0], cu_keep[B]) (offsets are global across launches)
  const int kfirst = p.cu_keep[0];
  const int ktot = p.cu_keep[p.B] - kfirst;
  if (fused) {
    // rows per select workgroup: at least 4, and about one workgroup per CU (256) for the
    // gather (a select workgroup's LDS, ~105 KB with 16 scores per thread down to ~57 KB
    // with 4, leaves room for one or two per CU)
    int R = 1;
    if (hidden != nullptr && ktot > 0) {
      R = (ktot + 255) / 256;
      R = R < 4 ? 4 : (R > 4096 ? 4096 : R);
    }
    p.hidden = static_cast<const uint4*>(hidden);
    p.out = static_cast<uint4*>(out);
    p.words_per_row = static_cast<int>(row_bytes / 16);
    p.rows_per_wg = R;
    p.cu_swg[0] = 0;
    for (int b = 0; b < p.B; ++b) {
      const int K = p.cu_keep[b + 1] - p.cu_keep[b];
      p.cu_swg[b + 1] = p.cu_swg[b] + ((hidden != nullptr && K > 0) ? (K + R - 1) / R : 1);
    }
    const dim3 grid(p.cu_swg[p.B]);
    const size_t dyn = static_cast<size_t>(R) * sizeof(int);
    if (nmax <= kSelThreads * 4) hipLaunchKernelGGL(ddae_select_gather<4>, grid, dim3(kSelThreads), dyn, stream, p);
    else if (nmax <= kSelThreads * 8) hipLaunchKernelGGL(ddae_select_gather<8>, grid, dim3(kSelThreads), dyn, stream, p);
    else if (nmax <= kSelThreads * 12) hipLaunchKernelGGL(ddae_select_gather<12>, grid, dim3(kSelThreads), dyn, stream, p);
    else hipLaunchKernelGGL(ddae_select_gather<kSelR>, grid, dim3(kSelThreads), dyn, stream, p);
    return check_launch("ddae_select_gather");
  }
  hipLaunchKernelGGL(ddae_select, dim3(p.B), dim3(kSelThreads), 0, stream, p);
  pace_status_t st = check_launch("ddae_select");
  if (st != PACE_OK) return st;
  if (hidden != nullptr && ktot > 0) {
    const int words = static_cast<int>(row_bytes / 16);
    hipLaunchKernelGGL(gather_rows, dim3(ktot), dim3(256), 0, stream,
                       static_cast<const uint4*>(hidden), p.idx + kfirst,
                       static_cast<uint4*>(out) + static_cast<long long>(kfirst) * words, ktot, words,
                       p.nv_total);
    st = check_launch("gather_rows");
    if (st != PACE_OK) return st;
  }
  return PACE_OK;
}

void size_select(Sizer& s, int nv_total, int nseg) {
  s.take<MapPartial>((nv_total + kMapTokens - 1) / kMapTokens + nseg);   // map partials
  s.take<float>(nv_total);   // vraw
  s.take<float>(nv_total);   // lraw
  s.take<float>(nv_total);   // scores (when the caller passes none)
  s.take<float>(4 * nseg);   // fusion stats (when the caller passes none)
}

}  // namespace

// ---------------------------------------------------------------- allocation-free selection
// Scratch of pace_ddae_select_varlen_noalloc: a device array of fixed size, one copy per GPU
// (each holds it until the process ends), standing in for the caller's workspace.  Nothing in
// it must start at zero: every selection writes each value it later reads.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in): it looks up the
// array's device address once per device, with that device current, and passes that.
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

pace_status_t scratch_on_current_device(void** out) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(PACE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(PACE_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* ptr = nullptr;
    const hipError_t r = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (r != hipSuccess || ptr == nullptr)
      return set_error(PACE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(r));
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return PACE_OK;
}
}  // namespace
}  // namespace pace

using namespace pace;

extern "C" {

size_t pace_ddae_select_workspace_size(int nv_total, int nseg) {
  if (nv_total < 0 || nseg < 0) return 0;
  Sizer s;
  size_select(s, nv_total, nseg);
  return s.off;
}

pace_status_t pace_ddae_select_varlen(const float* vis_mass, int Hv, int merge,
                                      const int32_t* vis_perm, const float* llm_mass, int Hl,
                                      int B, const int* nv_host, const int* keep_host, int mode,
                                      float tau, float w_llm_fixed, const void* hidden,
                                      size_t row_bytes, int32_t* idx_out, float* score_out,
                                      float* fuse_out, void* out, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(B >= 1, "pace_ddae_select: B=%d must be >= 1", B);
  PACE_REQUIRE(nv_host && keep_host, "pace_ddae_select: null host count arrays");
  PACE_REQUIRE(Hv >= 1 && Hl >= 1 && merge >= 1, "pace_ddae_select: Hv=%d Hl=%d merge=%d", Hv, Hl,
               merge);
  PACE_REQUIRE(mode == 0 || mode == 1, "pace_ddae_select: mode=%d must be 0 or 1", mode);
  PACE_REQUIRE(mode == 1 || (tau > 0.f && isfinite(tau)), "pace_ddae_select: tau must be > 0");
  PACE_REQUIRE(vis_mass && llm_mass && idx_out, "pace_ddae_select: null device pointer");
  SelectParams p{};
  std::vector<int> cu_nv(B + 1, 0), cu_keep(B + 1, 0);
  for (int b = 0; b < B; ++b) {
    PACE_REQUIRE(nv_host[b] >= 1, "pace_ddae_select: image %d has %d tokens", b, nv_host[b]);
    PACE_REQUIRE(keep_host[b] >= 0 && keep_host[b] <= nv_host[b],
                 "pace_ddae_select: K=%d outside [0, %d] for image %d", keep_host[b], nv_host[b], b);
    PACE_REQUIRE(static_cast<long long>(cu_nv[b]) + nv_host[b] < (1ll << 30),
                 "pace_ddae_select: too many tokens");
    cu_nv[b + 1] = cu_nv[b] + nv_host[b];
    cu_keep[b + 1] = cu_keep[b] + keep_host[b];
  }
  const int nv_total = cu_nv[B];
  PACE_REQUIRE(merge != 4 || aligned16(vis_mass), "pace_ddae_select: vis_mass must be 16-byte aligned");
  if (hidden != nullptr) {
    PACE_REQUIRE(out != nullptr, "pace_ddae_select: out is null while hidden is given");
    PACE_REQUIRE(row_bytes > 0 && row_bytes % 16 == 0,
                 "pace_ddae_select: row_bytes=%zu must be a positive multiple of 16", row_bytes);
    PACE_REQUIRE(aligned16(hidden) && aligned16(out), "pace_ddae_select: hidden/out not 16-byte aligned");
  }
  const size_t need = pace_ddae_select_workspace_size(nv_total, B);
  if (workspace == nullptr || workspace_bytes < need)
    return set_error(PACE_ERR_WORKSPACE, "pace_ddae_select: workspace %zu < %zu bytes",
                     workspace_bytes, need);
  if (vis_perm != nullptr && debug_checks()) {
    std::vector<int32_t> perm(nv_total);
    pace_status_t chk = copy_to_host(perm.data(), vis_perm, nv_total, stream);
    if (chk != PACE_OK) return chk;
    for (int b = 0; b < B; ++b)
      for (int i = cu_nv[b]; i < cu_nv[b + 1]; ++i)
        PACE_REQUIRE(perm[i] >= 0 && perm[i] < nv_host[b],
                     "pace_ddae_select: vis_perm[%d] = %d outside [0, %d) for image %d", i, perm[i], nv_host[b], b);
  }
  Carver c(workspace, workspace_bytes);
  p.part = c.take<MapPartial>((nv_total + kMapTokens - 1) / kMapTokens + B);
  p.vraw = c.take<float>(nv_total);
  p.lraw = c.take<float>(nv_total);
  float* sc = c.take<float>(nv_total);
  float* fz = c.take<float>(4 * B);
  p.scores = score_out ? score_out : sc;
  p.fuse = fuse_out ? fuse_out : fz;
  p.vis_mass = vis_mass;
  p.vis_perm = vis_perm;
  p.llm_mass = llm_mass;
  p.scores_in = nullptr;
  p.idx = idx_out;
  p.vis_stride = static_cast<long long>(nv_total) * merge;
  p.Hv = Hv; p.merge = merge; p.Hl = Hl; p.nv_total = nv_total;
  p.mode = mode; p.tau = tau; p.w_llm_fixed = w_llm_fixed;
  // Images are independent: a batch of more than PACE_MAX_SEGMENTS images runs as consecutive
  // launches of at most that many (the offsets travel in the kernel arguments).  Every kernel
  // indexes tokens and kept rows by their global offsets, so a launch takes its images' slice
  // of cu_nv / cu_keep unchanged; only the per-image fusion weights are indexed per launch.
  for (int b0 = 0; b0 < B; b0 += PACE_MAX_SEGMENTS) {
    const int nb = B - b0 < PACE_MAX_SEGMENTS ? B - b0 : PACE_MAX_SEGMENTS;
    SelectParams q = p;
    for (int j = 0; j <= nb; ++j) {
      q.cu_nv[j] = cu_nv[b0 + j];
      q.cu_keep[j] = cu_keep[b0 + j];
    }
    q.B = nb;
    q.fuse = p.fuse + 4 * b0;
    const pace_status_t st = run_select(q, hidden, row_bytes, out, stream, true);
    if (st != PACE_OK) return st;
  }
  return PACE_OK;
}

pace_status_t pace_ddae_select(const float* vis_mass, int Hv, int merge, const int32_t* vis_perm,
                               const float* llm_mass, int Hl, int Nv, int mode, float tau,
                               float w_llm_fixed, int K, const void* hidden, size_t row_bytes,
                               int32_t* idx_out, float* score_out, float* fuse_out, void* out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const int nv[1] = {Nv};
  const int kk[1] = {K};
  return pace_ddae_select_varlen(vis_mass, Hv, merge, vis_perm, llm_mass, Hl, 1, nv, kk, mode, tau,
                                 w_llm_fixed, hidden, row_bytes, idx_out, score_out, fuse_out, out,
                                 workspace, workspace_bytes, stream);
}

size_t pace_ddae_select_noalloc_max_bytes(void) { return kNoAllocScratchBytes; }

pace_status_t pace_ddae_select_varlen_noalloc(const float* vis_mass, int Hv, int merge,
                                              const int32_t* vis_perm, const float* llm_mass, int Hl,
                                              int B, const int* nv_host, const int* keep_host, int mode,
                                              float tau, float w_llm_fixed, const void* hidden,
                                              size_t row_bytes, int32_t* idx_out, float* score_out,
                                              float* fuse_out, void* out, hipStream_t stream) {
  PACE_REQUIRE(B >= 1, "pace_ddae_select_varlen_noalloc: B=%d must be >= 1", B);
  PACE_REQUIRE(nv_host && keep_host, "pace_ddae_select_varlen_noalloc: null host count arrays");
  long long nv_total = 0;
  for (int b = 0; b < B; ++b) {
    PACE_REQUIRE(nv_host[b] >= 1, "pace_ddae_select_varlen_noalloc: image %d has %d tokens", b, nv_host[b]);
    nv_total += nv_host[b];
  }
  PACE_REQUIRE(nv_total < (1ll << 30), "pace_ddae_select_varlen_noalloc: too many tokens");
  const size_t need = pace_ddae_select_workspace_size(static_cast<int>(nv_total), B);
  if (need > kNoAllocScratchBytes)
    return set_error(PACE_ERR_WORKSPACE,
                     "pace_ddae_select_varlen_noalloc: %lld tokens in %d images need %zu bytes of scratch, "
                     "more than the %zu of the static scratch; use pace_ddae_select_varlen with a workspace",
                     nv_total, B, need, kNoAllocScratchBytes);
  void* ws = nullptr;
  pace_status_t st = scratch_on_current_device(&ws);
  if (st != PACE_OK) return st;
  return pace_ddae_select_varlen(vis_mass, Hv, merge, vis_perm, llm_mass, Hl, B, nv_host, keep_host, mode,
                                 tau, w_llm_fixed, hidden, row_bytes, idx_out, score_out, fuse_out, out, ws,
                                 kNoAllocScratchBytes, stream);
}

pace_status_t pace_topk_gather(const float* scores, int N, int K, const void* hidden,
                               size_t row_bytes, int32_t* idx_out, void* out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  PACE_REQUIRE(N >= 1, "pace_topk_gather: N=%d must be >= 1", N);
  PACE_REQUIRE(K >= 0 && K <= N, "pace_topk_gather: K=%d outside [0, %d]", K, N);
  PACE_REQUIRE(scores && idx_out, "pace_topk_gather: null device pointer");
  if (hidden != nullptr) {
    PACE_REQUIRE(out != nullptr, "pace_topk_gather: out is null while hidden is given");
    PACE_REQUIRE(row_bytes > 0 && row_bytes % 16 == 0,
                 "pace_topk_gather: row_bytes=%zu must be a positive multiple of 16", row_bytes);
    PACE_REQUIRE(aligned16(hidden) && aligned16(out), "pace_topk_gather: hidden/out not 16-byte aligned");
  }
  SelectParams p{};
  p.B = 1;
  p.cu_nv[0] = 0; p.cu_nv[1] = N;
  p.cu_keep[0] = 0; p.cu_keep[1] = K;
  p.nv_total = N;
  p.scores_in = scores;
  p.scores = nullptr;
  p.idx = idx_out;
  return run_select(p, hidden, row_bytes, out, stream, false);
}

pace_status_t pace_gather_rows(const void* src, int src_rows, size_t row_bytes,
                               const int32_t* idx, int n_idx, void* dst, hipStream_t stream) {
  PACE_REQUIRE(n_idx >= 0 && src_rows >= 0, "pace_gather_rows: n_idx=%d src_rows=%d", n_idx, src_rows);
  if (n_idx == 0) return PACE_OK;
  PACE_REQUIRE(src && idx && dst, "pace_gather_rows: null device pointer");
  PACE_REQUIRE(row_bytes > 0 && row_bytes % 16 == 0,
               "pace_gather_rows: row_bytes=%zu must be a positive multiple of 16", row_bytes);
  PACE_REQUIRE(row_bytes / 16 < (1u << 30), "pace_gather_rows: rows too long");
  PACE_REQUIRE(aligned16(src) && aligned16(dst), "pace_gather_rows: src/dst not 16-byte aligned");
  hipLaunchKernelGGL(gather_rows, dim3(n_idx), dim3(256), 0, stream, static_cast<const uint4*>(src), idx,
                     static_cast<uint4*>(dst), n_idx, static_cast<int>(row_bytes / 16), src_rows);
  return check_launch("gather_rows");
}

}  // extern "C"
