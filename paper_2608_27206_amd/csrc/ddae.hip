// DDAE (Section 3.3, "Extract"): token maps, min-max normalisation, std confidences,
// softmax(sigma / tau) fusion, top-K ranking and the gather of the kept rows.
//
// Three launches per call:
//   ddae_token_maps   grid-wide: head sums (and 2x2 merge + permutation for S_vis)
//                     -> raw S_vis, S_llm per LLM visual token (HBM-bound read of the masses)
//   ddae_select       one workgroup per image: min/max, means, stds, weights, S_final,
//                     radix top-K with lower-index ties, ascending compaction (images of
//                     up to 16,384 tokens entirely in registers, larger ones from memory)
//   gather_rows       grid-wide 16-byte row copy of the kept hidden states
#include <math.h>

#include "pace_internal.h"

namespace pace {
namespace {

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
};

__device__ __forceinline__ int find_segment(const SelectParams& p, int i) {
  int lo = 0, hi = p.B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.cu_nv[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Four lanes per token, each summing every fourth head; combined by shuffles in a fixed
// order (deterministic).
__global__ __launch_bounds__(256) void ddae_token_maps(const SelectParams p) {
  const int i = blockIdx.x * 64 + (threadIdx.x >> 2);
  const int part = threadIdx.x & 3;
  const bool valid = i < p.nv_total;
  const int ii = valid ? i : 0;
  const int b = find_segment(p, ii);
  const int base = p.cu_nv[b];
  const int local = p.vis_perm ? p.vis_perm[ii] : (ii - base);
  const long long patch0 = static_cast<long long>(base + local) * p.merge;
  float v = 0.f;
  if (valid) {
    if (p.merge == 4) {
      for (int h = part; h < p.Hv; h += 4) {
        const float4 m = *reinterpret_cast<const float4*>(p.vis_mass + h * p.vis_stride + patch0);
        v += (m.x + m.y) + (m.z + m.w);
      }
    } else {
      for (int h = part; h < p.Hv; h += 4) {
        const float* row = p.vis_mass + h * p.vis_stride + patch0;
        for (int t = 0; t < p.merge; ++t) v += row[t];
      }
    }
  }
  float l = 0.f;
  if (valid)
    for (int h = part; h < p.Hl; h += 4) l += p.llm_mass[static_cast<long long>(h) * p.nv_total + ii];
  v += __shfl_xor(v, 1, 64);
  l += __shfl_xor(l, 1, 64);
  v += __shfl_xor(v, 2, 64);
  l += __shfl_xor(l, 2, 64);
  if (valid && part == 0) {
    p.vraw[i] = v;
    p.lraw[i] = l;
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
  if (need_maps && p.nv_total > 0) {
    const int blocks = (p.nv_total + 63) / 64;
    hipLaunchKernelGGL(ddae_token_maps, dim3(blocks), dim3(256), 0, stream, p);
    pace_status_t st = check_launch("ddae_token_maps");
    if (st != PACE_OK) return st;
  }
  hipLaunchKernelGGL(ddae_select, dim3(p.B), dim3(kSelThreads), 0, stream, p);
  pace_status_t st = check_launch("ddae_select");
  if (st != PACE_OK) return st;
  const int ktot = p.cu_keep[p.B];
  if (hidden != nullptr && ktot > 0) {
    const int words = static_cast<int>(row_bytes / 16);
    hipLaunchKernelGGL(gather_rows, dim3(ktot), dim3(256), 0, stream,
                       static_cast<const uint4*>(hidden), p.idx, static_cast<uint4*>(out), ktot,
                       words, p.nv_total);
    st = check_launch("gather_rows");
    if (st != PACE_OK) return st;
  }
  return PACE_OK;
}

void size_select(Sizer& s, int nv_total, int nseg) {
  s.take<float>(nv_total);   // vraw
  s.take<float>(nv_total);   // lraw
  s.take<float>(nv_total);   // scores (when the caller passes none)
  s.take<float>(4 * nseg);   // fusion stats (when the caller passes none)
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
  PACE_REQUIRE(B >= 1 && B <= PACE_MAX_SEGMENTS, "pace_ddae_select: B=%d not in [1, %d]", B,
               PACE_MAX_SEGMENTS);
  PACE_REQUIRE(nv_host && keep_host, "pace_ddae_select: null host count arrays");
  PACE_REQUIRE(Hv >= 1 && Hl >= 1 && merge >= 1, "pace_ddae_select: Hv=%d Hl=%d merge=%d", Hv, Hl,
               merge);
  PACE_REQUIRE(mode == 0 || mode == 1, "pace_ddae_select: mode=%d must be 0 or 1", mode);
  PACE_REQUIRE(mode == 1 || (tau > 0.f && isfinite(tau)), "pace_ddae_select: tau must be > 0");
  PACE_REQUIRE(vis_mass && llm_mass && idx_out, "pace_ddae_select: null device pointer");
  SelectParams p{};
  p.cu_nv[0] = 0;
  p.cu_keep[0] = 0;
  for (int b = 0; b < B; ++b) {
    PACE_REQUIRE(nv_host[b] >= 1, "pace_ddae_select: image %d has %d tokens", b, nv_host[b]);
    PACE_REQUIRE(keep_host[b] >= 0 && keep_host[b] <= nv_host[b],
                 "pace_ddae_select: K=%d outside [0, %d] for image %d", keep_host[b], nv_host[b], b);
    PACE_REQUIRE(static_cast<long long>(p.cu_nv[b]) + nv_host[b] < (1ll << 30),
                 "pace_ddae_select: too many tokens");
    p.cu_nv[b + 1] = p.cu_nv[b] + nv_host[b];
    p.cu_keep[b + 1] = p.cu_keep[b] + keep_host[b];
  }
  const int nv_total = p.cu_nv[B];
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
  Carver c(workspace, workspace_bytes);
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
  p.Hv = Hv; p.merge = merge; p.Hl = Hl; p.B = B; p.nv_total = nv_total;
  p.mode = mode; p.tau = tau; p.w_llm_fixed = w_llm_fixed;
  return run_select(p, hidden, row_bytes, out, stream, true);
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
