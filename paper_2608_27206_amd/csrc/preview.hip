// APC's shallow feature preview (Section 3.2, "Shallow Feature Preview": the vision encoder's
// initial block, K = 1, at the original resolution): patch embedding, RMSNorm, window
// attention with residual, RMSNorm and SwiGLU MLP with residual, with caller-supplied weights.
// Its token embeddings feed pace_apc_density_features.
//
// Kernels:
//   preview_patchify  patch pixels (x/127.5 - 1) in the caller's token order, bf16, rows
//                     zero-padded to a multiple of 8 values
//   gemm_bf16_nt      C = A B^T on bf16 MFMA (32x32x16), fp32 accumulation, with the block's
//                     epilogues fused: + bias, + residual, or SwiGLU of interleaved gate/up
//                     columns; bf16 out
//   rmsnorm_bf16      one wave per row
// The attention step is pace_vit_attention over the windows.
#include <math.h>

#include "pace_internal.h"

namespace pace {
namespace {

typedef __bf16 gbf16x8 __attribute__((ext_vector_type(8)));
typedef float gf32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (finite values)
  return static_cast<uint16_t>(u >> 16);
}
__device__ __forceinline__ float from_bf16(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// ---------------------------------------------------------------- patchify
__global__ __launch_bounds__(256) void preview_patchify(const uint8_t* __restrict__ img, int W, int P, int gw,
                                                        const int32_t* __restrict__ order, int N, int Kp,
                                                        uint16_t* __restrict__ X) {
  const long long idx = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<long long>(N) * Kp) return;
  const int t = static_cast<int>(idx / Kp), e = static_cast<int>(idx - static_cast<long long>(t) * Kp);
  float v = 0.f;
  if (e < 3 * P * P) {
    const int r = e / (3 * P), rem = e - r * 3 * P;
    const int c = rem / 3, ch = rem - c * 3;
    const int patch = order[t];
    const int py = patch / gw, px = patch - py * gw;
    const long long off = (static_cast<long long>(py * P + r) * W + px * P + c) * 3 + ch;
    v = static_cast<float>(img[off]) * (1.0f / 127.5f) - 1.0f;
  }
  X[idx] = to_bf16(v);
}

// ---------------------------------------------------------------- GEMM
// C[M, N] = A[M, K] B[N, K]^T.  A 128x128 output tile per workgroup, 4 waves of 64x64 (2x2
// MFMA tiles of 32x32), K in steps of 32 through LDS, double buffered: the global loads of step
// t+1 are in flight while step t is multiplied.  Rows past M or N and columns past K load as
// zeros (range-checked buffer loads), so tails need no branches.
constexpr int kGM = 128, kGN = 128, kGK = 32;
constexpr int kGS = kGK + 8;   // LDS row stride (elements)

enum { kEpiBias = 0, kEpiResidual = 1, kEpiSwiglu = 2 };

struct GemmParams {
  const uint16_t* A;
  const uint16_t* B;
  const float* bias;     // [N] or null
  const uint16_t* R;     // residual [M, N] (kEpiResidual)
  uint16_t* C;           // [M, N], or [M, N / 2] for kEpiSwiglu
  int M, N, K;
  int lda, ldb, ldc, ldr;
  int mode;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t grsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
constexpr unsigned kGOut = 0x7FFFFFF0u;

__global__ __launch_bounds__(256, 2) void gemm_bf16_nt(const GemmParams p) {
  __shared__ __align__(16) uint16_t As[2][kGM * kGS];
  __shared__ __align__(16) uint16_t Bs[2][kGN * kGS];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, c32 = lane & 31;
  const int bm = blockIdx.y * kGM, bn = blockIdx.x * kGN;
  const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
  const auto ra = grsrc(p.A, static_cast<unsigned>(static_cast<long long>(p.M) * p.lda * 2));
  const auto rb = grsrc(p.B, static_cast<unsigned>(static_cast<long long>(p.N) * p.ldb * 2));
  // this thread's two 16-byte chunks of each tile: chunk c = tid + 256 u -> row c / 4, k chunk c % 4
  int arow[2], brow[2], kc[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = tid + 256 * u;
    arow[u] = c >> 2;
    brow[u] = c >> 2;
    kc[u] = (c & 3) * 8;
  }
  auto load = [&](int k0, uint4* va, uint4* vb) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = k0 + kc[u];
      const bool kok = k < p.K;
      const int ma = bm + arow[u], nb = bn + brow[u];
      const unsigned oa = (kok && ma < p.M) ? static_cast<unsigned>((static_cast<long long>(ma) * p.lda + k) * 2) : kGOut;
      const unsigned ob = (kok && nb < p.N) ? static_cast<unsigned>((static_cast<long long>(nb) * p.ldb + k) * 2) : kGOut;
      va[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, oa, 0, 0));
      vb[u] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, ob, 0, 0));
    }
  };
  auto store = [&](int buf, const uint4* va, const uint4* vb) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      *reinterpret_cast<uint4*>(&As[buf][arow[u] * kGS + kc[u]]) = va[u];
      *reinterpret_cast<uint4*>(&Bs[buf][brow[u] * kGS + kc[u]]) = vb[u];
    }
  };
  gf32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = gf32x16{};
  const int nk = (p.K + kGK - 1) / kGK;
  uint4 va[2], vb[2];
  load(0, va, vb);
  store(0, va, vb);
  __syncthreads();
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) load((t + 1) * kGK, va, vb);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      gbf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const gbf16x8*>(&As[buf][(wm + 32 * i + c32) * kGS + kk * 16 + g * 8]);
        b[i] = *reinterpret_cast<const gbf16x8*>(&Bs[buf][(wn + 32 * i + c32) * kGS + kk * 16 + g * 8]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (t + 1 < nk) store(buf ^ 1, va, vb);
    __syncthreads();
  }
  // epilogue: register 4 jj + ii of tile (i, j) is row wm + 32 i + 8 jj + 4 g + ii, column
  // wn + 32 j + c32
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = bn + wn + 32 * j + c32;
    const float bias = (p.bias != nullptr && n < p.N) ? p.bias[n] : 0.f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = bm + wm + 32 * i + 8 * (r >> 2) + 4 * g + (r & 3);
        float v = acc[i][j][r] + bias;
        if (p.mode == kEpiSwiglu) {
          // columns 2f (gate) and 2f + 1 (up) sit in neighbouring lanes
          const float other = __shfl_xor(v, 1, 64);
          if ((c32 & 1) == 0 && m < p.M && n < p.N) {
            const float gate = v, up = other;
            p.C[static_cast<long long>(m) * p.ldc + (n >> 1)] = to_bf16(gate / (1.0f + expf(-gate)) * up);
          }
        } else if (m < p.M && n < p.N) {
          if (p.mode == kEpiResidual) v += from_bf16(p.R[static_cast<long long>(m) * p.ldr + n]);
          p.C[static_cast<long long>(m) * p.ldc + n] = to_bf16(v);
        }
      }
  }
}

// ---------------------------------------------------------------- RMSNorm
struct NormAdd { __device__ float operator()(float a, float b) const { return a + b; } };

// y = x / sqrt(mean(x^2) + eps) * gamma, one wave per row, rows of D values (D % 8 == 0).
__global__ __launch_bounds__(256) void rmsnorm_bf16(const uint16_t* __restrict__ x, const float* __restrict__ gamma,
                                                    uint16_t* __restrict__ y, int M, int D, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const uint4* xr = reinterpret_cast<const uint4*>(x + static_cast<long long>(row) * D);
  uint4* yr = reinterpret_cast<uint4*>(y + static_cast<long long>(row) * D);
  const int nch = D / 8;
  float ss = 0.f;
  for (int c = lane; c < nch; c += 64) {
    const uint4 v = xr[c];
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float a = __uint_as_float(u[q] << 16), b = __uint_as_float(u[q] & 0xFFFF0000u);
      ss += a * a + b * b;
    }
  }
  ss = wave_reduce_dpp(ss, NormAdd{});
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
  for (int c = lane; c < nch; c += 64) {
    const uint4 v = xr[c];
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = c * 8 + 2 * q;
      const float a = __uint_as_float(u[q] << 16) * inv * gamma[e];
      const float b = __uint_as_float(u[q] & 0xFFFF0000u) * inv * gamma[e + 1];
      o[q] = static_cast<uint32_t>(to_bf16(a)) | (static_cast<uint32_t>(to_bf16(b)) << 16);
    }
    yr[c] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

pace_status_t launch_gemm(const GemmParams& p, hipStream_t stream) {
  dim3 grid((p.N + kGN - 1) / kGN, (p.M + kGM - 1) / kGM);
  hipLaunchKernelGGL(gemm_bf16_nt, grid, dim3(256), 0, stream, p);
  return check_launch("gemm_bf16_nt");
}

}  // namespace
}  // namespace pace

using namespace pace;

extern "C" {

pace_status_t pace_gemm_bf16(const uint16_t* A, const uint16_t* B, const float* bias, const uint16_t* residual,
                             uint16_t* C, int M, int N, int K, int epilogue, hipStream_t stream) {
  PACE_REQUIRE(A && B && C, "pace_gemm_bf16: null device pointer");
  PACE_REQUIRE(M >= 1 && N >= 1 && K >= 8 && K % 8 == 0,
               "pace_gemm_bf16: M=%d N=%d K=%d (K a positive multiple of 8)", M, N, K);
  PACE_REQUIRE(aligned16(A) && aligned16(B), "pace_gemm_bf16: A and B must be 16-byte aligned");
  PACE_REQUIRE(epilogue >= 0 && epilogue <= 2, "pace_gemm_bf16: epilogue %d not in {0, 1, 2}", epilogue);
  PACE_REQUIRE(epilogue != 1 || residual != nullptr, "pace_gemm_bf16: residual epilogue without residual");
  PACE_REQUIRE(epilogue != 2 || N % 2 == 0, "pace_gemm_bf16: SwiGLU needs an even N");
  PACE_REQUIRE(static_cast<long long>(M) * K * 2 < (1ll << 30) && static_cast<long long>(N) * K * 2 < (1ll << 30),
               "pace_gemm_bf16: an operand spans 1 GiB or more");
  GemmParams p{};
  p.A = A; p.B = B; p.bias = bias; p.R = residual; p.C = C;
  p.M = M; p.N = N; p.K = K;
  p.lda = K; p.ldb = K; p.ldc = (epilogue == 2) ? N / 2 : N; p.ldr = N;
  p.mode = epilogue;
  return launch_gemm(p, stream);
}

size_t pace_apc_preview_workspace_size(int N, int dim, int ffn, int patch) {
  if (N <= 0 || dim <= 0 || ffn <= 0 || patch <= 0) return 0;
  const int kp = (3 * patch * patch + 7) / 8 * 8;
  Sizer s;
  s.take<uint16_t>(static_cast<size_t>(N) * kp);        // patch rows
  for (int i = 0; i < 7; ++i) s.take<uint16_t>(static_cast<size_t>(N) * dim);   // h0 u q k v o h1
  s.take<uint16_t>(static_cast<size_t>(N) * ffn);       // SwiGLU hidden
  return s.off;
}

pace_status_t pace_apc_preview(const uint8_t* img, int H, int W, int patch, const int32_t* token_patch,
                               const int32_t* cu_windows, int nwin, int max_window,
                               const pace_preview_weights* w, uint16_t* out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(img && token_patch && cu_windows && w && out, "pace_apc_preview: null pointer");
  PACE_REQUIRE(patch >= 1 && patch <= 16 && H >= patch && W >= patch && H % patch == 0 && W % patch == 0,
               "pace_apc_preview: H=%d W=%d must be multiples of patch=%d (1..16)", H, W, patch);
  const int gh = H / patch, gw = W / patch;
  const long long Nl = static_cast<long long>(gh) * gw;
  PACE_REQUIRE(Nl < (1 << 24), "pace_apc_preview: too many patches");
  const int N = static_cast<int>(Nl);
  const int D = w->dim, F = w->ffn;
  PACE_REQUIRE(D >= 80 && D % 80 == 0 && F >= 8 && F % 8 == 0,
               "pace_apc_preview: dim=%d must be a multiple of 80 and ffn=%d of 8", D, F);
  PACE_REQUIRE(nwin >= 1 && max_window >= 1 && max_window <= N && max_window < 1024,
               "pace_apc_preview: nwin=%d max_window=%d (windows are shorter than 1024 tokens)", nwin, max_window);
  PACE_REQUIRE(w->pe && w->g1 && w->wq && w->wk && w->wv && w->wo && w->g2 && w->wgu && w->wd,
               "pace_apc_preview: a weight pointer is null");
  PACE_REQUIRE(aligned16(out), "pace_apc_preview: out must be 16-byte aligned");
  const int kp = (3 * patch * patch + 7) / 8 * 8;
  const size_t need = pace_apc_preview_workspace_size(N, D, F, patch);
  if (workspace == nullptr || workspace_bytes < need)
    return set_error(PACE_ERR_WORKSPACE, "pace_apc_preview: workspace %zu < %zu bytes", workspace_bytes, need);
  pace_status_t st = check_offsets(cu_windows, nwin, N, max_window, "pace_apc_preview: cu_windows", stream);
  if (st != PACE_OK) return st;
  if (debug_checks()) {
    st = check_values(token_patch, N, nullptr, 0, N - 1, "pace_apc_preview: token_patch", stream);
    if (st != PACE_OK) return st;
  }
  Carver c(workspace, workspace_bytes);
  uint16_t* X = c.take<uint16_t>(static_cast<size_t>(N) * kp);
  uint16_t* h0 = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* u = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* q = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* k = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* v = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* o = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* h1 = c.take<uint16_t>(static_cast<size_t>(N) * D);
  uint16_t* hm = c.take<uint16_t>(static_cast<size_t>(N) * F);

  const long long total = static_cast<long long>(N) * kp;
  hipLaunchKernelGGL(preview_patchify, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0, stream,
                     img, W, patch, gw, token_patch, N, kp, X);
  if ((st = check_launch("preview_patchify")) != PACE_OK) return st;
  if ((st = pace_gemm_bf16(X, w->pe, nullptr, nullptr, h0, N, D, kp, 0, stream)) != PACE_OK) return st;
  hipLaunchKernelGGL(rmsnorm_bf16, dim3((N + 3) / 4), dim3(256), 0, stream, h0, w->g1, u, N, D, 1e-6f);
  if ((st = check_launch("rmsnorm_bf16")) != PACE_OK) return st;
  if ((st = pace_gemm_bf16(u, w->wq, w->bq, nullptr, q, N, D, D, 0, stream)) != PACE_OK) return st;
  if ((st = pace_gemm_bf16(u, w->wk, w->bk, nullptr, k, N, D, D, 0, stream)) != PACE_OK) return st;
  if ((st = pace_gemm_bf16(u, w->wv, w->bv, nullptr, v, N, D, D, 0, stream)) != PACE_OK) return st;
  if ((st = pace_vit_attention(q, k, v, N, D / 80, 80, cu_windows, nwin, max_window, 1.0f / sqrtf(80.f), o,
                               nullptr, nullptr, nullptr, 0, stream)) != PACE_OK)
    return st;
  if ((st = pace_gemm_bf16(o, w->wo, w->bo, h0, h1, N, D, D, 1, stream)) != PACE_OK) return st;
  hipLaunchKernelGGL(rmsnorm_bf16, dim3((N + 3) / 4), dim3(256), 0, stream, h1, w->g2, u, N, D, 1e-6f);
  if ((st = check_launch("rmsnorm_bf16")) != PACE_OK) return st;
  if ((st = pace_gemm_bf16(u, w->wgu, w->bgu, nullptr, hm, N, 2 * F, D, 2, stream)) != PACE_OK) return st;
  return pace_gemm_bf16(hm, w->wd, w->bd, h1, out, N, D, F, 1, stream);
}

}  // extern "C"
