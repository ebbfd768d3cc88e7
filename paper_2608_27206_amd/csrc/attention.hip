// Attention with per-key mass for the two read-outs DDAE fuses (Section 3.3): the
// vision encoder's self-attention (window and full segments; S_vis from the full
// block) and the LLM's causal grouped-query prefill attention (S_llm from the text
// query rows).  No attention matrix is ever stored.
//
// The kernels (MFMA 32x32x16, bf16 inputs except the fp16 PV product of attn_fwd_rot, fp32
// accumulation):
//
//  attn_fwd   query-stationary.  A workgroup = 4 waves x 32 query rows of one
//             (segment, head).  K and V tiles of 64 keys are staged through LDS by
//             DMA (double buffered).  Each wave computes S^T = K Q^T so that every
//             lane owns one query row (the MFMA accumulator column) and 16 keys of it:
//             the row max and row sum are in-lane, plus one exchange between the two
//             half-waves.  Online softmax in the log2 domain, P^T feeds O^T = V^T P^T
//             straight from registers (no LDS round trip); V^T comes from transposing
//             LDS reads of the row-major V tile.  For head dim 80 the PV product is
//             padded to 96 rows.  Writes O (bf16, through LDS so that each row is stored
//             contiguously) and the natural-log LSE (fp32).  Causal segments (the
//             prefill), short segments and head dim 128.
//
//  attn_fwd_rot  the same computation for long segments at head dim 80, with 12 waves
//             per workgroup in three groups that rotate through three phases (see the
//             kernel), so that VALU and MFMA work of different waves overlap; its PV
//             product runs in fp16 on V^T tiles that attn_vt_clear + attn_v_amax +
//             attn_vt_prep write once per call (scaled per segment and KV head into fp16's
//             range, a row of ones for the row sums).
//
//  attn_window  segments of at most 64 tokens (the 8x8-patch windows): O, LSE and the
//             per-key mass in one pass, since a window's row max and sum are final after
//             its single key tile; O goes out through LDS, row by row.
//
//  attn_mass  key-stationary.  A workgroup = 4 waves x 64 keys of one (segment,
//             head); K stays in registers, query tiles of 64 rows stream through LDS
//             (three buffers, up to three workgroups per CU).  P = exp2(S * scale * log2 e -
//             LSE * log2 e) is the exact normalised probability; each lane accumulates
//             column sums for its 16 keys in fp32, and one butterfly over the half-wave
//             finishes the sum.  Writes mass[h, key] once (no atomics, deterministic).  At
//             head dim 80 without a mask it is pipelined inside each wave, one 32 x 32
//             block at a time.
//
// Operand layouts of v_mfma_f32_32x32x16_bf16 (wave64, lane l, g = l / 32):
//   A (32 x 16): lane l holds A[l % 32][8g .. 8g+7]
//   B (16 x 32): lane l holds B[8g .. 8g+7][l % 32]
//   C (32 x 32): lane l holds C[8j + 4g + i][l % 32] in register 4j + i (j, i < 4)
// The k index within a chunk is only ever contracted, so both operands may use any
// common permutation of it.
#include <math.h>

#include <type_traits>

#include <vector>

#include "pace_internal.h"

namespace pace {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) {
  bf16x8 r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &r, 4);
  return u;
}

__device__ __forceinline__ bf16x8 pack_bf16x8(const float* x) {
  uint4 u;
  u.x = pack_bf16x2(x[0], x[1]);
  u.y = pack_bf16x2(x[2], x[3]);
  u.z = pack_bf16x2(x[4], x[5]);
  u.w = pack_bf16x2(x[6], x[7]);
  return as_bf16x8(u);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// max of three floats in one instruction.  fmaxf on values fresh from an MFMA costs an extra
// canonicalising v_max per operand; the inputs here are finite or -inf, never NaN, so the
// plain instruction gives the same result.
__device__ __forceinline__ float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Buffer resource over `bytes` bytes from `base`: loads at offsets past the end return 0
// (the hardware range check), so tile loads need neither branches nor clamps.  The whole
// offset always goes in the VGPR operand, which the range check covers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
constexpr unsigned kOutOfRange = 0x7FFFFFF0u;

// A wave's 32 query rows of O, stored through LDS.  Lane (c32, g) holds in its O^T
// accumulators the values dv = 32 t2 + 8 j + 4 g + i of row c32; they go to the wave's own
// LDS rows (`stage`, stride D + 8) as bf16 of value * inv_l * 2^unshift, then each lane stores
// 16-byte chunks, so each row's D values are written contiguously (straight from the
// accumulators, every store instruction wrote 8-byte pieces of 32 rows one token apart, which
// the write path serves far more slowly).  `ro` covers the segment's rows of this head, row0
// is the wave's first row in it; rows at or past the segment end fall outside `ro` and are
// dropped.  Every wave of the workgroup calls this once its last LDS read is behind a
// workgroup barrier (the staging rows overlay the tile buffers).
template <int D, int NT>
__device__ __forceinline__ void store_o_staged(const f32x16 (&oacc)[NT], float inv_l, int unshift,
                                               uint16_t* stage, __amdgpu_buffer_rsrc_t ro, int row0,
                                               int qstride) {
  constexpr int OS = D + 8, CPR = D / 8;
  const int lane = threadIdx.x & 63, g = lane >> 5, c32 = lane & 31;
#pragma unroll
  for (int t2 = 0; t2 < NT; ++t2) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dv = t2 * 32 + g * 4 + 8 * j;
      if (dv < D) {
        float ov[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) ov[i] = __builtin_amdgcn_ldexpf(oacc[t2][4 * j + i] * inv_l, unshift);
        uint2 pk;
        pk.x = pack_bf16x2(ov[0], ov[1]);
        pk.y = pack_bf16x2(ov[2], ov[3]);
        *reinterpret_cast<uint2*>(&stage[c32 * OS + dv]) = pk;
      }
    }
  }
  __syncthreads();
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int c = lane; c < 32 * CPR; c += 64) {
    const int r = c / CPR, cc = c - (c / CPR) * CPR;
    const u32x4 val = *reinterpret_cast<const u32x4*>(&stage[r * OS + cc * 8]);
    __builtin_amdgcn_raw_buffer_store_b128(val, ro, static_cast<unsigned>((row0 + r) * qstride + cc * 8) * 2u, 0, 0);
  }
}

typedef __attribute__((address_space(3))) const char lds_char;
typedef int i32x4 __attribute__((ext_vector_type(4)));

// The same buffer resource as four scalar words, for the DMA below.
__device__ __forceinline__ i32x4 make_dma_rsrc(const void* base, unsigned bytes) {
  const unsigned long long a = reinterpret_cast<unsigned long long>(base);
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(a & 0xffffffffull));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<int>((a >> 32) & 0xffffull));   // stride 0
  r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
  r.w = 0x00020000;
  return r;
}

// Buffer-to-LDS DMA: every lane's 16 bytes land at lds + 16 * lane (lds is wave-uniform);
// lanes whose offset is out of range write zeros.  Issued from inline assembly so that the
// compiler does not track it: otherwise it places a wait for every DMA in flight before
// each later LDS read, which would stall on the prefetch just issued.  Completion is
// awaited explicitly with wait_vmem() and a barrier before the tile is read.
__device__ __forceinline__ unsigned lds_u32(const void* p) {
  return static_cast<unsigned>(reinterpret_cast<unsigned long long>((const lds_char*)p));
}
__device__ __forceinline__ void dma16(i32x4 r, unsigned lds, unsigned voff) {
  const unsigned m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :: "v"(voff), "s"(r), "{m0}"(m0) : "memory");
}
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// The same resource moved `bytes` forward (base up, size down by the same amount): an offset v
// into the result reads what v + bytes reads from the original, range check included.  Scalar
// arithmetic only, so a loop that walks tiles keeps its per-lane offsets constant.
__device__ __forceinline__ i32x4 rsrc_advance(i32x4 r, unsigned bytes) {
  const unsigned long long a =
      ((static_cast<unsigned long long>(static_cast<unsigned>(r.y)) & 0xffffull) << 32 | static_cast<unsigned>(r.x)) + bytes;
  r.x = static_cast<int>(a & 0xffffffffull);
  r.y = (r.y & ~0xffff) | static_cast<int>((a >> 32) & 0xffffull);
  r.z = static_cast<int>(static_cast<unsigned>(r.z) - bytes);
  return r;
}
// As dma16 with 4 bytes per lane (lds + 4 * lane).
__device__ __forceinline__ void dma4(i32x4 r, unsigned lds, unsigned voff) {
  const unsigned m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds"
               :: "v"(voff), "s"(r), "{m0}"(m0) : "memory");
}
// Waits until at most n (wave-uniform, <= 7) of this wave's vector memory operations are
// outstanding: the older ones, issued first, have completed.
__device__ __forceinline__ void wait_vmem_upto(int n) {
  switch (n) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(1)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt vmcnt(3)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt vmcnt(5)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(7)" ::: "memory"); break;
  }
}

// Compile-time loop: f(integral_constant<int, I>) for I in [B, E), so register arrays
// are only ever indexed by constants.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ---------------------------------------------------------------- forward
struct FwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;              // [Hq, Ntot] or null
  const int32_t* cu;       // [nseg + 1]
  int Ntot, Hq, Hkv, group;
  int nseg, nqt;           // q tiles per segment in the grid
  float scale_log2;        // scale * log2(e)
  const uint16_t* vt;      // fp16 V^T tiles (rotation kernel only)
  long long vt_cols;
  const uint32_t* vt_amax; // [nseg, Hkv] largest |v| per (segment, KV head) as bf16 bits (rotation only)
};

constexpr int kBM = 128;   // query rows per workgroup
constexpr int kBN = 64;    // keys per tile
constexpr int kThreads = 256;

template <int D>
struct FwdCfg {
  static constexpr int DV = (D == 80) ? 96 : D;   // PV rows incl. padding
  static constexpr int NT = DV / 32;              // O^T accumulator tiles
  static constexpr int KC = D / 16;               // QK^T k-chunks
  static constexpr int KS = D + 8;                // LDS row stride of K (elements)
  static constexpr int VS = D + 16;               // LDS row stride of V (elements)
  static constexpr int KROW = KS / 8;             // 16-byte chunks per K row (incl. padding)
  static constexpr int VROW = VS / 8;             // 16-byte chunks per V row (incl. padding)
  static constexpr int KINST = kBN * KROW / 64;   // wave-wide DMA loads per K tile
  static constexpr int VINST = kBN * VROW / 64;   // wave-wide DMA loads per V tile
  static constexpr int KPW = (KINST + 3) / 4;     // per wave (4 waves)
  static constexpr int VPW = (VINST + 3) / 4;
};

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

// ds_read_b64_tr_b16: within each 16-lane group, destination lane i, slot j receives
// element (i % 4) of the 8 bytes addressed by source lane 4j + i/4.
__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
  v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
  uint2 u;
  __builtin_memcpy(&u, &r, 8);
  return u;
}

// Rows whose running max grows by less than this (log2 units) keep their old max:
// probabilities then stay below 2^8, harmless in fp32 accumulators and bf16 operands,
// and the O accumulators are rescaled only when some row's max really moves.
constexpr float kRescaleSlack = 8.0f;

// The forward kernel.  Per 64-key tile t, every wave:
//   - issues S^T(t+1) = K(t+1) Q^T on the MFMA pipe (K runs one tile ahead in LDS),
//   - runs the online softmax of S^T(t) on the VALU while those MFMAs execute,
//   - accumulates O^T += V(t)^T P^T(t).
// K and V tiles are row-major in LDS.  The A operand V^T of the PV product is read with
// transposing LDS reads whose source addresses also apply the key permutation that
// matches the accumulator layout of P^T: A slot (g, 4*rd + j) holds key 8*rd + 4*g + j of
// each 16-key chunk.
template <int D, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd(const FwdParams p) {
  using C = FwdCfg<D>;
  __shared__ __align__(16) uint16_t Ks[2][kBN * C::KS];
  __shared__ __align__(16) uint16_t Vs[2][kBN * C::VS];

  const int lb = remap_block_id(blockIdx.x, gridDim.x);
  const int per_head = p.nseg * p.nqt;
  const int h = lb / per_head;
  const int rem = lb - h * per_head;
  const int seg = rem / p.nqt;
  int qt = rem - seg * p.nqt;
  if (CAUSAL) qt = p.nqt - 1 - qt;   // longest causal rows first
  const int s0 = p.cu[seg];
  const int L = p.cu[seg + 1] - s0;
  const int q0 = qt * kBM;
  if (q0 >= L) return;
  const int kvh = h / p.group;
  // the wave index is wave-uniform: keep it in an SGPR (DMA destinations must be uniform)
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 5, c32 = lane & 31;
  const int qrow = q0 + w * 32 + c32;
  const int qstride = p.Hq * D;
  const int kvstride = p.Hkv * D;
  const uint16_t* kbase = p.k + static_cast<long long>(s0) * kvstride + kvh * D;
  const uint16_t* vbase = p.v + static_cast<long long>(s0) * kvstride + kvh * D;

  // Q, K and V of this (segment, head) as buffer resources: rows past the segment end fall
  // outside the range and load as zeros.
  const unsigned seg_bytes_q = static_cast<unsigned>((L - 1) * qstride + D) * 2u;
  const unsigned seg_bytes_kv = static_cast<unsigned>((L - 1) * kvstride + D) * 2u;
  const auto rq = make_rsrc(p.q + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q);
  const auto rk = make_dma_rsrc(kbase, seg_bytes_kv);
  const auto rv = make_dma_rsrc(vbase, seg_bytes_kv);

  bf16x8 qf[C::KC];
  {
    const unsigned qoff = static_cast<unsigned>(qrow * qstride + g * 8) * 2u;
#pragma unroll
    for (int c = 0; c < C::KC; ++c) qf[c] = as_bf16x8(buf_load16(rq, qoff + c * 32, 0));
  }

  // Tile loads go straight from the buffers to LDS (DMA), 64 16-byte chunks per wave-wide
  // load, chunks in LDS order: chunk c of a tile is row c / ROW, column chunk c % ROW; the
  // padding column of each row reads out of range (zeros).  Wave w issues loads w, w+4, ...
  unsigned koff[C::KPW], voff[C::VPW];
  static_for<0, C::KPW>([&](auto I) __attribute__((always_inline)) {
    const int c = (w + 4 * I) * 64 + lane;
    const int r = c / C::KROW, cc = c % C::KROW;
    koff[I] = (cc < D / 8 && w + 4 * I < C::KINST) ? static_cast<unsigned>(r * kvstride + cc * 8) * 2u
                                                    : kOutOfRange;
  });
  static_for<0, C::VPW>([&](auto I) __attribute__((always_inline)) {
    const int c = (w + 4 * I) * 64 + lane;
    const int r = c / C::VROW, cc = c % C::VROW;
    voff[I] = (cc < D / 8 && w + 4 * I < C::VINST) ? static_cast<unsigned>(r * kvstride + cc * 8) * 2u
                                                    : kOutOfRange;
  });
  const unsigned tile_bytes = static_cast<unsigned>(kBN * kvstride) * 2u;
  const unsigned ks_lds = lds_u32(&Ks[0][0]), vs_lds = lds_u32(&Vs[0][0]);
  auto load_k = [&](int t, int buf) __attribute__((always_inline)) {
    static_for<0, C::KPW>([&](auto I) __attribute__((always_inline)) {
      if (w + 4 * I < C::KINST) dma16(rk, ks_lds + (buf * kBN * C::KS + (w + 4 * I) * 512) * 2, koff[I] + t * tile_bytes);
    });
  };
  auto load_v = [&](int t, int buf) __attribute__((always_inline)) {
    static_for<0, C::VPW>([&](auto I) __attribute__((always_inline)) {
      if (w + 4 * I < C::VINST) dma16(rv, vs_lds + (buf * kBN * C::VS + (w + 4 * I) * 512) * 2, voff[I] + t * tile_bytes);
    });
  };

  // transposed-read source addresses (elements, within a V tile) for this lane
  const int grp = lane >> 4, li = lane & 15;
  const int tr_row = 4 * (grp >> 1) + (li >> 2);          // + 8*rd + 16*chunk
  const int tr_col = 16 * (grp & 1) + 4 * (li & 3);       // + 32*t (dv)
  const int tr_base = tr_row * C::VS + tr_col;

  auto qk = [&](int buf, f32x16* s) __attribute__((always_inline)) {
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const uint16_t* kp = &Ks[buf][(st * 32 + c32) * C::KS + g * 8];
      bf16x8 kf[C::KC];
#pragma unroll
      for (int c = 0; c < C::KC; ++c) kf[c] = *reinterpret_cast<const bf16x8*>(kp + c * 16);
      s[st] = mfma(kf[0], qf[0], f32x16{});
#pragma unroll
      for (int c = 1; c < C::KC; ++c) s[st] = mfma(kf[c], qf[c], s[st]);
    }
  };

  f32x16 oacc[C::NT];
#pragma unroll
  for (int t = 0; t < C::NT; ++t) oacc[t] = f32x16{};
  float m_used = -INFINITY;   // max used in the exponentials (log2 domain), per query row
  float l_part[4] = {0.f, 0.f, 0.f, 0.f};   // this lane's share of the row sum, 4 chains

  // Masks, tile max and the (rare) rescale of the accumulators for the tile in s.
  auto tile_max = [&](f32x16* s, int kt) __attribute__((always_inline)) {
    const bool need_mask = (kt + kBN > L) || (CAUSAL && kt + kBN - 1 > q0 + w * 32);
    if (need_mask) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt + st * 32 + g * 4 + 8 * (r >> 2) + (r & 3);
          const bool ok = (key < L) && (!CAUSAL || key <= qrow);
          if (!ok) s[st][r] = -INFINITY;
        }
    }
    // max over the 32 in-lane values in 16 three-input maxima (10 triples, the last pair folded
    // into the first), then across the half-waves, which hold the same query rows
    float m1[10];
#pragma unroll
    for (int i = 0; i < 10; ++i) {
      const int a = 3 * i;
      m1[i] = vmax3(s[a >> 4][a & 15], s[(a + 1) >> 4][(a + 1) & 15], s[(a + 2) >> 4][(a + 2) & 15]);
    }
    m1[0] = vmax3(m1[0], s[1][14], s[1][15]);
    const float m2a = vmax3(m1[0], m1[1], m1[2]), m2b = vmax3(m1[3], m1[4], m1[5]);
    const float m2c = vmax3(m1[6], m1[7], m1[8]);
    float mx = vmax3(vmax3(m2a, m2b, m2c), m1[9], m1[9]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = vmax3(__uint_as_float(sw[0]), __uint_as_float(sw[1]), __uint_as_float(sw[1])) * p.scale_log2;
    }
    // lazy rescale: only when some row's max moved up by more than the slack
    if (__builtin_amdgcn_ballot_w64(mx > m_used + kRescaleSlack) != 0ull) {
      const float m_new = fmaxf(m_used, mx);
      const float alpha = fast_exp2(m_used - m_new);
      m_used = m_new;
#pragma unroll
      for (int t2 = 0; t2 < C::NT; ++t2)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t2][r] *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i) l_part[i] *= alpha;
    }
  };

  // exp, row sum and bf16 packing of the tile in s, then O^T += V^T P^T (buffer BUF)
  auto exp_pv = [&](f32x16* s, int buf) __attribute__((always_inline)) {
    const float m_off = (m_used == -INFINITY) ? 0.f : m_used;
    bf16x8 pb[2][2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      float pv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        pv[r] = fast_exp2(s[st][r] * p.scale_log2 - m_off);
        l_part[r & 3] += pv[r];
      }
      pb[st][0] = pack_bf16x8(&pv[0]);
      pb[st][1] = pack_bf16x8(&pv[8]);
    }
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const uint16_t* vp = &Vs[buf][(st * 32 + hh * 16) * C::VS + tr_base];
#pragma unroll
        for (int t2 = 0; t2 < C::NT; ++t2) {
          const uint2 lo = lds_read_tr16(vp + t2 * 32);
          const uint2 hi = lds_read_tr16(vp + 8 * C::VS + t2 * 32);
          oacc[t2] = mfma(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pb[st][hh], oacc[t2]);
        }
      }
  };

  const int kend = CAUSAL ? min(L, q0 + kBM) : L;
  const int ntiles = (kend + kBN - 1) / kBN;
  // prologue: K(0) and V(0) into buffer 0, K(1) into buffer 1
  load_k(0, 0);
  load_v(0, 0);
  if (ntiles > 1) load_k(1, 1);
  wait_vmem();
  __syncthreads();
  f32x16 sa[2], sb[2];
  qk(0, sa);

  // Iteration t: K(t+1) and V(t) are in LDS.  DMA K(t+2) and V(t+1) into the buffers that
  // held K(t) and V(t-1) (every wave is past their last use: it passed this barrier), then
  // one straight-line region interleaves S^T(t+1) = K(t+1) Q^T on the MFMA pipe with the
  // exponentials of tile t on the VALU, and O^T += V(t)^T P^T(t).
  auto iteration = [&](auto BUF, auto HAS_NEXT, int t, f32x16* s_cur, f32x16* s_next)
      __attribute__((always_inline)) {
    constexpr int buf = decltype(BUF)::value;
    constexpr bool has_next = decltype(HAS_NEXT)::value;
    // every wave is past its reads of K(t) (also the prologue's) before K(t+2) replaces it
    wait_vmem();
    __syncthreads();
    if (t + 2 < ntiles) load_k(t + 2, buf);
    if (has_next) load_v(t + 1, buf ^ 1);
    tile_max(s_cur, t * kBN);
    if constexpr (has_next) {
      qk(buf ^ 1, s_next);
      exp_pv(s_cur, buf);
      // request: LDS reads issued a few MFMAs ahead of their use; every MFMA followed by a
      // slice of the exponential/row-sum/packing VALU work
      __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
      static_for<0, 2 * C::KC>([&](auto I) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, (I + 3 < 2 * C::KC) ? 1 : 2, 0);
      });
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
      static_for<0, 4 * C::NT>([&](auto) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      });
    } else {
      exp_pv(s_cur, buf);
    }
  };
  int t = 0;
  for (; t + 2 < ntiles; t += 2) {
    iteration(std::integral_constant<int, 0>{}, std::true_type{}, t, sa, sb);
    iteration(std::integral_constant<int, 1>{}, std::true_type{}, t + 1, sb, sa);
  }
  if (t + 1 < ntiles) {
    iteration(std::integral_constant<int, 0>{}, std::true_type{}, t, sa, sb);
    iteration(std::integral_constant<int, 1>{}, std::false_type{}, t + 1, sb, sa);
  } else {
    iteration(std::integral_constant<int, 0>{}, std::false_type{}, t, sa, sb);
  }

  // epilogue: normalise, store O (bf16) and LSE
  const float lp = (l_part[0] + l_part[1]) + (l_part[2] + l_part[3]);
  const float l = lp + __shfl_xor(lp, 32, 64);
  const float inv_l = 1.f / l;
  if (qrow < L && g == 0 && p.lse)
    p.lse[static_cast<long long>(h) * p.Ntot + s0 + qrow] = (m_used + __builtin_amdgcn_logf(l)) * kLn2;
  // O through each wave's own rows of the K buffers (4 waves x 32 rows fill them exactly),
  // once every wave is past its last tile reads
  static_assert(4 * 32 * (D + 8) <= 2 * kBN * C::KS, "staged O does not fit the K buffers");
  __syncthreads();
  store_o_staged<D>(oacc, inv_l, 0, &Ks[0][0] + w * 32 * (D + 8),
                    make_rsrc(p.o + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q), q0 + w * 32, qstride);
}

// ---------------------------------------------------------------- forward, rotation
// For long segments without a causal mask at head dim 80.  A workgroup = 12 waves x 32 query
// rows in three groups of four; wave w runs on SIMD w % 4, so every SIMD holds one wave of
// each group.  Each wave processes a 64-key tile t in three phases, one per time slot:
//   A1: row max (and rare rescale) of S^T(t), the first kA1Vals exponentials per lane;
//   A2: the remaining exponentials and the fp16 packing of P^T(t);
//   B : S^T(t+1) = K(t+1) Q^T and O^T += V(t)^T P^T(t), all 22 MFMAs of the tile.
// Group g runs g slots behind group 0 and a workgroup barrier ends every slot, so in each
// slot two waves per SIMD issue VALU work (a single wave cannot keep the VALU busy) while
// the third keeps the matrix pipe busy.
//
// The PV product runs in fp16 on V^T tiles that attn_vt_prep writes once per call: row 80
// of each tile is all ones, so O^T's padding row 80 accumulates the row sums of P and the
// VALU adds no sums.  P is exp2(s * scale * log2 e - m + 7) <= 2^15 (lazy rescaling keeps
// s * scale * log2 e - m <= 8), so it stays far from fp16's overflow and its small values
// keep 11 significant bits down to 2^-21 of the row max; the row sums therefore carry at
// most 2^-12 relative rounding, against 2^-9 for bf16 P.
// K rows enter the MFMA in a permuted order (bits 2 and 3 of the row index swapped), which
// puts each lane's keys in the order the B operand of the PV product takes them, so V^T
// tiles are in plain key order.  Group 0 issues the DMA of K(t+2) and V^T(t+2) during its
// phase A2 of tile t and awaits it before the barrier that ends its phase A1 of tile t+1.
// K runs through three LDS buffers (read in phase B of the tile before), V^T through four
// (read in phase B of its own tile, up to three slots later).

// fp16 V^T tiles in the workspace, [H][kVtRows][vt_cols]: segment s owns the 64-column
// aligned range [vt_start(s), vt_start(s+1)), vt_start(s) = 64 ceil(cu[s] / 64) + 64 s, which
// is at least 64 ceil(L_s / 64) columns wide, so no 64-key tile reads another segment's
// columns.  Column vt_start(s) + j holds key j of the segment for j < L_s and zero past it.
// Rows 0..79 are V^T scaled by 2^n (n = vt_shift of the segment and KV head, exact: a power of
// two), row 80 is one for the segment's keys.
constexpr int kVtRows = 81;

__host__ __device__ inline long long vt_cols(int N, int nseg) { return 64ll * ((N + 63) / 64) + 64ll * nseg; }
__device__ __forceinline__ int vt_start(int cu_s, int s) { return 64 * ((cu_s + 63) / 64) + 64 * s; }

// fp16 keeps 11 significant bits between 2^-14 and 65504; bf16 keeps 8 over fp32's exponent
// range.  Scaling a (segment, KV head)'s V by 2^n with n = 142 - E, E the biased exponent of its
// largest |v| (1 for subnormals), puts that largest value in [2^15, 2^16), where bf16's largest
// value is 65280 < 65504; every value down to 2^-32 of the largest then converts to fp16 exactly,
// and smaller ones (at most 2^-32 of the largest) keep fewer bits.  All-zero V takes n = 0.
__device__ __forceinline__ int vt_shift(uint32_t amax_bits) {
  if (amax_bits == 0u) return 0;
  const int e = static_cast<int>((amax_bits >> 7) & 0xffu);
  return 142 - (e > 0 ? e : 1);
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f16x8 as_f16x8(uint4 u) {
  f16x8 r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}
__device__ __forceinline__ f32x16 mfma_f16(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  f32x2 v = {a, b};
  f16x2 r = __builtin_convertvector(v, f16x2);
  uint32_t u;
  __builtin_memcpy(&u, &r, 4);
  return u;
}

struct VtParams {
  const uint16_t* v;     // bf16 [N, H, 80]
  uint16_t* vt;          // fp16 [H, kVtRows, cols]
  uint32_t* amax;        // [nseg, H] largest |v| of each (segment, head), bf16 bits
  const int32_t* cu;
  int H, tiles;          // tiles: 64-column blocks per segment in the grid
  long long cols;
};

// Clears the per-(segment, head) maxima (a kernel, not a memset, so that a captured graph
// replays it like any other launch).
__global__ __launch_bounds__(256) void attn_vt_clear(uint32_t* amax, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) amax[i] = 0u;
}

// Largest |v| of every (segment, head): a workgroup reads kAmaxTok consecutive token rows of one
// segment ([tokens, H, 80] bf16, 16-byte chunks; consecutive threads read consecutive chunks),
// keeps one maximum per chunk slot of a row, folds the 10 slots of each head through LDS and
// raises the head's maximum with an atomic max on the bf16 bit pattern of |v| (monotone in |v|
// for non-NaN values).
constexpr int kAmaxTok = 128;
constexpr int kAmaxMaxHeads = 256;
__global__ __launch_bounds__(256) void attn_v_amax(const VtParams p) {
  __shared__ uint32_t sm[kAmaxMaxHeads * 10];
  const int s = blockIdx.x / p.tiles, b = blockIdx.x - s * p.tiles;   // tiles: blocks per segment
  const int c0 = p.cu[s], L = p.cu[s + 1] - c0;
  const int t0 = b * kAmaxTok;
  if (t0 >= L) return;   // the whole workgroup leaves together
  const int nt = min(kAmaxTok, L - t0);
  const int slots = p.H * 10;
  const uint4* base = reinterpret_cast<const uint4*>(p.v + static_cast<long long>(c0 + t0) * p.H * 80);
  for (int slot = threadIdx.x; slot < slots; slot += 256) {
    uint32_t m = 0u;
#pragma unroll 8
    for (int r = 0; r < nt; ++r) {
      const uint4 u = base[static_cast<long long>(r) * slots + slot];
      const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) m = max(m, max(w4[e] & 0x7fffu, (w4[e] >> 16) & 0x7fffu));
    }
    sm[slot] = m;
  }
  __syncthreads();
  for (int h = threadIdx.x; h < p.H; h += 256) {
    uint32_t m = 0u;
#pragma unroll
    for (int c = 0; c < 10; ++c) m = max(m, sm[h * 10 + c]);
    if (m != 0u) atomicMax(&p.amax[s * p.H + h], m);
  }
}

// One workgroup per (64-column block of a segment, head): V rows in, fp16 V^T rows out, each
// value scaled by 2^vt_shift of its (segment, head) (exact), which keeps every finite bf16 V
// within fp16's range.
__global__ __launch_bounds__(256) void attn_vt_prep(const VtParams p) {
  __shared__ __align__(16) uint16_t T[kVtRows][64 + 8];
  const int s = blockIdx.x / p.tiles, t = blockIdx.x - (blockIdx.x / p.tiles) * p.tiles;
  const int h = blockIdx.y;
  const int c0 = p.cu[s], L = p.cu[s + 1] - c0;
  const int col0 = vt_start(c0, s);
  const int width = vt_start(p.cu[s + 1], s + 1) - col0;
  if (64 * t >= width) return;   // the whole workgroup leaves together
  const int tid = threadIdx.x;
  const int shift = vt_shift(p.amax[s * p.H + h]);
  for (int c = tid; c < 64 * 10; c += 256) {
    const int key = c / 10, ch = c - (c / 10) * 10;
    const int j = 64 * t + key;
    uint4 u = make_uint4(0u, 0u, 0u, 0u);
    if (j < L) u = *reinterpret_cast<const uint4*>(p.v + (static_cast<long long>(c0 + j) * p.H + h) * 80 + ch * 8);
    const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t pk = pack_f16x2(__builtin_amdgcn_ldexpf(__uint_as_float(w4[e] << 16), shift),
                                     __builtin_amdgcn_ldexpf(__uint_as_float(w4[e] & 0xffff0000u), shift));
      T[ch * 8 + 2 * e][key] = static_cast<uint16_t>(pk & 0xffffu);
      T[ch * 8 + 2 * e + 1][key] = static_cast<uint16_t>(pk >> 16);
    }
  }
  if (tid < 64) T[80][tid] = (64 * t + tid < L) ? static_cast<uint16_t>(0x3C00) : static_cast<uint16_t>(0);
  __syncthreads();
  for (int c = tid; c < kVtRows * 8; c += 256) {
    const int d = c >> 3, col = 64 * t + 8 * (c & 7);
    if (col < width)
      *reinterpret_cast<uint4*>(p.vt + (static_cast<long long>(h) * kVtRows + d) * p.cols + col0 + col) =
          *reinterpret_cast<const uint4*>(&T[d][col - 64 * t]);
  }
}

// Workgroup barrier that also fences the instruction scheduler, so no computation
// migrates between the two sides of a phase boundary.
__device__ __forceinline__ void phase_sync() {
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  __builtin_amdgcn_sched_barrier(0);
}

constexpr int kRotWaves = 12;
constexpr int kRotThreads = 64 * kRotWaves;
constexpr int kRotBM = 32 * kRotWaves;                // query rows per workgroup
constexpr int kVtStride = kBN + 8;                    // LDS row stride of a V^T tile (elements)
constexpr int kVtChunks = kVtRows * (kVtStride / 8);  // 16-byte DMA chunks per V^T tile
constexpr int kVtInst = (kVtChunks + 63) / 64;        // wave-wide DMA loads per V^T tile
constexpr int kVtPW = (kVtInst + 3) / 4;              // per wave of group 0
constexpr int kA1Vals = 16;                           // exponentials per lane in phase A1 (of 32)
constexpr float kP16Shift = 7.0f;                     // log2 of P's scale factor

// Row order of K in S^T = K Q^T: bits 2 and 3 of the row index swapped (an involution).
__device__ __forceinline__ int swap_bits23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

template <int D>
__global__ __launch_bounds__(kRotThreads, 1) void attn_fwd_rot(const FwdParams p) {
  static_assert(D == 80, "the rotation kernel is laid out for head dim 80");
  using C = FwdCfg<D>;
  __shared__ __align__(16) uint16_t Ks[3][kBN * C::KS];
  __shared__ __align__(16) uint16_t Vt[4][C::DV * kVtStride];   // fp16 V^T tiles (rows 81.. unused)

  const int lb = remap_block_id(blockIdx.x, gridDim.x);
  const int per_head = p.nseg * p.nqt;
  const int h = lb / per_head;
  const int rem = lb - h * per_head;
  const int seg = rem / p.nqt;
  const int qt = rem - seg * p.nqt;
  const int s0 = p.cu[seg];
  const int L = p.cu[seg + 1] - s0;
  const int q0 = qt * kRotBM;
  if (q0 >= L) return;   // the whole workgroup leaves together
  const int kvh = h / p.group;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = w >> 2, wl = w & 3;
  const int lane = tid & 63, g = lane >> 5, c32 = lane & 31;
  const int qrow = q0 + w * 32 + c32;
  const int qstride = p.Hq * D;
  const int kvstride = p.Hkv * D;

  const unsigned seg_bytes_q = static_cast<unsigned>((L - 1) * qstride + D) * 2u;
  const unsigned seg_bytes_kv = static_cast<unsigned>((L - 1) * kvstride + D) * 2u;
  const auto rq = make_rsrc(p.q + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q);
  const auto rk = make_dma_rsrc(p.k + static_cast<long long>(s0) * kvstride + kvh * D, seg_bytes_kv);
  const auto rvt = make_dma_rsrc(p.vt + static_cast<long long>(kvh) * kVtRows * p.vt_cols,
                                 static_cast<unsigned>(kVtRows * p.vt_cols * 2));

  bf16x8 qf[C::KC];
  {
    const unsigned qoff = static_cast<unsigned>(qrow * qstride + g * 8) * 2u;
#pragma unroll
    for (int c = 0; c < C::KC; ++c) qf[c] = as_bf16x8(buf_load16(rq, qoff + c * 32, 0));
  }

  // DMA chunk offsets, issued by the 4 waves of group 0
  unsigned koff[C::KPW], vtoff[kVtPW];
  static_for<0, C::KPW>([&](auto I) __attribute__((always_inline)) {
    const int c = (wl + 4 * I) * 64 + lane;
    const int r = c / C::KROW, cc = c % C::KROW;
    koff[I] = (cc < D / 8 && wl + 4 * I < C::KINST) ? static_cast<unsigned>(r * kvstride + cc * 8) * 2u
                                                     : kOutOfRange;
  });
  const long long vcol0 = vt_start(s0, seg);
  static_for<0, kVtPW>([&](auto I) __attribute__((always_inline)) {
    const int c = (wl + 4 * I) * 64 + lane;
    const int d = c / (kVtStride / 8), cc = c % (kVtStride / 8);
    vtoff[I] = (cc < kBN / 8 && d < kVtRows && wl + 4 * I < kVtInst)
                   ? static_cast<unsigned>((d * p.vt_cols + vcol0 + cc * 8) * 2)
                   : kOutOfRange;
  });
  const unsigned tile_bytes = static_cast<unsigned>(kBN * kvstride) * 2u;
  const unsigned ks_lds = lds_u32(&Ks[0][0]), vt_lds = lds_u32(&Vt[0][0]);
  // tile t of K and V^T: the resources move to the tile (scalar work), the lane offsets stay
  auto load_kv = [&](int t, int kbuf, int vbuf) __attribute__((always_inline)) {
    const i32x4 rkt = rsrc_advance(rk, static_cast<unsigned>(t) * tile_bytes);
    const i32x4 rvtt = rsrc_advance(rvt, static_cast<unsigned>(t) * (kBN * 2));
    static_for<0, C::KPW>([&](auto I) __attribute__((always_inline)) {
      if (wl + 4 * I < C::KINST)
        dma16(rkt, ks_lds + (kbuf * kBN * C::KS + (wl + 4 * I) * 512) * 2, koff[I]);
    });
    static_for<0, kVtPW>([&](auto I) __attribute__((always_inline)) {
      if (wl + 4 * I < kVtInst)
        dma16(rvtt, vt_lds + (vbuf * C::DV * kVtStride + (wl + 4 * I) * 512) * 2, vtoff[I]);
    });
  };

  f32x16 s[2];
  const int krow = swap_bits23(c32);
  // half st of S^T(tile in K buffer kb): key rows 32 st + swap_bits23(0..31)
  auto qk_half = [&](int kb, int st) __attribute__((always_inline)) {
    const uint16_t* kp = &Ks[kb][(st * 32 + krow) * C::KS + g * 8];
    bf16x8 kf[C::KC];
#pragma unroll
    for (int c = 0; c < C::KC; ++c) kf[c] = *reinterpret_cast<const bf16x8*>(kp + c * 16);
    s[st] = mfma(kf[0], qf[0], f32x16{});
#pragma unroll
    for (int c = 1; c < C::KC; ++c) s[st] = mfma(kf[c], qf[c], s[st]);
  };

  f32x16 oacc[C::NT];
#pragma unroll
  for (int t2 = 0; t2 < C::NT; ++t2) oacc[t2] = f32x16{};
  float m_used = -INFINITY;
  float m_thresh = -INFINITY;   // m_used + kRescaleSlack
  float m_off = 0.f;            // m_used - kP16Shift (set at the first tile, whose max is finite)
  uint32_t pw[2][2][4];   // packed fp16 P^T: [half][16-key chunk][pair]

  // exponentials and fp16 packing of values [R0, R1) of the 32 per lane (pairs)
  auto exps = [&](auto R0, auto R1) __attribute__((always_inline)) {
    static_for<decltype(R0)::value / 2, decltype(R1)::value / 2>([&](auto J) __attribute__((always_inline)) {
      constexpr int r = 2 * decltype(J)::value, st = r >> 4, rr = r & 15;
      const float e0 = fast_exp2(s[st][rr] * p.scale_log2 - m_off);
      const float e1 = fast_exp2(s[st][rr + 1] * p.scale_log2 - m_off);
      pw[st][rr >> 3][(rr & 7) >> 1] = pack_f16x2(e0, e1);
      // pin the results to this phase: left alone, the compiler sinks them past the barrier
      asm volatile("" : "+v"(pw[st][rr >> 3][(rr & 7) >> 1]));
    });
  };

  // Phase A1: mask keys past the segment end (only a partial last tile has any), row max,
  // (rare) rescale, first exponentials
  auto phase_a1 = [&](int kt) __attribute__((always_inline)) {
    if (kt + kBN > L) {
      // register r of half st holds key kt + 32 st + swap_bits23(8 (r / 4) + 4 g + r % 4),
      // that is kt + 8 g + a constant
      const int lim = __builtin_amdgcn_readfirstlane(L - kt) - 8 * g;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (st * 32 + 16 * (r >> 3) + 4 * ((r >> 2) & 1) + (r & 3) >= lim) s[st][r] = -INFINITY;
    }
    // 32 values in 16 three-way maxima: 10 triples, the last pair folded into the first
    float m1[10];
#pragma unroll
    for (int i = 0; i < 10; ++i) {
      const int a = 3 * i;
      m1[i] = vmax3(s[a >> 4][a & 15], s[(a + 1) >> 4][(a + 1) & 15], s[(a + 2) >> 4][(a + 2) & 15]);
    }
    m1[0] = vmax3(m1[0], s[1][14], s[1][15]);
    const float m2a = vmax3(m1[0], m1[1], m1[2]), m2b = vmax3(m1[3], m1[4], m1[5]);
    const float m2c = vmax3(m1[6], m1[7], m1[8]);
    float mx = vmax3(vmax3(m2a, m2b, m2c), m1[9], m1[9]);
    {   // the two half-waves hold the same query rows: exchange halves without an LDS round trip
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = vmax3(__uint_as_float(sw[0]), __uint_as_float(sw[1]), __uint_as_float(sw[1])) * p.scale_log2;
    }
    if (__builtin_amdgcn_ballot_w64(mx > m_thresh) != 0ull) {
      const float m_new = fmaxf(m_used, mx);
      const float alpha = fast_exp2(m_used - m_new);
      m_used = m_new;
      m_thresh = m_new + kRescaleSlack;
      m_off = m_new - kP16Shift;
#pragma unroll
      for (int t2 = 0; t2 < C::NT; ++t2)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t2][r] *= alpha;
    }
    exps(std::integral_constant<int, 0>{}, std::integral_constant<int, kA1Vals>{});
  };

  // Phase B: S^T(next) from K buffer kb and O^T += V^T P^T from V^T buffer vb.  The K
  // fragments are read first and the V^T fragments while the S^T MFMAs run (the two halves'
  // chains interleaved), a few reads ahead of their MFMAs throughout.
  auto phase_b = [&](int kb, int vb) __attribute__((always_inline)) {
    const uint16_t* kp = &Ks[kb][krow * C::KS + g * 8];
    bf16x8 k0[C::KC], k1[C::KC];
#pragma unroll
    for (int c = 0; c < C::KC; ++c) {
      k0[c] = *reinterpret_cast<const bf16x8*>(kp + c * 16);
      k1[c] = *reinterpret_cast<const bf16x8*>(kp + 32 * C::KS + c * 16);
    }
    uint4 va[12];
    const uint16_t* vp = &Vt[vb][c32 * kVtStride + g * 8];
#pragma unroll
    for (int f = 0; f < 12; ++f) {
      const int st = f / 6, hh = (f / 3) & 1, t2 = f % 3;
      va[f] = *reinterpret_cast<const uint4*>(vp + t2 * 32 * kVtStride + st * 32 + hh * 16);
    }
    s[0] = mfma(k0[0], qf[0], f32x16{});
    s[1] = mfma(k1[0], qf[0], f32x16{});
#pragma unroll
    for (int c = 1; c < C::KC; ++c) {
      s[0] = mfma(k0[c], qf[c], s[0]);
      s[1] = mfma(k1[c], qf[c], s[1]);
    }
#pragma unroll
    for (int f = 0; f < 12; ++f) {
      const int st = f / 6, hh = (f / 3) & 1, t2 = f % 3;
      const uint4 bp = make_uint4(pw[st][hh][0], pw[st][hh][1], pw[st][hh][2], pw[st][hh][3]);
      oacc[t2] = mfma_f16(as_f16x8(va[f]), as_f16x8(bp), oacc[t2]);
    }
    // issue order: six reads, each pair of S^T MFMAs followed by two more reads, then each
    // PV MFMA followed by one more read (about six reads in flight throughout)
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
    static_for<0, 5>([&](auto) __attribute__((always_inline)) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    });
    static_for<0, 6>([&](auto) __attribute__((always_inline)) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    });
    __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
  };

  // O^T += V^T P^T alone (the last tile): A = V^T fragment, B = packed P^T
  auto pv = [&](int vb) __attribute__((always_inline)) {
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int t2 = 0; t2 < C::NT; ++t2) {
          const uint4 a = *reinterpret_cast<const uint4*>(
              &Vt[vb][(t2 * 32 + c32) * kVtStride + st * 32 + hh * 16 + g * 8]);
          const uint4 bp = make_uint4(pw[st][hh][0], pw[st][hh][1], pw[st][hh][2], pw[st][hh][3]);
          oacc[t2] = mfma_f16(as_f16x8(a), as_f16x8(bp), oacc[t2]);
        }
  };

  const int ntiles = (L + kBN - 1) / kBN;
  if (grp == 0) {
    load_kv(0, 0, 0);
    if (ntiles > 1) load_kv(1, 1, 1);
    wait_vmem();
  }
  phase_sync();
  qk_half(0, 0);
  qk_half(0, 1);
  for (int i = 0; i < grp; ++i) phase_sync();   // group g runs g slots behind
  int t = 0, kb = 0;                            // kb = t % 3
  for (; t + 1 < ntiles; ++t) {
    const int kb1 = (kb == 2) ? 0 : kb + 1, kb2 = (kb1 == 2) ? 0 : kb1 + 1;
    phase_a1(t * kBN);
    if (grp == 0) wait_vmem();   // K(t+1) and V^T(t+1), issued during phase A2 of tile t-1
    phase_sync();
    exps(std::integral_constant<int, kA1Vals>{}, std::integral_constant<int, 32>{});
    if (grp == 0 && t + 2 < ntiles) load_kv(t + 2, kb2, (t + 2) & 3);
    phase_sync();
    phase_b(kb1, t & 3);
    phase_sync();
    kb = kb1;
  }
  // last tile: nothing left to load or to multiply ahead
  phase_a1(t * kBN);
  phase_sync();
  exps(std::integral_constant<int, kA1Vals>{}, std::integral_constant<int, 32>{});
  phase_sync();
  pv(t & 3);
  phase_sync();
  for (int i = grp; i < 2; ++i) phase_sync();   // equal barrier counts in every group

  // row 80 of O^T (register 8 of block 2 in the lanes of half 0) is the row sum of P; the
  // V^T tiles carry V scaled by 2^shift, undone here (exact)
  const float l = __shfl(oacc[2][8], c32, 64);
  const float inv_l = 1.f / l;
  const int unshift = -vt_shift(p.vt_amax[seg * p.Hkv + kvh]);
  if (qrow < L && g == 0 && p.lse)
    p.lse[static_cast<long long>(h) * p.Ntot + s0 + qrow] = (m_off + __builtin_amdgcn_logf(l)) * kLn2;
  // O through each wave's own 32 rows: waves 0-5 in the V^T buffers, 6-11 in the K buffers
  // (every wave is past its last tile reads: the barriers above)
  static_assert(6 * 32 * (D + 8) <= 4 * C::DV * kVtStride && 6 * 32 * (D + 8) <= 3 * kBN * C::KS,
                "staged O does not fit the tile buffers");
  uint16_t* stage = (w < 6) ? &Vt[0][0] + w * 32 * (D + 8) : &Ks[0][0] + (w - 6) * 32 * (D + 8);
  store_o_staged<D>(oacc, inv_l, unshift, stage,
                    make_rsrc(p.o + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q), q0 + w * 32, qstride);
}

// ---------------------------------------------------------------- windows, fused mass
// Segments of at most 64 tokens (the 8x8-patch windows of the vision encoder), with the
// mass in the same pass: every key of a window fits in one tile, so each row's max and sum
// are final after one S^T tile and P = exp2(S * scale * log2 e - m) / l is exact in
// registers.  A workgroup = 2 waves x 32 query rows = one (window, head): K and V are staged
// once (DMA), each wave produces its rows' O and LSE, writes its exact P to LDS, and the
// column sums over the window's query rows give the mass of each key.  Q, K and V are read
// from HBM once, instead of twice for the forward + mass passes.
constexpr int kWinWaves = 2;
constexpr int kWinThreads = 64 * kWinWaves;
constexpr int kWinMax = 32 * kWinWaves;   // longest segment (tokens)
constexpr int kPbStride = kBN + 4;        // LDS row stride of the P tile (floats)

template <int D>
__global__ __launch_bounds__(kWinThreads) void attn_window(const FwdParams p, float* __restrict__ mass) {
  using C = FwdCfg<D>;
  constexpr int KPW = (C::KINST + kWinWaves - 1) / kWinWaves;
  constexpr int VPW = (C::VINST + kWinWaves - 1) / kWinWaves;
  // K and V tiles; after the PV product the same space holds P[query][key]
  __shared__ __align__(16) uint16_t lds[kBN * (C::KS + C::VS)];
  static_assert(kWinMax * kPbStride * 4 <= kBN * (C::KS + C::VS) * 2, "P tile does not fit");
  uint16_t* Ks = lds;
  uint16_t* Vs = lds + kBN * C::KS;
  float* Pb = reinterpret_cast<float*>(lds);

  // window-major order: the heads of a window are neighbours in the logical order, hence on
  // the same XCD at about the same time, so the cache lines holding a token's rows of all
  // heads (160 bytes per head) are fetched from HBM once and served from L2 for the others
  const int lb = remap_block_id(blockIdx.x, gridDim.x);
  const int seg = lb / p.Hq;
  const int h = lb - seg * p.Hq;
  const int s0 = p.cu[seg];
  const int L = p.cu[seg + 1] - s0;
  if (L <= 0) return;   // the whole workgroup leaves together
  const int kvh = h / p.group;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 5, c32 = lane & 31;
  const int qrow = w * 32 + c32;
  const int qstride = p.Hq * D;
  const int kvstride = p.Hkv * D;

  const unsigned seg_bytes_q = static_cast<unsigned>((L - 1) * qstride + D) * 2u;
  const unsigned seg_bytes_kv = static_cast<unsigned>((L - 1) * kvstride + D) * 2u;
  const auto rq = make_rsrc(p.q + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q);
  const auto rk = make_dma_rsrc(p.k + static_cast<long long>(s0) * kvstride + kvh * D, seg_bytes_kv);
  const auto rv = make_dma_rsrc(p.v + static_cast<long long>(s0) * kvstride + kvh * D, seg_bytes_kv);

  // K and V of the window into LDS (same chunk order as attn_fwd; wave w issues w, w+2, ...)
  const unsigned ks_lds = lds_u32(&Ks[0]), vs_lds = lds_u32(&Vs[0]);
  static_for<0, KPW>([&](auto I) __attribute__((always_inline)) {
    const int inst = w + kWinWaves * I;
    const int c = inst * 64 + lane;
    const int r = c / C::KROW, cc = c % C::KROW;
    if (inst < C::KINST)
      dma16(rk, ks_lds + inst * 1024, cc < D / 8 ? static_cast<unsigned>(r * kvstride + cc * 8) * 2u : kOutOfRange);
  });
  static_for<0, VPW>([&](auto I) __attribute__((always_inline)) {
    const int inst = w + kWinWaves * I;
    const int c = inst * 64 + lane;
    const int r = c / C::VROW, cc = c % C::VROW;
    if (inst < C::VINST)
      dma16(rv, vs_lds + inst * 1024, cc < D / 8 ? static_cast<unsigned>(r * kvstride + cc * 8) * 2u : kOutOfRange);
  });
  bf16x8 qf[C::KC];
  {
    const unsigned qoff = static_cast<unsigned>(qrow * qstride + g * 8) * 2u;
#pragma unroll
    for (int c = 0; c < C::KC; ++c) qf[c] = as_bf16x8(buf_load16(rq, qoff + c * 32, 0));
  }
  wait_vmem();
  __syncthreads();

  f32x16 s[2];
#pragma unroll
  for (int st = 0; st < 2; ++st) {
    const uint16_t* kp = &Ks[(st * 32 + c32) * C::KS + g * 8];
    bf16x8 kf[C::KC];
#pragma unroll
    for (int c = 0; c < C::KC; ++c) kf[c] = *reinterpret_cast<const bf16x8*>(kp + c * 16);
    s[st] = mfma(kf[0], qf[0], f32x16{});
#pragma unroll
    for (int c = 1; c < C::KC; ++c) s[st] = mfma(kf[c], qf[c], s[st]);
  }
  // keys past the window end, then the exact row max and sum
  float mx = -INFINITY;
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = st * 32 + g * 4 + 8 * (r >> 2) + (r & 3);
      if (key >= L) s[st][r] = -INFINITY;
      mx = fmaxf(mx, s[st][r]);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.scale_log2;
  float pv[2][16];
  float lp = 0.f;
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pv[st][r] = fast_exp2(s[st][r] * p.scale_log2 - mx);
      lp += pv[st][r];
    }
  const float l = lp + __shfl_xor(lp, 32, 64);
  const float inv_l = 1.f / l;

  // O^T = V^T P^T with the unnormalised P (as attn_fwd), then O = O^T / l
  f32x16 oacc[C::NT];
#pragma unroll
  for (int t2 = 0; t2 < C::NT; ++t2) oacc[t2] = f32x16{};
  const int tgrp = lane >> 4, li = lane & 15;
  const int tr_base = (4 * (tgrp >> 1) + (li >> 2)) * C::VS + 16 * (tgrp & 1) + 4 * (li & 3);
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const bf16x8 pb = pack_bf16x8(&pv[st][hh * 8]);
      const uint16_t* vp = &Vs[(st * 32 + hh * 16) * C::VS + tr_base];
#pragma unroll
      for (int t2 = 0; t2 < C::NT; ++t2) {
        const uint2 lo = lds_read_tr16(vp + t2 * 32);
        const uint2 hi = lds_read_tr16(vp + 8 * C::VS + t2 * 32);
        oacc[t2] = mfma(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pb, oacc[t2]);
      }
    }

  // O = O^T / l in bf16 through LDS, once both waves are done with K and V, then stored row
  // by row: a 16-byte chunk per lane, each row's D values contiguous.  (Stored straight from
  // the accumulators, every store instruction wrote 8-byte pieces of 32 rows 2,560 bytes
  // apart, which cost the write path about as much as the rest of the kernel.)
  __syncthreads();
  {
    constexpr int OS = D + 8;       // LDS row stride of the staged O (elements, 16-byte rows)
    constexpr int CPR = D / 8;      // 16-byte chunks per row
    static_assert(kWinMax * OS * 2 <= kBN * (C::KS + C::VS) * 2, "staged O does not fit");
    uint16_t* Ob = lds;
#pragma unroll
    for (int t2 = 0; t2 < C::NT; ++t2) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int dv = t2 * 32 + g * 4 + 8 * j;
        if (dv < D) {
          uint2 pk;
          pk.x = pack_bf16x2(oacc[t2][4 * j + 0] * inv_l, oacc[t2][4 * j + 1] * inv_l);
          pk.y = pack_bf16x2(oacc[t2][4 * j + 2] * inv_l, oacc[t2][4 * j + 3] * inv_l);
          *reinterpret_cast<uint2*>(&Ob[qrow * OS + dv]) = pk;
        }
      }
    }
    __syncthreads();
    // rows past the window end fall outside the resource (same extent as Q's): dropped
    const auto ro = make_rsrc(p.o + static_cast<long long>(s0) * qstride + h * D, seg_bytes_q);
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int c = tid; c < kWinMax * CPR; c += kWinThreads) {
      const int r = c / CPR, cc = c - (c / CPR) * CPR;
      const u32x4 val = *reinterpret_cast<const u32x4*>(&Ob[r * OS + cc * 8]);
      __builtin_amdgcn_raw_buffer_store_b128(val, ro, r < L ? static_cast<unsigned>(r * qstride + cc * 8) * 2u : kOutOfRange,
                                            0, 0);
    }
  }
  if (qrow < L && g == 0 && p.lse)
    p.lse[static_cast<long long>(h) * p.Ntot + s0 + qrow] = (mx + __builtin_amdgcn_logf(l)) * kLn2;

  // exact P of this lane's row (zero for rows past the window) into LDS, 4 keys per store,
  // once every thread has read its chunks of the staged O
  __syncthreads();
  const float rowf = (qrow < L) ? inv_l : 0.f;
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float4 v4 = make_float4(pv[st][4 * j] * rowf, pv[st][4 * j + 1] * rowf, pv[st][4 * j + 2] * rowf,
                              pv[st][4 * j + 3] * rowf);
      *reinterpret_cast<float4*>(&Pb[qrow * kPbStride + st * 32 + 8 * j + 4 * g]) = v4;
    }
  __syncthreads();
  // mass of key k: its column of P summed over the window's rows (rows past the window
  // hold zeros); thread k sums rows 0-31 and thread k + 64 rows 32-63, in a fixed order
  const int key = tid & 63, half = tid >> 6;
  float m4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < 32; ++q) m4[q & 3] += Pb[(half * 32 + q) * kPbStride + key];
  const float part = (m4[0] + m4[1]) + (m4[2] + m4[3]);
  __syncthreads();
  if (half == 1) Pb[key] = part;
  __syncthreads();
  if (half == 0 && key < L) mass[static_cast<long long>(h) * p.Ntot + s0 + key] = part + Pb[key];
}

// ---------------------------------------------------------------- mass
struct MassParams {
  const uint16_t* q;
  const uint16_t* k;
  const float* lse;          // [Hq, Ntot]
  float* mass;               // [Hq, mass_stride]
  const int32_t* cu;         // [nseg + 1]
  const int32_t* key_start;  // [nseg] first key receiving mass (relative), or null = 0
  const int32_t* key_len;    // [nseg] keys receiving mass, or null = all from key_start
  const int32_t* q_start;    // [nseg] first querying row (relative), or null = 0
  const int32_t* q_len;      // [nseg] querying rows, or null = whole segment
  const int32_t* mass_off;   // [nseg] column offset of the segment's keys in mass, or null = cu[s]
  long long mass_stride;
  int Ntot, Hq, Hkv, group;
  int nseg, nkt;             // key tiles per segment in the grid
  float scale_log2;
};

constexpr int kMassKeys = 256;   // keys per workgroup (4 waves x 64)
constexpr int kMassQ = 64;       // query rows per tile (two MFMA column blocks of 32)

template <int D>
struct MassCfg {
  static constexpr int KC = D / 16;
  static constexpr int QROW = D / 8 + 1;                     // 16-byte chunks per Q row (odd)
  static constexpr int QS = QROW * 8;                        // LDS row stride (elements)
  static constexpr int QINST = (kMassQ * QROW + 63) / 64;    // wave-wide DMA loads per Q tile
  static constexpr int QBUF = QINST * 512;                   // elements per buffer (incl. overhang)
  static constexpr int QPW = (QINST + 3) / 4;
};

// The mass kernel.  Every wave keeps 64 keys (two sets of 32) of K in registers as the A
// operand and streams 64-row query tiles through LDS (DMA, two tiles ahead).  Per tile it
// computes S^T(t) = K Q(t)^T on the MFMA pipe, then on the VALU
// P = exp2(S * scale * log2 e - LSE * log2 e), the exact normalised probability, summed per
// key in fp32 (each lane owns 16 keys of one query column).
template <int D, bool CAUSAL>
__global__ __launch_bounds__(kThreads, (D == 80 && !CAUSAL) ? 3 : 2) void attn_mass(const MassParams p) {
  using C = MassCfg<D>;
  __shared__ __align__(16) uint16_t Qs[3][C::QBUF];
  __shared__ __align__(16) float Ls[3][kMassQ];   // LSE of each Q tile's rows (natural log)

  const int lb = remap_block_id(blockIdx.x, gridDim.x);
  const int per_head = p.nseg * p.nkt;
  const int h = lb / per_head;
  const int rem = lb - h * per_head;
  const int seg = rem / p.nkt;
  const int kt = rem - seg * p.nkt;
  const int s0 = p.cu[seg];
  const int L = p.cu[seg + 1] - s0;
  // keys [kst, kst + klen) of the segment receive mass
  const int kst = p.key_start ? p.key_start[seg] : 0;
  const int klen = p.key_len ? p.key_len[seg] : L - kst;
  if (kt * kMassKeys >= klen) return;
  const int k0 = kst + kt * kMassKeys;
  const int kend = kst + klen;
  const int qs = p.q_start ? p.q_start[seg] : 0;
  const int ql = p.q_len ? p.q_len[seg] : L;
  const long long moff = p.mass_off ? p.mass_off[seg] : s0;
  const int kvh = h / p.group;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 5, c32 = lane & 31;
  const int qstride = p.Hq * D;
  const int kvstride = p.Hkv * D;
  const int kw0 = k0 + w * 64;   // first key of this wave

  // K fragments (A operand of S^T = K Q^T) for the wave's two 32-key sets; keys past the
  // receiving range load as zeros (their mass is never written)
  const auto rk = make_rsrc(p.k + static_cast<long long>(s0) * kvstride + kvh * D,
                            static_cast<unsigned>((kend - 1) * kvstride + D) * 2u);
  bf16x8 kf[2][C::KC];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const unsigned off = static_cast<unsigned>((kw0 + ks * 32 + c32) * kvstride + g * 8) * 2u;
#pragma unroll
    for (int c = 0; c < C::KC; ++c) kf[ks][c] = as_bf16x8(buf_load16(rk, off + c * 32, 0));
  }

  // querying rows [qs, qs + ql) of the segment: Q rows and their LSE
  const auto rq = make_dma_rsrc(p.q + static_cast<long long>(s0 + qs) * qstride + h * D,
                                ql > 0 ? static_cast<unsigned>((ql - 1) * qstride + D) * 2u : 0u);
  const auto rl = make_dma_rsrc(p.lse + static_cast<long long>(h) * p.Ntot + s0 + qs,
                                static_cast<unsigned>(ql) * 4u);
  unsigned qoff[C::QPW];
  static_for<0, C::QPW>([&](auto I) __attribute__((always_inline)) {
    const int c = (w + 4 * I) * 64 + lane;
    const int r = c / C::QROW, cc = c % C::QROW;
    qoff[I] = (cc < D / 8 && r < kMassQ && w + 4 * I < C::QINST)
                  ? static_cast<unsigned>(r * qstride + cc * 8) * 2u : kOutOfRange;
  });
  const unsigned qtile_bytes = static_cast<unsigned>(kMassQ * qstride) * 2u;
  const unsigned qs_lds = lds_u32(&Qs[0][0]);
  // The LSE rows of a tile come with its Q rows, by DMA from the wave with the fewest Q chunks.
  constexpr int kLseWave = C::QINST % 4;
  const unsigned ls_lds = lds_u32(&Ls[0][0]);
  auto load_q = [&](int t, int buf) __attribute__((always_inline)) {
    static_for<0, C::QPW>([&](auto I) __attribute__((always_inline)) {
      if (w + 4 * I < C::QINST) dma16(rq, qs_lds + (buf * C::QBUF + (w + 4 * I) * 512) * 2, qoff[I] + t * qtile_bytes);
    });
    if (w == kLseWave) dma4(rl, ls_lds + buf * kMassQ * 4, static_cast<unsigned>(t * kMassQ + lane) * 4u);
  };
  // DMA instructions this wave issues per tile
  int dma_per_tile = (w == kLseWave) ? 1 : 0;
  static_for<0, C::QPW>([&](auto I) __attribute__((always_inline)) { dma_per_tile += (w + 4 * I < C::QINST) ? 1 : 0; });
  // LSE of this lane's query row of the tile in buffer buf (log2 units); rows past the range
  // get +inf -> P = 0
  auto load_lse2 = [&](int t, int buf, int u) __attribute__((always_inline)) {
    const int r = t * kMassQ + u * 32 + c32;
    const float v = Ls[buf][u * 32 + c32];
    return (r < ql) ? v * kLog2e : INFINITY;
  };
  // S^T of the 32-row half u of the query tile in buffer buf
  auto s_tile = [&](int buf, int u, f32x16* s) __attribute__((always_inline)) {
    const uint16_t* qp = &Qs[buf][(u * 32 + c32) * C::QS + g * 8];
    bf16x8 qb[C::KC];
#pragma unroll
    for (int c = 0; c < C::KC; ++c) qb[c] = *reinterpret_cast<const bf16x8*>(qp + c * 16);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      s[ks] = mfma(kf[ks][0], qb[0], f32x16{});
#pragma unroll
      for (int c = 1; c < C::KC; ++c) s[ks] = mfma(kf[ks][c], qb[c], s[ks]);
    }
  };

  float macc[2][16];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int r = 0; r < 16; ++r) macc[ks][r] = 0.f;

  auto accumulate = [&](f32x16* s, float l2, int t, int u) __attribute__((always_inline)) {
    const int qrow = qs + t * kMassQ + u * 32 + c32;
    // causal masking only where some key of the wave lies after some row of the half tile
    const bool need_mask = CAUSAL && (kw0 + 63 > qs + t * kMassQ + u * 32);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float pr = fast_exp2(s[ks][r] * p.scale_log2 - l2);
        if (need_mask) {
          const int key = kw0 + ks * 32 + g * 4 + 8 * (r >> 2) + (r & 3);
          if (key > qrow) pr = 0.f;
        }
        macc[ks][r] += pr;
      }
  };

  // Three query-tile buffers: Q(t+2) and its LSE rows are loaded while Q(t) is read, into the
  // buffer of Q(t-1) that every wave left behind at this iteration's barrier.
  const int ntiles = (ql + kMassQ - 1) / kMassQ;
  if constexpr (D == 80 && !CAUSAL) {
    // Pipelined within the wave, one 32-key x 32-row block of S^T at a time: the tile's blocks
    // (half u, key set ks) go in the order (0,0) (0,1) (1,0) (1,1), and the MFMAs of each block
    // are issued among the VALU work (exponentials and sums) of the block before it; the last
    // block's VALU work moves to the next iteration, under the first block's MFMAs (it reads
    // no LDS, so it may cross the barrier).  Two blocks of S^T are live at a time.  Every
    // key's sum takes its terms in the same order as in the unpipelined loop below.
    auto chain = [&](int ks, const bf16x8* qb) __attribute__((always_inline)) {
      f32x16 r = mfma(kf[ks][0], qb[0], f32x16{});
#pragma unroll
      for (int c = 1; c < C::KC; ++c) r = mfma(kf[ks][c], qb[c], r);
      return r;
    };
    auto sums = [&](const f32x16& sv, float l2, int ks) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) macc[ks][r] += fast_exp2(sv[r] * p.scale_log2 - l2);
    };
    auto q_frags = [&](int buf, int u, bf16x8* qb) __attribute__((always_inline)) {
      const uint16_t* qp = &Qs[buf][(u * 32 + c32) * C::QS + g * 8];
#pragma unroll
      for (int c = 0; c < C::KC; ++c) qb[c] = *reinterpret_cast<const bf16x8*>(qp + c * 16);
    };
    // one MFMA among every six VALU instructions of the block before (the MFMAs go early)
    auto interleave = [&]() __attribute__((always_inline)) {
      static_for<0, C::KC>([&](auto) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      });
    };
    if (ntiles > 0) {
      load_q(0, 0);
      if (ntiles > 1) load_q(1, 1);
      f32x16 s3 = f32x16{};    // block (1,1) of the previous tile
      float l2p = INFINITY;    // its rows' LSE: +inf makes the first iteration's sums add zeros
      // tile t in buffer buf = t % 3; only the LAST tile can hold rows past the querying range
      // (ntiles = ceil(ql / 64)), so only it masks them
      auto tile = [&](int buf, auto LAST, int t) __attribute__((always_inline)) {
        constexpr bool last = decltype(LAST)::value;
        wait_vmem_upto(last ? 0 : dma_per_tile);
        __syncthreads();
        float l2a, l2b;
        if constexpr (last) {
          l2a = load_lse2(t, buf, 0);
          l2b = load_lse2(t, buf, 1);
        } else {
          l2a = Ls[buf][c32] * kLog2e;
          l2b = Ls[buf][32 + c32] * kLog2e;
        }
        const int buf2 = (buf == 0) ? 2 : buf - 1;   // (t + 2) % 3
        if (t + 2 < ntiles) load_q(t + 2, buf2);
        bf16x8 qa[C::KC], qc[C::KC];
        q_frags(buf, 0, qa);
        __builtin_amdgcn_sched_barrier(0);
        const f32x16 s0 = chain(0, qa);
        sums(s3, l2p, 1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        q_frags(buf, 1, qc);
        const f32x16 s1 = chain(1, qa);
        sums(s0, l2a, 0);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        const f32x16 s2 = chain(0, qc);
        sums(s1, l2a, 1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        s3 = chain(1, qc);
        sums(s2, l2b, 0);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        l2p = l2b;
      };
      int buf = 0;
      for (int t = 0; t + 1 < ntiles; ++t) {
        tile(buf, std::false_type{}, t);
        buf = (buf == 2) ? 0 : buf + 1;
      }
      tile(buf, std::true_type{}, ntiles - 1);
      sums(s3, l2p, 1);
    }
  } else if (ntiles > 0) {
    load_q(0, 0);
    if (ntiles > 1) load_q(1, 1);
    int buf = 0;
    for (int t = 0; t < ntiles; ++t) {
      // tile t's DMA (issued two iterations ago) has landed once at most tile t+1's
      // instructions are outstanding
      wait_vmem_upto(t + 1 < ntiles ? dma_per_tile : 0);
      __syncthreads();
      const float l2a = load_lse2(t, buf, 0), l2b = load_lse2(t, buf, 1);
      const int buf2 = (buf == 0) ? 2 : buf - 1;   // (t + 2) % 3
      if (t + 2 < ntiles) load_q(t + 2, buf2);
      f32x16 sa[2], sb[2];
      s_tile(buf, 0, sa);
      s_tile(buf, 1, sb);
      accumulate(sa, l2a, t, 0);
      accumulate(sb, l2b, t, 1);
      buf = (buf == 2) ? 0 : buf + 1;
    }
  }
  // column sums over the 32 query lanes of each half-wave
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float x = macc[ks][r];
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
      macc[ks][r] = x;
    }
  float* mrow = p.mass + static_cast<long long>(h) * p.mass_stride + moff;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if (c32 == r) {
        const int key = kw0 + ks * 32 + g * 4 + 8 * (r >> 2) + (r & 3);
        if (key < kend) mrow[key - kst] = macc[ks][r];
      }
    }
}

// Segments at least this long (without a causal mask, head dim 80) take the rotation
// forward kernel; at head dim 128 its per-wave state would not fit in registers.
constexpr int kRotMinSeg = 1024;

template <int D>
pace_status_t launch_attention(FwdParams fp, bool causal, int max_seglen, const MassParams* mp,
                               int nmass, hipStream_t stream) {
  if (!causal && mp != nullptr && nmass > 0 && max_seglen <= kWinMax && mp->mass_stride == fp.Ntot &&
      mp->key_start == nullptr && mp->key_len == nullptr && mp->q_start == nullptr && mp->q_len == nullptr &&
      mp->mass_off == nullptr) {
    hipLaunchKernelGGL((attn_window<D>), dim3(fp.nseg * fp.Hq), dim3(kWinThreads), 0, stream, fp, mp->mass);
    return check_launch("attn_window");
  }
  if (causal) {
    fp.nqt = (max_seglen + kBM - 1) / kBM;
    hipLaunchKernelGGL((attn_fwd<D, true>), dim3(fp.nqt * fp.nseg * fp.Hq), dim3(kThreads), 0, stream, fp);
  } else if (D == 80 && max_seglen >= kRotMinSeg) {
    VtParams vp{};
    vp.v = fp.v; vp.vt = const_cast<uint16_t*>(fp.vt); vp.amax = const_cast<uint32_t*>(fp.vt_amax);
    vp.cu = fp.cu; vp.H = fp.Hkv; vp.cols = fp.vt_cols;
    vp.tiles = (max_seglen + 128 + kBN - 1) / kBN;   // a segment owns at most L + 127 columns
    const int namax = fp.nseg * fp.Hkv;
    hipLaunchKernelGGL(attn_vt_clear, dim3((namax + 255) / 256), dim3(256), 0, stream, vp.amax, namax);
    VtParams ap = vp;
    ap.tiles = (max_seglen + kAmaxTok - 1) / kAmaxTok;
    hipLaunchKernelGGL(attn_v_amax, dim3(ap.tiles * fp.nseg), dim3(256), 0, stream, ap);
    hipLaunchKernelGGL(attn_vt_prep, dim3(vp.tiles * fp.nseg, fp.Hkv), dim3(256), 0, stream, vp);
    pace_status_t st = check_launch("attn_vt_prep");
    if (st != PACE_OK) return st;
    fp.nqt = (max_seglen + kRotBM - 1) / kRotBM;
    hipLaunchKernelGGL((attn_fwd_rot<80>), dim3(fp.nqt * fp.nseg * fp.Hq), dim3(kRotThreads), 0, stream, fp);
  } else {
    fp.nqt = (max_seglen + kBM - 1) / kBM;
    hipLaunchKernelGGL((attn_fwd<D, false>), dim3(fp.nqt * fp.nseg * fp.Hq), dim3(kThreads), 0, stream, fp);
  }
  pace_status_t st = check_launch("attn_fwd");
  if (st != PACE_OK || mp == nullptr || nmass == 0) return st;
  if (causal)
    hipLaunchKernelGGL((attn_mass<D, true>), dim3(nmass), dim3(kThreads), 0, stream, *mp);
  else
    hipLaunchKernelGGL((attn_mass<D, false>), dim3(nmass), dim3(kThreads), 0, stream, *mp);
  return check_launch("attn_mass");
}

}  // namespace
}  // namespace pace

using namespace pace;

extern "C" {

size_t pace_vit_attention_workspace_size(int N, int H, int d, int nseg, int max_seglen) {
  if (N < 0 || H < 0 || nseg < 0) return 0;
  size_t bytes = align_up(static_cast<size_t>(N) * H * sizeof(float), 256);
  if (d == 80 && max_seglen >= kRotMinSeg) {
    bytes += align_up(static_cast<size_t>(H) * kVtRows * static_cast<size_t>(vt_cols(N, nseg)) * 2, 256);
    bytes += static_cast<size_t>(nseg) * H * sizeof(uint32_t);
  }
  return bytes;
}

size_t pace_prefill_attention_workspace_size(int Ntot, int Hq) {
  if (Ntot < 0 || Hq < 0) return 0;
  return static_cast<size_t>(Ntot) * Hq * sizeof(float);
}

pace_status_t pace_vit_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v, int N,
                                 int H, int d, const int32_t* cu_seqlens, int nseg, int max_seglen,
                                 float scale, uint16_t* o, float* lse, float* mass,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(q && k && v && o && cu_seqlens, "pace_vit_attention: null device pointer");
  PACE_REQUIRE(aligned16(q) && aligned16(k) && aligned16(v) && aligned16(o),
               "pace_vit_attention: q/k/v/o must be 16-byte aligned");
  PACE_REQUIRE(N >= 1 && H >= 1 && nseg >= 1 && max_seglen >= 1 && max_seglen <= N,
               "pace_vit_attention: N=%d H=%d nseg=%d max_seglen=%d", N, H, nseg, max_seglen);
  PACE_REQUIRE(isfinite(scale) && scale > 0.f, "pace_vit_attention: scale must be positive");
  if (d != 80 && d != 128)
    return set_error(PACE_ERR_UNSUPPORTED, "pace_vit_attention: head dim %d not in {80, 128}", d);
  const long long nqt = (max_seglen + kBM - 1) / kBM;
  const long long nkt = (max_seglen + kMassKeys - 1) / kMassKeys;
  PACE_REQUIRE(nqt * nseg * H < (1ll << 31) && 2ll * max_seglen * H * d < (1ll << 31),
               "pace_vit_attention: a segment must span less than 2 GiB of q/k/v");
  pace_status_t chk = check_offsets(cu_seqlens, nseg, N, max_seglen, "pace_vit_attention: cu_seqlens", stream);
  if (chk != PACE_OK) return chk;
  float* lse_buf = lse;
  const bool rot = d == 80 && max_seglen >= kRotMinSeg;
  const long long cols = vt_cols(N, nseg);
  PACE_REQUIRE(!rot || static_cast<long long>(kVtRows) * cols * 2 < (1ll << 31),
               "pace_vit_attention: N + 64 nseg too large for the V^T tiles");
  if (rot && H > kAmaxMaxHeads)
    return set_error(PACE_ERR_UNSUPPORTED, "pace_vit_attention: %d heads at head dim 80 on segments of >= %d "
                     "tokens (at most %d)", H, kRotMinSeg, kAmaxMaxHeads);
  if ((mass != nullptr && lse == nullptr) || rot) {
    const size_t need = pace_vit_attention_workspace_size(N, H, d, nseg, max_seglen);
    if (workspace == nullptr || workspace_bytes < need)
      return set_error(PACE_ERR_WORKSPACE, "pace_vit_attention: workspace %zu < %zu bytes",
                       workspace_bytes, need);
    PACE_REQUIRE(aligned16(workspace), "pace_vit_attention: workspace must be 16-byte aligned");
    if (lse == nullptr && mass != nullptr) lse_buf = static_cast<float*>(workspace);
  }
  FwdParams fp{};
  fp.q = q; fp.k = k; fp.v = v; fp.o = o; fp.lse = lse_buf; fp.cu = cu_seqlens;
  if (rot) {
    const size_t vt_off = align_up(static_cast<size_t>(N) * H * sizeof(float), 256);
    const size_t amax_off = vt_off + align_up(static_cast<size_t>(H) * kVtRows * static_cast<size_t>(cols) * 2, 256);
    fp.vt = reinterpret_cast<const uint16_t*>(static_cast<char*>(workspace) + vt_off);
    fp.vt_amax = reinterpret_cast<const uint32_t*>(static_cast<char*>(workspace) + amax_off);
    fp.vt_cols = cols;
  }
  fp.Ntot = N; fp.Hq = H; fp.Hkv = H; fp.group = 1;
  fp.nseg = nseg; fp.nqt = static_cast<int>(nqt);
  fp.scale_log2 = scale * kLog2e;
  MassParams mp{};
  mp.q = q; mp.k = k; mp.lse = lse_buf; mp.mass = mass; mp.cu = cu_seqlens;
  mp.mass_stride = N;
  mp.Ntot = N; mp.Hq = H; mp.Hkv = H; mp.group = 1;
  mp.nseg = nseg; mp.nkt = static_cast<int>(nkt);
  mp.scale_log2 = fp.scale_log2;
  const int nmass = mass ? static_cast<int>(nkt * nseg * H) : 0;
  if (d == 80) return launch_attention<80>(fp, false, max_seglen, mass ? &mp : nullptr, nmass, stream);
  return launch_attention<128>(fp, false, max_seglen, mass ? &mp : nullptr, nmass, stream);
}

pace_status_t pace_vit_attention_mass(const uint16_t* q, const uint16_t* k, int N, int H, int d,
                                      const int32_t* cu_seqlens, int nseg, int max_seglen,
                                      float scale, const float* lse, float* mass,
                                      hipStream_t stream) {
  PACE_REQUIRE(q && k && cu_seqlens && lse && mass, "pace_vit_attention_mass: null device pointer");
  PACE_REQUIRE(aligned16(q) && aligned16(k), "pace_vit_attention_mass: q/k must be 16-byte aligned");
  PACE_REQUIRE(N >= 1 && H >= 1 && nseg >= 1 && max_seglen >= 1 && max_seglen <= N,
               "pace_vit_attention_mass: N=%d H=%d nseg=%d max_seglen=%d", N, H, nseg, max_seglen);
  PACE_REQUIRE(isfinite(scale) && scale > 0.f, "pace_vit_attention_mass: scale must be positive");
  if (d != 80 && d != 128)
    return set_error(PACE_ERR_UNSUPPORTED, "pace_vit_attention_mass: head dim %d not in {80, 128}", d);
  const long long nkt = (max_seglen + kMassKeys - 1) / kMassKeys;
  PACE_REQUIRE(nkt * nseg * H < (1ll << 31) && 2ll * max_seglen * H * d < (1ll << 31),
               "pace_vit_attention_mass: a segment must span less than 2 GiB of q/k");
  pace_status_t chk = check_offsets(cu_seqlens, nseg, N, max_seglen, "pace_vit_attention_mass: cu_seqlens",
                                    stream);
  if (chk != PACE_OK) return chk;
  MassParams mp{};
  mp.q = q; mp.k = k; mp.lse = lse; mp.mass = mass; mp.cu = cu_seqlens;
  mp.mass_stride = N;
  mp.Ntot = N; mp.Hq = H; mp.Hkv = H; mp.group = 1;
  mp.nseg = nseg; mp.nkt = static_cast<int>(nkt);
  mp.scale_log2 = scale * kLog2e;
  const int nmass = static_cast<int>(nkt * nseg * H);
  if (d == 80)
    hipLaunchKernelGGL((attn_mass<80, false>), dim3(nmass), dim3(kThreads), 0, stream, mp);
  else
    hipLaunchKernelGGL((attn_mass<128, false>), dim3(nmass), dim3(kThreads), 0, stream, mp);
  return check_launch("attn_mass");
}

pace_status_t pace_prefill_attention_with_mass(
    const uint16_t* q, const uint16_t* k, const uint16_t* v, int Ntot, int Hq, int Hkv, int d,
    const int32_t* cu_seqlens, int B, int max_seqlen, const int32_t* vis_start, const int32_t* vis_len,
    const int32_t* cu_vis, int nvis_total, int max_vis_len, const int32_t* mq_start,
    const int32_t* mq_len, int max_mq_len, float scale, uint16_t* o, float* lse, float* mass,
    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  PACE_REQUIRE(q && k && v && o && cu_seqlens, "pace_prefill_attention_with_mass: null device pointer");
  PACE_REQUIRE(aligned16(q) && aligned16(k) && aligned16(v) && aligned16(o),
               "pace_prefill_attention_with_mass: q/k/v/o must be 16-byte aligned");
  PACE_REQUIRE(Ntot >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0,
               "pace_prefill_attention_with_mass: Ntot=%d Hq=%d Hkv=%d (Hq %% Hkv must be 0)", Ntot,
               Hq, Hkv);
  PACE_REQUIRE(B >= 1 && max_seqlen >= 1 && max_seqlen <= Ntot,
               "pace_prefill_attention_with_mass: B=%d max_seqlen=%d", B, max_seqlen);
  PACE_REQUIRE(isfinite(scale) && scale > 0.f, "pace_prefill_attention_with_mass: scale must be positive");
  if (d != 80 && d != 128)
    return set_error(PACE_ERR_UNSUPPORTED, "pace_prefill_attention_with_mass: head dim %d not in {80, 128}", d);
  const bool want_mass = mass != nullptr;
  if (want_mass) {
    PACE_REQUIRE(vis_len && cu_vis && mq_start && mq_len,
                 "pace_prefill_attention_with_mass: mass needs vis_len, cu_vis, mq_start, mq_len");
    PACE_REQUIRE(nvis_total >= 0 && max_vis_len >= 0 && max_vis_len <= max_seqlen && max_mq_len >= 0 &&
                     max_mq_len <= max_seqlen,
                 "pace_prefill_attention_with_mass: nvis_total=%d max_vis_len=%d max_mq_len=%d",
                 nvis_total, max_vis_len, max_mq_len);
  }
  const long long nqt = (max_seqlen + kBM - 1) / kBM;
  const long long nkt = (max_vis_len + kMassKeys - 1) / kMassKeys;
  PACE_REQUIRE(nqt * B * Hq < (1ll << 31) && 2ll * max_seqlen * Hq * d < (1ll << 31),
               "pace_prefill_attention_with_mass: a sequence must span less than 2 GiB of q");
  if (debug_checks()) {
    pace_status_t chk = check_offsets(cu_seqlens, B, Ntot, max_seqlen,
                                      "pace_prefill_attention_with_mass: cu_seqlens", stream);
    if (chk != PACE_OK) return chk;
    if (want_mass) {
      std::vector<int32_t> cu(B + 1), vs(B, 0), vl(B), cv(B + 1), ms(B), ml(B);
      if ((vis_start && (chk = copy_to_host(vs.data(), vis_start, B, stream)) != PACE_OK) ||
          (chk = copy_to_host(cu.data(), cu_seqlens, B + 1, stream)) != PACE_OK ||
          (chk = copy_to_host(vl.data(), vis_len, B, stream)) != PACE_OK ||
          (chk = copy_to_host(cv.data(), cu_vis, B + 1, stream)) != PACE_OK ||
          (chk = copy_to_host(ms.data(), mq_start, B, stream)) != PACE_OK ||
          (chk = copy_to_host(ml.data(), mq_len, B, stream)) != PACE_OK)
        return chk;
      PACE_REQUIRE(cv[0] == 0 && cv[B] <= nvis_total, "pace_prefill_attention_with_mass: cu_vis range");
      for (int b = 0; b < B; ++b) {
        const int L = cu[b + 1] - cu[b];
        PACE_REQUIRE(vs[b] >= 0 && vl[b] >= 0 && vs[b] + vl[b] <= L && vl[b] <= max_vis_len &&
                         cv[b + 1] - cv[b] == vl[b],
                     "pace_prefill_attention_with_mass: sequence %d: visual tokens [%d, %d + %d), cu_vis step %d, "
                     "length %d", b, vs[b], vs[b], vl[b], cv[b + 1] - cv[b], L);
        PACE_REQUIRE(ms[b] >= 0 && ml[b] >= 0 && ml[b] <= max_mq_len && ms[b] + ml[b] <= L,
                     "pace_prefill_attention_with_mass: sequence %d: query rows [%d, %d + %d) outside [0, %d]",
                     b, ms[b], ms[b], ml[b], L);
      }
    }
  }
  float* lse_buf = lse;
  if (lse == nullptr) {
    const size_t need = pace_prefill_attention_workspace_size(Ntot, Hq);
    if (workspace == nullptr || workspace_bytes < need)
      return set_error(PACE_ERR_WORKSPACE, "pace_prefill_attention_with_mass: workspace %zu < %zu bytes",
                       workspace_bytes, need);
    lse_buf = static_cast<float*>(workspace);
  }
  FwdParams fp{};
  fp.q = q; fp.k = k; fp.v = v; fp.o = o; fp.lse = lse_buf; fp.cu = cu_seqlens;
  fp.Ntot = Ntot; fp.Hq = Hq; fp.Hkv = Hkv; fp.group = Hq / Hkv;
  fp.nseg = B; fp.nqt = static_cast<int>(nqt);
  fp.scale_log2 = scale * kLog2e;
  MassParams mp{};
  mp.q = q; mp.k = k; mp.lse = lse_buf; mp.mass = mass; mp.cu = cu_seqlens;
  mp.key_start = vis_start; mp.key_len = vis_len; mp.q_start = mq_start; mp.q_len = mq_len; mp.mass_off = cu_vis;
  mp.mass_stride = nvis_total;
  mp.Ntot = Ntot; mp.Hq = Hq; mp.Hkv = Hkv; mp.group = Hq / Hkv;
  mp.nseg = B; mp.nkt = static_cast<int>(nkt);
  mp.scale_log2 = fp.scale_log2;
  // the mass kernel also runs when no row queries (it then writes zeros)
  const int nmass = (want_mass && nkt > 0) ? static_cast<int>(nkt * B * Hq) : 0;
  if (d == 80) return launch_attention<80>(fp, true, max_seqlen, want_mass ? &mp : nullptr, nmass, stream);
  return launch_attention<128>(fp, true, max_seqlen, want_mass ? &mp : nullptr, nmass, stream);
}

}  // extern "C"
