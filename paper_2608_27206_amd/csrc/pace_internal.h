// Internal helpers shared by the libpace translation units: error reporting,
// argument checks, XCD-aware block numbering and block-wide primitives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "../../include/pace.h"

namespace pace {

// ---------------------------------------------------------------- errors
pace_status_t set_error(pace_status_t st, const char* fmt, ...);
pace_status_t check_launch(const char* what);

// Validation of device-side metadata, done only when the environment variable PACE_DEBUG
// is "1" (it copies the arrays to the host and synchronises the stream).  Each returns
// PACE_OK when checks are off or pass, PACE_ERR_INVALID_ARG with a message otherwise.
bool debug_checks();
// Segment offsets cu [n + 1]: cu[0] = 0, nondecreasing, cu[n] <= total, every segment at
// most max_len long.
pace_status_t check_offsets(const int32_t* cu, int n, long long total, int max_len, const char* what,
                            hipStream_t stream);
// Per-segment values v [n] within [lo, hi_b] where hi_b = upper[b] (or hi when upper is null)
// and at most vmax.
pace_status_t check_values(const int32_t* v, int n, const int32_t* upper_host, int lo, int vmax,
                           const char* what, hipStream_t stream);
// Copies n ints from the device (synchronous on the stream).
pace_status_t copy_to_host(int32_t* dst, const int32_t* src, int n, hipStream_t stream);

#define PACE_REQUIRE(cond, ...)                                   \
  do {                                                            \
    if (!(cond)) return ::pace::set_error(PACE_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Carves aligned sub-buffers out of a caller workspace.
struct Carver {
  char* base;
  size_t cap;
  size_t off = 0;
  Carver(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  template <typename T>
  T* take(size_t count) {
    off = align_up(off, 256);
    T* p = reinterpret_cast<T*>(base + off);
    off += count * sizeof(T);
    return p;
  }
  bool ok() const { return off <= cap; }
};

// Size-only twin of Carver, used by the *_workspace_size functions.
struct Sizer {
  size_t off = 0;
  template <typename T>
  void take(size_t count) {
    off = align_up(off, 256);
    off += count * sizeof(T);
  }
};

// ---------------------------------------------------------------- device helpers
// MI355X places consecutive workgroups of a launch on its 8 XCDs round-robin.
// remap_block_id turns the hardware order into a "logical" order in which every
// XCD receives one contiguous range of logical ids, so neighbouring tiles (same
// head, same K/V stream) share that XCD's L2.
constexpr int kNumXcd = 8;

__device__ __forceinline__ int remap_block_id(int bid, int nblocks) {
  const int xcd = bid % kNumXcd;
  const int slot = bid / kNumXcd;
  const int q = nblocks / kNumXcd;
  const int r = nblocks % kNumXcd;
  return (xcd < r) ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_min(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fminf(x, __shfl_xor(x, o, 64));
  return x;
}

// ---------------------------------------------------------------- range-checked buffers
// A buffer resource over `bytes` bytes from `base`: loads past the end return 0 and stores
// past the end are dropped by the hardware range check, so ragged tails need no branches
// (a branch around every store makes the compiler wait for all memory traffic in flight at
// each one).  Offsets are in bytes and go in the VGPR operand, which the check covers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t range_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float rload_f32(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void rstore_b32(__amdgpu_buffer_rsrc_t r, unsigned off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
}
constexpr unsigned kNoStore = 0x7FFFFFF0u;   // an offset past every range: the store is dropped

// ---------------------------------------------------------------- DPP wave primitives
// Data-parallel-primitive lane moves run inside the VALU (a few cycles), where __shfl goes
// through the LDS crossbar (ds_bpermute, ~100+ cycles of latency per step).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, 0xf, 0xf, true));
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(x)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(x));
  const uint32_t lo = dpp_u32<CTRL>(static_cast<uint32_t>(b));
  const uint32_t hi = dpp_u32<CTRL>(static_cast<uint32_t>(b >> 32));
  return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}
__device__ __forceinline__ double readlane_f64(double x, int lane) {
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(x));
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(b), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(b >> 32), lane);
  return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowShr1 = 0x111;

// Inclusive prefix sum over the 64 lanes (lane order).  Within each row of 16 lanes by
// shifted DPP adds (lanes shifted in from outside the row read 0), then the totals of
// the lower rows via readlane.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += dpp_u32<kDppRowShr1>(x);
  x += dpp_u32<kDppRowShr1 + 1>(x);
  x += dpp_u32<kDppRowShr1 + 3>(x);
  x += dpp_u32<kDppRowShr1 + 7>(x);
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 15);
  const uint32_t r1 = __builtin_amdgcn_readlane(x, 31);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Reduction over the 64 lanes to a wave-uniform value.  Butterfly within each row of 16
// (every lane of a row ends with the bit-identical row result, since each step combines
// the same two values in both lanes), then the four rows in a fixed order.
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce_dpp(T x, Op op) {
  if constexpr (sizeof(T) == 8) {
    x = op(x, dpp_f64<kDppQuadXor1>(x));
    x = op(x, dpp_f64<kDppQuadXor2>(x));
    x = op(x, dpp_f64<kDppRowHalfMirror>(x));
    x = op(x, dpp_f64<kDppRowMirror>(x));
    return op(op(readlane_f64(x, 0), readlane_f64(x, 16)), op(readlane_f64(x, 32), readlane_f64(x, 48)));
  } else {
    x = op(x, dpp_f32<kDppQuadXor1>(x));
    x = op(x, dpp_f32<kDppQuadXor2>(x));
    x = op(x, dpp_f32<kDppRowHalfMirror>(x));
    x = op(x, dpp_f32<kDppRowMirror>(x));
    const float a = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 0));
    const float b = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 16));
    const float c = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 32));
    const float d = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 48));
    return op(op(a, b), op(c, d));
  }
}

// Block-wide reductions with a fixed combination order (deterministic).
// `red` must hold at least blockDim.x / 64 floats; all threads must call.
template <int OP>  // 0 sum, 1 max, 2 min
__device__ float block_reduce(float x, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  x = (OP == 0) ? wave_sum(x) : (OP == 1) ? wave_max(x) : wave_min(x);
  __syncthreads();
  if (lane == 0) red[w] = x;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < nw; ++i) {
    const float y = red[i];
    r = (OP == 0) ? r + y : (OP == 1) ? fmaxf(r, y) : fminf(r, y);
  }
  return r;
}

// Order-preserving map of fp32 to uint32 (larger float -> larger key); -0 maps like +0.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Adds the active lanes' bins to an LDS histogram.  Keys that share leading digits often
// land in one bin for a whole wave: then a single atomic adds the wave's count.
__device__ __forceinline__ void histogram_add(uint32_t* hist, bool active, uint32_t bin) {
  const unsigned long long act = __ballot(active);
  if (act == 0ull) return;
  const int leader = __ffsll(static_cast<long long>(act)) - 1;
  const uint32_t lead_bin = __builtin_amdgcn_readlane(bin, leader);
  const unsigned long long same = __ballot(active && bin == lead_bin);
  if (same == act) {
    if ((threadIdx.x & 63) == leader) atomicAdd(&hist[lead_bin], static_cast<uint32_t>(__popcll(act)));
  } else if (active) {
    atomicAdd(&hist[bin], 1u);
  }
}

// Radix selection of the k-th largest key (1 <= k <= n) among n keys produced by
// `get(i)`, by one workgroup, most significant byte first.
// Returns the key T of the k-th largest element and writes *need = how many
// elements equal to T belong to the top k (the lowest-index ones, by convention).
// `hist` is LDS scratch of 256 uint32 plus 8 extra words.  All threads must call.
template <typename Get>
__device__ uint32_t block_radix_select(int n, int k, Get get, uint32_t* hist, int* need) {
  uint32_t prefix = 0, mask = 0;
  int remaining = k;
  uint32_t* sel = hist + 256;  // [0]: digit, [1]: remaining
  if (threadIdx.x == 0) { sel[0] = 0; sel[1] = static_cast<uint32_t>(k); }
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int i0 = 0; i0 < n; i0 += blockDim.x) {
      const int i = i0 + threadIdx.x;
      const uint32_t key = (i < n) ? get(i) : 0u;
      const bool active = (i < n) && (key & mask) == prefix;
      const uint32_t bin = (key >> shift) & 255u;
      // values with a common leading part land in one bin: one atomic per wave then
      histogram_add(hist, active, bin);
    }
    __syncthreads();
    // Suffix sums over digits (high to low) by the first wave: lane j holds digits
    // 4j..4j+3 in descending order of its slice.
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      const int dhi = 255 - 4 * lane;  // this lane handles digits dhi, dhi-1, dhi-2, dhi-3
      uint32_t c0 = hist[dhi], c1 = hist[dhi - 1], c2 = hist[dhi - 2], c3 = hist[dhi - 3];
      uint32_t tot = c0 + c1 + c2 + c3;
      // inclusive scan of tot over lanes (lane 0 = highest digits)
      uint32_t incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      uint32_t before = incl - tot;  // count of elements with digits above dhi
      const uint32_t rem = static_cast<uint32_t>(remaining);
      uint32_t cs[4] = {c0, c1, c2, c3};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (before < rem && before + cs[t] >= rem) {
          sel[0] = static_cast<uint32_t>(dhi - t);
          sel[1] = rem - before;
        }
        before += cs[t];
      }
    }
    __syncthreads();
    const uint32_t digit = sel[0];
    remaining = static_cast<int>(sel[1]);
    prefix |= digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  *need = remaining;
  return prefix;
}

// Radix selection as block_radix_select, over keys held in registers: thread t holds the
// keys of elements t * R + j (j < R) or, with STRIDED, of elements j * blockDim.x + t;
// element i is valid when i < n.  Same result (the k-th largest key T and *need, the
// number of elements equal to T in the top k); the keys are read once instead of once per
// pass.  All threads must call.
template <int R, bool STRIDED = false>
__device__ uint32_t block_radix_select_regs(const uint32_t (&key)[R], int n, int k, uint32_t* hist,
                                            int* need) {
  uint32_t prefix = 0, mask = 0;
  int remaining = k;
  uint32_t* sel = hist + 256;  // [0]: digit, [1]: remaining
  const int base = STRIDED ? static_cast<int>(threadIdx.x) : static_cast<int>(threadIdx.x) * R;
  const int step = STRIDED ? static_cast<int>(blockDim.x) : 1;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const bool active = (base + j * step < n) && (key[j] & mask) == prefix;
      const uint32_t bin = (key[j] >> shift) & 255u;
      histogram_add(hist, active, bin);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      const int dhi = 255 - 4 * lane;
      const uint32_t c0 = hist[dhi], c1 = hist[dhi - 1], c2 = hist[dhi - 2], c3 = hist[dhi - 3];
      const uint32_t tot = c0 + c1 + c2 + c3;
      uint32_t incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      uint32_t before = incl - tot;
      const uint32_t rem = static_cast<uint32_t>(remaining);
      const uint32_t cs[4] = {c0, c1, c2, c3};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (before < rem && before + cs[t] >= rem) {
          sel[0] = static_cast<uint32_t>(dhi - t);
          sel[1] = rem - before;
        }
        before += cs[t];
      }
    }
    __syncthreads();
    const uint32_t digit = sel[0];
    remaining = static_cast<int>(sel[1]);
    prefix |= digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  *need = remaining;
  return prefix;
}

// Radix selection over keys held in registers (thread t holds element t * R + j in key[j],
// or with STRIDED element j * blockDim.x + t; element i is valid when i < n), with one LDS
// histogram per pass: `hist` holds 4 * 256 words that the caller zeroed before a barrier,
// and `sel` 2 words.  Two barriers per pass.  Returns the k-th largest key T (1 <= k <= n)
// and *need, the number of elements equal to T that belong to the top k (the lowest-index
// ones).  All threads must call.
template <int R, bool STRIDED>
__device__ uint32_t radix_select_prezeroed(const uint32_t (&key)[R], int n, int k, uint32_t* hist,
                                           uint32_t* sel, int* need) {
  uint32_t prefix = 0, mask = 0;
  uint32_t remaining = static_cast<uint32_t>(k);
  const int t = threadIdx.x;
#pragma unroll 1
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t* h = hist + 256 * pass;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int i = STRIDED ? j * static_cast<int>(blockDim.x) + t : t * R + j;
      const bool active = (i < n) && (key[j] & mask) == prefix;
      histogram_add(h, active, (key[j] >> shift) & 255u);
    }
    __syncthreads();
    if (t < 64) {
      // lane l covers digits 255 - 4l down to 252 - 4l (descending digit order)
      const int dhi = 255 - 4 * t;
      const uint32_t c0 = h[dhi], c1 = h[dhi - 1], c2 = h[dhi - 2], c3 = h[dhi - 3];
      const uint32_t tot = c0 + c1 + c2 + c3;
      uint32_t before = wave_incl_scan(tot) - tot;
      const uint32_t cs[4] = {c0, c1, c2, c3};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (before < remaining && before + cs[q] >= remaining) {
          sel[0] = static_cast<uint32_t>(dhi - q);
          sel[1] = remaining - before;
        }
        before += cs[q];
      }
    }
    // sel is rewritten only after the first barrier of the next pass, which every thread
    // reaches after reading it here
    __syncthreads();
    prefix |= sel[0] << shift;
    mask |= 255u << shift;
    remaining = sel[1];
  }
  *need = static_cast<int>(remaining);
  return prefix;
}

// Exclusive prefix sum of a per-thread count across the whole block (in thread order)
// plus the block total.  `cnt` is LDS scratch of blockDim.x/64 ints.
__device__ __forceinline__ int block_exclusive_sum(int v, int* cnt, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  __syncthreads();
  if (lane == 63) cnt[w] = incl;
  __syncthreads();
  int before = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    const int c = cnt[i];
    if (i < w) before += c;
    tot += c;
  }
  *total = tot;
  return before + incl - v;
}

// Exclusive prefix count of a per-thread flag across the whole block (in thread
// order) plus the block total.  `cnt` is LDS scratch of blockDim.x/64 ints.
__device__ __forceinline__ int block_exclusive_count(bool flag, int* cnt, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const unsigned long long m = __ballot(flag);
  const unsigned long long lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int in_wave = __popcll(m & lt);
  __syncthreads();
  if (lane == 0) cnt[w] = __popcll(m);
  __syncthreads();
  int before = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    const int c = cnt[i];
    if (i < w) before += c;
    tot += c;
  }
  *total = tot;
  return before + in_wave;
}

}  // namespace pace
