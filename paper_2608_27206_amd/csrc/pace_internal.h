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
