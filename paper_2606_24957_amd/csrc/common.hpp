// common.hpp -- device helpers shared by the libdustin kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dustin.h"

namespace dustin {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

// The order-preserving uint32 of an fp32 value (larger value, larger key; -0 and +0 alike;
// NaNs beyond +-inf by their sign bit): the ranking key of the top-k.  Its top 12 bits are
// the first digit of the top-k's radix selection (kDigitBins bins).
constexpr int kDigitBins = 4096;
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// D = A * B + C on one 16x16x32 bf16 MFMA tile.  Lane l holds A[l % 16][8 (l / 16) + e],
// B[8 (l / 16) + e][l % 16] (e = 0..7) and D[4 (l / 16) + e][l % 16] (e = 0..3).
__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& u) {
  return __builtin_bit_cast(bf16x8, u);
}

// Upper 16 bits of two fp32 values that are exact bf16 numbers, packed lo | hi << 16.
__device__ __forceinline__ uint32_t pack_exact_bf16(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// Round-to-nearest-even fp32 -> bf16 (NaN stays NaN), as raw bits.
__device__ __forceinline__ uint32_t bf16_rne_bits(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t h) { return __uint_as_float(h << 16); }

// Pairwise reductions across 16-lane rows using the gfx950 permlane swaps (VALU, no LDS
// traffic).  For every lane the two results of a swap of x with itself hold {x of this
// lane, x of lane ^ 16} (permlane16) or {x of this lane, x of lane ^ 32} (permlane32), so
// a symmetric operation over both is the butterfly step.
__device__ __forceinline__ float max_xor16(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Butterfly over lanes l ^ 16 and l ^ 32: combines the four 16-lane groups of a wave.
__device__ __forceinline__ float max_over_lane_groups(float x) { return max_xor32(max_xor16(x)); }
__device__ __forceinline__ float sum_over_lane_groups(float x) { return sum_xor32(sum_xor16(x)); }

// 2^x on the hardware exp unit (results below 2^-126 flush to zero).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Per-sequence sizes read from the device arrays and clamped to the host-checked bounds.
struct SeqDims {
  const int32_t* seq_lens;
  const int32_t* n_query;
  const int32_t* budget;
  const int32_t* m;
  int32_t max_len, nq_max, k_max, m_scalar;

  __device__ __forceinline__ int len(int b) const { return clampi(seq_lens[b], 0, max_len); }
  __device__ __forceinline__ int nq(int b) const { return n_query ? clampi(n_query[b], 0, nq_max) : nq_max; }
};

// Address arithmetic of one K or V cache (contiguous or paged); positions are clamped
// into [0, capacity) and page ids into [0, num_pages).
struct KvView {
  const uint16_t* data;
  int64_t stride_b, stride_n, stride_h, stride_page;
  const int32_t* page_table;
  int32_t page_shift, max_pages, num_pages;
  int64_t capacity;

  template <bool kPaged>
  __device__ __forceinline__ const uint16_t* row(int b, int64_t pos, int g) const {
    pos = pos < 0 ? 0 : (pos >= capacity ? capacity - 1 : pos);
    if constexpr (kPaged) {
      const int slot = (int)(pos >> page_shift);
      const int page = clampi(page_table[(int64_t)b * max_pages + slot], 0, num_pages - 1);
      return data + (int64_t)page * stride_page + (pos & ((1 << page_shift) - 1)) * stride_n +
             (int64_t)g * stride_h;
    } else {
      return data + (int64_t)b * stride_b + pos * stride_n + (int64_t)g * stride_h;
    }
  }
};

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

}  // namespace dustin
