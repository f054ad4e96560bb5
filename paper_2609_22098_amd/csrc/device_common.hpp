// Device-side building blocks shared by the expansion and verification kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/treespark.h"

namespace ts {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kNegInf = -__builtin_huge_valf();

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Philox4x32-10 round keys, precomputed on the host from the 64-bit seed
// (k0 = seed lo32, k1 = seed hi32; each round adds the Weyl constants).
struct PhiloxKeys {
  uint32_t k0[10];
  uint32_t k1[10];
};

// Philox4x32-10 (Salmon et al., SC'11): ten rounds of the multiply-hi/lo
// bijection.  Each 32x32 product is one 64-bit multiply.
__device__ __forceinline__ void philox10(uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3,
                                         const PhiloxKeys& k) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k.k0[r];
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k.k1[r];
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
  }
}

__device__ __forceinline__ uint32_t counter_word3(int request, int depth, uint32_t tag) {
  return ((uint32_t)request << 12) | ((uint32_t)depth << 4) | tag;
}

// u = ((w >> 9) + 0.5) * 2^-23, exact in fp32.
__device__ __forceinline__ float word_to_uniform(uint32_t w) {
  return __builtin_fmaf((float)(w >> 9), 1.1920928955078125e-07f, 5.9604644775390625e-08f);
}

// Gumbel-perturbed key in base-2 units: z * c - log2(-log2(u)) with c = log2(e) / T.
// It equals log2(e) * (z / T - log(-log u)) + log2(log 2): a fixed increasing
// affine map of the natural-log key, so both give the same order.
__device__ __forceinline__ float gumbel_key2(float z, float c, uint32_t w) {
  const float u = word_to_uniform(w);
  const float e2 = -__builtin_amdgcn_logf(u);  // -log2(u) > 0
  return __builtin_fmaf(z, c, -__builtin_amdgcn_logf(e2));
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// log p-hat = log sigmoid(a * logit(q0) + b) from lq = log q0 (§3.4 Eq. 3),
// without branches, on the base-2 exponential and logarithm of the vector
// unit.  logit = lq - log(1 - q0): 1 - q0 is the difference 1 - e^lq except
// near lq = 0, where that difference cancels and the Taylor series of
// -expm1(lq) (to the x^7 term; below 1e-8 relative for |lq| <= 0.3) is used.
// log sigmoid(y) = min(y, 0) - log(1 + e^-|y|).  The result is within 5e-7
// of the fp64 value relative to max(1, |log p-hat|), as for the libm
// functions.  lq >= 0 (and NaN) gives logit +inf; lq = -inf gives -inf.
__device__ __forceinline__ float log_phat(float lq, float a, float b) {
  const float e = exp2_fast(lq * kLog2e);
  const float x = lq;
  const float series =
      x * __builtin_fmaf(x, __builtin_fmaf(x, __builtin_fmaf(x, __builtin_fmaf(x, __builtin_fmaf(x,
          __builtin_fmaf(x, 1.0f / 5040.0f, 1.0f / 720.0f), 1.0f / 120.0f), 1.0f / 24.0f), 1.0f / 6.0f), 0.5f), 1.0f);
  const float one_minus_q0 = lq > -0.3f ? -series : 1.0f - e;
  const float logit = lq < 0.0f ? lq - __builtin_amdgcn_logf(one_minus_q0) * kLn2 : __builtin_huge_valf();
  const float y = a == 0.0f ? b : __builtin_fmaf(a, logit, b);
  const float t = exp2_fast(-__builtin_fabsf(y) * kLog2e);
  return fminf(y, 0.0f) - __builtin_amdgcn_logf(1.0f + t) * kLn2;
}

// Cross-lane moves with DPP (data-parallel primitives): the source lane's
// value moves inside the VALU operand path, without an LDS round trip.
// CTRL: 0xB1 = quad_perm [1,0,3,2], 0x4E = quad_perm [2,3,0,1],
// 0x141 = row_half_mirror (lane i <- 7 - i within 8), 0x140 = row_mirror
// (i <- 15 - i within 16), 0x111 + (n - 1) = row_shr:n, 0x138 = wave_shr:1
// (lane i <- i - 1 across the wave), 0x142 = row_bcast:15 (lane 15 of a row
// to every lane of the next row), 0x143 = row_bcast:31 (lane 31 to rows 2
// and 3); lanes without a source read 0.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

// Value of lane l (l wave-uniform), read through a scalar register.
__device__ __forceinline__ float lane_f32(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ int lane_i32(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

// Wave-wide (64 lanes) reductions in a fixed order: pairs, quads, halves of
// a row, rows (all lanes of a row end equal), then the four rows in order.
// Every lane gets the same value.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  return ((lane_f32(v, 0) + lane_f32(v, 16)) + lane_f32(v, 32)) + lane_f32(v, 48);
}
__device__ __forceinline__ int wave_sum_i32(int v) {
  v += dpp_i32<0xB1>(v);
  v += dpp_i32<0x4E>(v);
  v += dpp_i32<0x141>(v);
  v += dpp_i32<0x140>(v);
  return ((lane_i32(v, 0) + lane_i32(v, 16)) + lane_i32(v, 32)) + lane_i32(v, 48);
}

// Eight independent wave reductions, interleaved stage by stage so their
// latencies overlap; each result equals the single reduction's.
__device__ __forceinline__ void wave_max8(float (&x)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = fmaxf(x[k], dpp_f32<0xB1>(x[k]));
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = fmaxf(x[k], dpp_f32<0x4E>(x[k]));
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = fmaxf(x[k], dpp_f32<0x141>(x[k]));
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = fmaxf(x[k], dpp_f32<0x140>(x[k]));
#pragma unroll
  for (int k = 0; k < 8; ++k)
    x[k] = fmaxf(fmaxf(lane_f32(x[k], 0), lane_f32(x[k], 16)), fmaxf(lane_f32(x[k], 32), lane_f32(x[k], 48)));
}
__device__ __forceinline__ void wave_sum8(float (&x)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] += dpp_f32<0xB1>(x[k]);
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] += dpp_f32<0x4E>(x[k]);
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] += dpp_f32<0x141>(x[k]);
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] += dpp_f32<0x140>(x[k]);
#pragma unroll
  for (int k = 0; k < 8; ++k)
    x[k] = ((lane_f32(x[k], 0) + lane_f32(x[k], 16)) + lane_f32(x[k], 32)) + lane_f32(x[k], 48);
}

// Exchanges across rows with the gfx950 permlane swaps (no LDS round trip):
// xor16 gives lane i the value of lane i ^ 16, xor32 that of lane i ^ 32.
__device__ __forceinline__ uint32_t xor16_u32(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return ((threadIdx.x >> 4) & 1) ? r[0] : r[1];
}
__device__ __forceinline__ uint32_t xor32_u32(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return ((threadIdx.x >> 5) & 1) ? r[0] : r[1];
}
__device__ __forceinline__ float xor16_f32(float v) { return __uint_as_float(xor16_u32(__float_as_uint(v))); }
__device__ __forceinline__ float xor32_f32(float v) { return __uint_as_float(xor32_u32(__float_as_uint(v))); }
__device__ __forceinline__ int xor16_i32(int v) { return (int)xor16_u32((uint32_t)v); }
__device__ __forceinline__ int xor32_i32(int v) { return (int)xor32_u32((uint32_t)v); }

// Sum over the four lanes n, n + 16, n + 32, n + 48, in one order for all four.
__device__ __forceinline__ float cross_row_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float s = __uint_as_float(a[0]) + __uint_as_float(a[1]);  // rows (0+1), (2+3)
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
// max(a, b) as the median of (a, b, +inf): one v_med3_f32, which needs no
// NaN-quieting of its operands (the inputs here are never NaN).
// +inf from a register the compiler cannot see into, so that it keeps the
// median instruction instead of turning it back into a max (which would
// first quiet both operands).
__device__ __forceinline__ float opaque_inf() {
  float r;
  asm("v_mov_b32 %0, 0x7f800000" : "=v"(r));
  return r;
}
__device__ __forceinline__ float max2_med3(float a, float b) {
  return __builtin_amdgcn_fmed3f(a, b, opaque_inf());
}
// All ones on the lanes where keep holds, zero elsewhere, through an empty
// asm.  A choice between a loaded value and a constant written as a select
// may be turned back into a branch on the condition, with the load moved
// into it and waited for on its own; a mask the compiler cannot see into
// keeps such loads unconditional, so that they are in flight together.
__device__ __forceinline__ uint32_t opaque_mask(bool keep) {
  uint32_t m = keep ? 0xFFFFFFFFu : 0u;
  asm("" : "+v"(m));
  return m;
}
// v where the mask is all ones, `other` where it is zero.
__device__ __forceinline__ float keep_or(float v, uint32_t mask, float other) {
  return __uint_as_float((__float_as_uint(v) & mask) | (__float_as_uint(other) & ~mask));
}
__device__ __forceinline__ int keep_or(int v, uint32_t mask, int other) {
  return (int)(((uint32_t)v & mask) | ((uint32_t)other & ~mask));
}
// v where the mask is all ones, +0 where it is zero.
__device__ __forceinline__ float keep_or_zero(float v, uint32_t mask) {
  return __uint_as_float(__float_as_uint(v) & mask);
}

// Maximum over the four lanes n, n + 16, n + 32, n + 48 (each swap hands a
// lane both values of its pair, as in cross_row_sum).
__device__ __forceinline__ float cross_row_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m = max2_med3(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return max2_med3(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// wave_max for inputs that are never NaN: each step is one v_med3 with
// +inf, without the NaN-quieting of both operands that fmaxf needs.
__device__ __forceinline__ float wave_max_fin(float v) {
  v = max2_med3(v, dpp_f32<0xB1>(v));
  v = max2_med3(v, dpp_f32<0x4E>(v));
  v = max2_med3(v, dpp_f32<0x141>(v));
  v = max2_med3(v, dpp_f32<0x140>(v));
  return max2_med3(max2_med3(lane_f32(v, 0), lane_f32(v, 16)), max2_med3(lane_f32(v, 32), lane_f32(v, 48)));
}

// Maximum over each row of 16 lanes (every lane of the row gets it).
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  return fmaxf(v, dpp_f32<0x140>(v));
}

// DPP move with a row mask: rows outside `rows` keep 0 (the added term).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_rows_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xF, false));
}

// Inclusive prefix sum over the 64 lanes: a four-step scan inside each row of
// 16 (row_shr 1, 2, 4, 8), then the row totals passed on with the GFX9 row
// broadcasts: lane 15 of each even row to the odd row after it (rows 1 and
// 3), then lane 31 to rows 2 and 3.  With non-negative inputs every step
// adds non-negative terms, so the sums never decrease along the lanes.
__device__ __forceinline__ float wave_incl_scan(float x) {
  x += dpp_f32<0x111>(x);
  x += dpp_f32<0x112>(x);
  x += dpp_f32<0x114>(x);
  x += dpp_f32<0x118>(x);
  x += dpp_rows_f32<0x142, 0xA>(x);
  x += dpp_rows_f32<0x143, 0xC>(x);
  return x;
}

}  // namespace ts
