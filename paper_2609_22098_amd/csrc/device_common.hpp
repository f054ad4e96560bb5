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
// with log(1 - q0) = log1mexp(lq) in the two-branch form of Maechler (2012).
__device__ __forceinline__ float log_phat(float lq, float a, float b) {
  float logit;
  if (!(lq < 0.0f)) {
    logit = __builtin_huge_valf();
  } else {
    const float l1m = (lq > -kLn2) ? logf(-expm1f(lq)) : log1pf(-expf(lq));
    logit = lq - l1m;
  }
  const float x = (a == 0.0f) ? b : a * logit + b;
  if (x == __builtin_huge_valf()) return 0.0f;
  if (x == -__builtin_huge_valf()) return -__builtin_huge_valf();
  return (x >= 0.0f) ? -log1pf(expf(-x)) : x - log1pf(expf(x));
}

// Wave-wide reductions (64 lanes) with a fixed butterfly order.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace ts
