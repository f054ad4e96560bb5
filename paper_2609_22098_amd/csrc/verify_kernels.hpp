// Kernels of tree verification (ts_verify).
//
// T = 0 (§3.2 item 3): the greedy walk only needs the target argmax of each
// tree row, so one kernel computes every row's argmax (ties: smallest id) and
// the host descends the tree.
//
// T > 0 (§3.3, Proposition 1): at a visited node with children x_1..x_m in
// draw order, stage j tests u_j < p_j(x_j) / q_j(x_j) where
//   q_j = qT restricted to tokens not drawn before j, renormalised by R_j,
//   p_{j+1} = norm(max(p_j - q_j, 0)).
// At every stage the walk can reach, p_j(y) = max(alpha_j p(y) - beta_j qT(y), 0)
// for tokens not drawn before j (tokens drawn earlier have p_j = 0), with
//   alpha_1 = 1, beta_1 = 0,  beta'_j = beta_j + 1/R_j,
//   Z_j = sum_y max(alpha_j p(y) - beta'_j qT(y), 0),
//   alpha_{j+1} = alpha_j / Z_j,  beta_{j+1} = beta'_j / Z_j,
// so each rejected stage costs one vocabulary reduction.  The bonus token is
// a Gumbel-max draw from the final residual.  One workgroup handles one
// request's current node; qT comes from the logits z recomputed by pass 1 of
// the expansion (the proposal is rebuilt from U and the draw order, not stored).
#pragma once

#include "device_common.hpp"

namespace ts {

constexpr int kVerifyThreads = 256;

template <typename TT>
__device__ __forceinline__ float target_at(const TT* row, int y) {
  if constexpr (sizeof(TT) == 2)
    return bf16_to_f32(row[y]);
  else
    return row[y];
}

// Block-wide (256 threads) reductions with a fixed order: a wave butterfly,
// then the four wave results in wave order.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
// argmax by (value desc, id asc)
__device__ __forceinline__ void block_argmax(float& v, int& id, float* redv, int* redi) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(v, o, 64);
    const int oi = __shfl_xor(id, o, 64);
    if (ov > v || (ov == v && oi < id)) { v = ov; id = oi; }
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) { redv[wv] = v; redi[wv] = id; }
  __syncthreads();
  v = redv[0]; id = redi[0];
  for (int w = 1; w < 4; ++w)
    if (redv[w] > v || (redv[w] == v && redi[w] < id)) { v = redv[w]; id = redi[w]; }
}

// Greedy: argmax of each existing tree row.  rows[i] = request * cap + node.
template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_argmax_kernel(const TT* target, int V,
                                                                       const int* rows, int nrows,
                                                                       int* argmax_out,
                                                                       float* gap_out) {
  __shared__ float redv[4];
  __shared__ int redi[4];
  const int i = blockIdx.x;
  if (i >= nrows) return;
  const TT* row = target + (size_t)rows[i] * V;
  float bv = kNegInf, sv = kNegInf;
  int bi = 0x7FFFFFFF;
  for (int y = threadIdx.x; y < V; y += kVerifyThreads) {
    const float t = target_at(row, y);
    if (t > bv) { sv = bv; bv = t; bi = y; }
    else if (t > sv) sv = t;
  }
  float v = bv;
  int id = bi;
  block_argmax(v, id, redv, redi);
  // second-best value for near-tie reporting: the best value other than the argmax
  float s2 = (bi == id) ? sv : bv;
  s2 = block_max(s2, redv);
  if (threadIdx.x == 0) {
    argmax_out[i] = id;
    gap_out[i] = (v - s2) / fmaxf(1.0f, fabsf(v));
  }
}

struct VerifyItem {
  int32_t request;
  int32_t node;
  int32_t depth;
  int32_t m;      // children of the node in the tree (draw order)
  uint64_t path;
  int32_t zrow;   // row of the recomputed logits, -1 when m == 0
  int32_t pad;
  int32_t child_tok[TS_MAX_K];
};

struct VerifyResult {
  int32_t accepted;  // 1-based sibling index of the accepted child, 0 = none
  int32_t bonus;     // bonus token when accepted == 0
  float margin;      // smallest |log u - log ratio| (or bonus key gap)
  int32_t pad;
};

template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_stage_kernel(
    const TT* target, int cap, int V, const VerifyItem* items, int nitems, const float* zbuf,
    float T, PhiloxKeys keys, VerifyResult* results) {
  __shared__ float red[4];
  __shared__ int redi[4];
  __shared__ float sh[4];
  const int it = blockIdx.x;
  if (it >= nitems) return;
  const VerifyItem item = items[it];
  const TT* trow = target + ((size_t)item.request * cap + item.node) * V;
  const float* z = item.m > 0 ? zbuf + (size_t)item.zrow * V : nullptr;
  const float invT = 1.0f / T;
  const float c = kLog2e * invT;

  // log-sum-exp of t/T and z/T (fixed per-thread order, fixed block tree)
  float mt = kNegInf, mz = kNegInf;
  for (int y = threadIdx.x; y < V; y += kVerifyThreads) {
    mt = fmaxf(mt, target_at(trow, y));
    if (z) mz = fmaxf(mz, z[y]);
  }
  mt = block_max(mt, red);
  mz = block_max(mz, red);
  float st = 0.0f, sz = 0.0f;
  for (int y = threadIdx.x; y < V; y += kVerifyThreads) {
    st += exp2_fast((target_at(trow, y) - mt) * c);
    if (z) sz += exp2_fast((z[y] - mz) * c);
  }
  st = block_sum(st, red);
  sz = block_sum(sz, red);
  // natural-log normalisers of p = softmax(t/T) and qT = softmax(z/T)
  const float lse_t = mt * invT + logf(st);
  const float lse_z = z ? mz * invT + logf(sz) : 0.0f;

  float alpha = 1.0f, beta = 0.0f, R = 1.0f;
  int accepted = 0;
  float margin = __builtin_huge_valf();
  const uint32_t pc1 = (uint32_t)item.path, pc2 = (uint32_t)(item.path >> 32);
  for (int j = 1; j <= item.m; ++j) {
    const int x = item.child_tok[j - 1];
    const float lp = target_at(trow, x) * invT - lse_t;
    const float lq = z[x] * invT - lse_z;
    float log_pj;
    if (j == 1) {
      log_pj = lp;
    } else {
      const float pj = alpha * expf(lp) - beta * expf(lq);
      log_pj = pj > 0.0f ? logf(pj) : -__builtin_huge_valf();
    }
    const float log_ratio = log_pj - (lq - logf(R));
    uint32_t c0 = (uint32_t)j, c1 = pc1, c2 = pc2, c3 = counter_word3(item.request, item.depth, 2u);
    philox10(c0, c1, c2, c3, keys);
    const float lu = logf(word_to_uniform(c0));
    margin = fminf(margin, fabsf(lu - log_ratio));
    if (lu < log_ratio) { accepted = j; break; }
    // rejected: residual p_{j+1} and the remaining proposal mass R_{j+1}
    const float betap = beta + 1.0f / R;
    float zs = 0.0f, rs = 0.0f;
    for (int y = threadIdx.x; y < V; y += kVerifyThreads) {
      const float py = exp2_fast((target_at(trow, y) - mt) * c) / st;
      const float qy = exp2_fast((z[y] - mz) * c) / sz;
      zs += fmaxf(alpha * py - betap * qy, 0.0f);
      bool drawn = false;
      for (int s = 0; s < j; ++s) drawn |= (item.child_tok[s] == y);
      if (!drawn) rs += qy;
    }
    zs = block_sum(zs, red);
    rs = block_sum(rs, sh);
    if (zs > 0.0f) {
      alpha = alpha / zs;
      beta = betap / zs;
    }
    R = rs;
  }
  if (accepted == 0) {
    // bonus: argmax over y with residual r(y) > 0 of log2 r(y) - log2(-log2 u_y)
    float bv = kNegInf, sv = kNegInf;
    int bi = 0x7FFFFFFF;
    const uint32_t c3b = counter_word3(item.request, item.depth, 3u);
    for (int y4 = threadIdx.x * 4; y4 < V; y4 += kVerifyThreads * 4) {
      uint32_t c0 = (uint32_t)y4 >> 2, c1 = pc1, c2 = pc2, c3 = c3b;
      philox10(c0, c1, c2, c3, keys);
      const uint32_t w[4] = {c0, c1, c2, c3};
      for (int q = 0; q < 4; ++q) {
        const int y = y4 + q;
        if (y >= V) break;
        float l2r;
        if (item.m == 0) {
          l2r = (target_at(trow, y) - mt) * c - __builtin_amdgcn_logf(st);
        } else {
          const float py = exp2_fast((target_at(trow, y) - mt) * c) / st;
          const float qy = exp2_fast((z[y] - mz) * c) / sz;
          const float ry = alpha * py - beta * qy;
          if (!(ry > 0.0f)) continue;
          l2r = __builtin_amdgcn_logf(ry);
        }
        const float key = l2r - __builtin_amdgcn_logf(-__builtin_amdgcn_logf(word_to_uniform(w[q])));
        if (key > bv) { sv = bv; bv = key; bi = y; }
        else if (key > sv) sv = key;
      }
    }
    float v = bv;
    int id = bi;
    block_argmax(v, id, red, redi);
    float s2 = (bi == id) ? sv : bv;
    s2 = block_max(s2, red);
    if (threadIdx.x == 0) {
      // gap in natural-log units
      const float gap = (v - s2) * kLn2 / fmaxf(1.0f, fabsf(v * kLn2));
      margin = fminf(margin, gap);
      results[it].bonus = id;
    }
  }
  if (threadIdx.x == 0) {
    results[it].accepted = accepted;
    results[it].margin = margin;
    if (accepted) results[it].bonus = -1;
  }
}

}  // namespace ts
