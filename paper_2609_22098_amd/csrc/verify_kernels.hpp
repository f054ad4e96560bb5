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
// a Gumbel-max draw from the final residual.  qT comes from the logits z
// recomputed by the expansion's streaming pass (the proposal is rebuilt from U
// and the draw order, not stored).  R_j is summed from positive terms only
// (tokens that are not children, plus the children not yet drawn), so it
// keeps its relative precision when one child holds almost all of qT.
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

// ---- T > 0: passes over (item, vocabulary chunk) workgroups ----------------
//
// One level of the walk is a fixed sequence of launches over the items (the
// requests still walking, each at its current node): pass A, stages 1..m_max,
// the bonus pass and the resolve kernel.  No launch needs the host in between:
// every workgroup first rebuilds its item's state (normalisers, alpha, beta,
// the stages already decided) from the chunk partials of the earlier
// launches, in one fixed order, so all workgroups of an item agree bit for bit.
// All logits are handled in base-2 units (x = logit * log2(e) / T).

constexpr int kVChunkQuantum = 4 * kVerifyThreads;  // tokens per sweep of a workgroup

struct VPartA {  // per (item, chunk)
  float mt;      // max of the target's x over the chunk
  float mz;      // max of the draft's x over the chunk (items with children)
  double st;     // sum of 2^(x_t - mt) over the chunk
  double snc;    // sum of 2^(x_z - mz) over the chunk's tokens that are not children
};

struct VBonusPart {  // per (item, chunk): best and second-best bonus key
  float best, second;
  int32_t idx, pad;
};

struct VerifyPass {
  const void* target;  // [R][cap][V]
  int cap, V;
  const VerifyItem* items;
  int nitems;
  const float* zbuf;   // recomputed draft logits, row items[i].zrow
  float c;             // log2(e) / T
  PhiloxKeys keys;
  int nchunks, chunk;  // chunk: multiple of kVChunkQuantum
  VPartA* pa;          // [nitems][nchunks]
  double* zp;          // [TS_MAX_K][nitems][nchunks]: chunk shares of Z_j
  VBonusPart* bp;      // [nitems][nchunks]
  VerifyResult* results;
};

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// State of one item after the stages before `upto` (computed by one whole
// wave; every lane ends with the same values).
struct VState {
  float Lt, Lz;       // base-2 log normalisers of p = softmax(t/T) and qT = softmax(z/T)
  float alpha, beta;  // residual p_s = max(alpha p - beta qT, 0) at the stage reached
  float betap;        // beta + 1 / R_s at the stage reached
  int accepted;       // stage (1-based) whose child was accepted, 0 if none so far
  int reached;        // stage reached (its test rejected or not run), m + 1 after all
  float margin;       // smallest |log u - log ratio| over the tests run (natural log)
};

template <typename TT>
__device__ VState verify_state(const VerifyPass& vp, const VerifyItem& item, int it, int upto) {
  const int lane = threadIdx.x & 63;
  const int nc = vp.nchunks;
  const VPartA* pa = vp.pa + (size_t)it * nc;
  float mt = kNegInf, mz = kNegInf;
  for (int k = lane; k < nc; k += 64) {
    mt = fmaxf(mt, pa[k].mt);
    mz = fmaxf(mz, pa[k].mz);
  }
  mt = wave_max(mt);
  mz = wave_max(mz);
  double st = 0.0, snc = 0.0;
  for (int k = lane; k < nc; k += 64) {
    st += pa[k].st * (double)exp2_fast(pa[k].mt - mt);
    if (item.m > 0) snc += pa[k].snc * (double)exp2_fast(pa[k].mz - mz);
  }
  st = wave_sum_f64(st);
  snc = wave_sum_f64(snc);
  VState v;
  v.Lt = mt + (float)log2(st);
  v.alpha = 1.0f;
  v.beta = 0.0f;
  v.betap = 1.0f;
  v.accepted = 0;
  v.reached = 1;
  v.margin = __builtin_huge_valf();
  v.Lz = 0.0f;
  const int m = item.m;
  if (m == 0) return v;
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const float* zrow = vp.zbuf + (size_t)item.zrow * vp.V;
  // suffix sums of the proposal mass: suf[s] = non-children + children s..m
  double suf[TS_MAX_K + 1];
  {
    double acc = snc;
    suf[TS_MAX_K] = acc;
#pragma unroll
    for (int s = TS_MAX_K - 1; s >= 0; --s) {
      if (s < m) acc += (double)exp2_fast(zrow[item.child_tok[s]] * vp.c - mz);
      suf[s] = acc;
    }
  }
  v.Lz = mz + (float)log2(suf[0]);
  const uint32_t pc1 = (uint32_t)item.path, pc2 = (uint32_t)(item.path >> 32);
  const uint32_t c3 = counter_word3(item.request, item.depth, 2u);
  const int last = upto < m ? upto : m;
#pragma unroll 1
  for (int s = 1; s <= last; ++s) {
    const int x = item.child_tok[s - 1];
    const float lp = target_at(trow, x) * vp.c - v.Lt;
    const float lq = zrow[x] * vp.c - v.Lz;
    float lpj;
    if (s == 1) {
      lpj = lp;
    } else {
      const float pj = v.alpha * exp2_fast(lp) - v.beta * exp2_fast(lq);
      lpj = pj > 0.0f ? __builtin_amdgcn_logf(pj) : kNegInf;
    }
    double Rs = 0.0;
#pragma unroll
    for (int k = 0; k < TS_MAX_K; ++k)
      if (k == s - 1) Rs = suf[k] / suf[0];
    const float lr = lpj - (lq - (float)log2(Rs));
    uint32_t w0 = (uint32_t)s, w1 = pc1, w2 = pc2, w3 = c3;
    philox10(w0, w1, w2, w3, vp.keys);
    const float lu = __builtin_amdgcn_logf(word_to_uniform(w0));
    v.margin = fminf(v.margin, fabsf(lu - lr) * kLn2);
    v.betap = v.beta + (float)(1.0 / Rs);
    v.reached = s;
    if (lu < lr) {
      v.accepted = s;
      return v;
    }
    if (s == upto) return v;  // the caller reduces Z_s
    const double* zs = vp.zp + ((size_t)(s - 1) * vp.nitems + it) * nc;
    double Z = 0.0;
    for (int k = lane; k < nc; k += 64) Z += zs[k];
    Z = wave_sum_f64(Z);
    if (Z > 0.0) {
      v.alpha = (float)(v.alpha / Z);
      v.beta = (float)(v.betap / Z);
    }
    v.reached = s + 1;
  }
  return v;
}

// Shares the state of wave 0 with the workgroup.
__device__ __forceinline__ VState share_state(const VState& v, VState* sh) {
  if (threadIdx.x == 0) *sh = v;
  __syncthreads();
  return *sh;
}

// Children of the item inside [y0, y1), first n of them, into LDS; returns the count.
__device__ __forceinline__ int chunk_children(const VerifyItem& item, int n, int y0, int y1, int* loc,
                                              int* cnt) {
  if (threadIdx.x == 0) {
    int k = 0;
    for (int s = 0; s < n; ++s) {
      const int x = item.child_tok[s];
      if (x >= y0 && x < y1) loc[k++] = x;
    }
    *cnt = k;
  }
  __syncthreads();
  return *cnt;
}

__device__ __forceinline__ bool is_listed(int y, const int* loc, int n) {
  bool hit = false;
  for (int k = 0; k < n; ++k) hit |= (loc[k] == y);
  return hit;
}

// Fixed-order workgroup reductions in double.
__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  v = wave_sum_f64(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// Pass A: per-chunk maxima and sums of the target and draft rows.
template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_pass_a_kernel(VerifyPass vp) {
  __shared__ float red[4];
  __shared__ double redd[4];
  __shared__ int loc[TS_MAX_K];
  __shared__ int cnt;
  const int it = blockIdx.x / vp.nchunks, ck = blockIdx.x % vp.nchunks;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  const int y0 = ck * vp.chunk, y1 = min(vp.V, y0 + vp.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const float* zrow = item.m > 0 ? vp.zbuf + (size_t)item.zrow * vp.V : nullptr;
  const int nloc = item.m > 0 ? chunk_children(item, item.m, y0, y1, loc, &cnt) : 0;
  float mt = kNegInf, mz = kNegInf;
  for (int b = y0 + 4 * threadIdx.x; b < y1; b += kVChunkQuantum) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = b + e;
      if (y < y1) {
        mt = fmaxf(mt, target_at(trow, y) * vp.c);
        if (zrow) mz = fmaxf(mz, zrow[y] * vp.c);
      }
    }
  }
  mt = block_max(mt, red);
  mz = block_max(mz, red);
  float st = 0.0f, snc = 0.0f;
  for (int b = y0 + 4 * threadIdx.x; b < y1; b += kVChunkQuantum) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = b + e;
      if (y < y1) {
        st += exp2_fast(target_at(trow, y) * vp.c - mt);
        if (zrow && !(nloc && is_listed(y, loc, nloc))) snc += exp2_fast(zrow[y] * vp.c - mz);
      }
    }
  }
  const double dst = block_sum_f64((double)st, redd);
  const double dsnc = block_sum_f64((double)snc, redd);
  if (threadIdx.x == 0) {
    VPartA r;
    r.mt = mt;
    r.mz = mz;
    r.st = dst;
    r.snc = dsnc;
    vp.pa[(size_t)it * vp.nchunks + ck] = r;
  }
}

// Stage j: if the item's walk reaches stage j and child j is rejected, this
// workgroup adds its chunk's share of Z_j = sum max(alpha_j p - beta'_j qT, 0)
// over tokens not drawn up to j.
template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_stage_kernel(VerifyPass vp, int j) {
  __shared__ VState sh;
  __shared__ double redd[4];
  __shared__ int loc[TS_MAX_K];
  __shared__ int cnt;
  const int it = blockIdx.x / vp.nchunks, ck = blockIdx.x % vp.nchunks;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  if (item.m < j) return;
  VState v;
  if (threadIdx.x < 64) v = verify_state<TT>(vp, item, it, j);
  v = share_state(v, &sh);
  if (v.accepted != 0 || v.reached != j) return;
  const int y0 = ck * vp.chunk, y1 = min(vp.V, y0 + vp.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const float* zrow = vp.zbuf + (size_t)item.zrow * vp.V;
  const int nloc = chunk_children(item, j, y0, y1, loc, &cnt);
  float acc = 0.0f;
  for (int b = y0 + 4 * threadIdx.x; b < y1; b += kVChunkQuantum) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = b + e;
      if (y < y1 && !(nloc && is_listed(y, loc, nloc))) {
        const float p = exp2_fast(target_at(trow, y) * vp.c - v.Lt);
        const float q = exp2_fast(zrow[y] * vp.c - v.Lz);
        acc += fmaxf(v.alpha * p - v.betap * q, 0.0f);
      }
    }
  }
  const double z = block_sum_f64((double)acc, redd);
  if (threadIdx.x == 0) vp.zp[((size_t)(j - 1) * vp.nitems + it) * vp.nchunks + ck] = z;
}

// Bonus: when every child was rejected (or there is none), the chunk's best
// Gumbel-max key log2 r(y) - log2(-log2 u_y) over the final residual r.
template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_bonus_kernel(VerifyPass vp) {
  __shared__ VState sh;
  __shared__ float redv[4];
  __shared__ int redi[4];
  __shared__ int loc[TS_MAX_K];
  __shared__ int cnt;
  const int it = blockIdx.x / vp.nchunks, ck = blockIdx.x % vp.nchunks;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  VState v;
  if (threadIdx.x < 64) v = verify_state<TT>(vp, item, it, TS_MAX_K + 1);
  v = share_state(v, &sh);
  if (v.accepted != 0) return;
  const int y0 = ck * vp.chunk, y1 = min(vp.V, y0 + vp.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const float* zrow = item.m > 0 ? vp.zbuf + (size_t)item.zrow * vp.V : nullptr;
  const int nloc = item.m > 0 ? chunk_children(item, item.m, y0, y1, loc, &cnt) : 0;
  const uint32_t pc1 = (uint32_t)item.path, pc2 = (uint32_t)(item.path >> 32);
  const uint32_t c3 = counter_word3(item.request, item.depth, 3u);
  float bv = kNegInf, sv = kNegInf;
  int bi = 0x7FFFFFFF;
  for (int b = y0 + 4 * threadIdx.x; b < y1; b += kVChunkQuantum) {
    uint32_t w0 = (uint32_t)b >> 2, w1 = pc1, w2 = pc2, w3 = c3;
    philox10(w0, w1, w2, w3, vp.keys);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = b + e;
      if (y >= y1) break;
      float l2r;
      if (!zrow) {
        l2r = target_at(trow, y) * vp.c - v.Lt;
      } else {
        if (nloc && is_listed(y, loc, nloc)) continue;
        const float p = exp2_fast(target_at(trow, y) * vp.c - v.Lt);
        const float q = exp2_fast(zrow[y] * vp.c - v.Lz);
        const float r = v.alpha * p - v.beta * q;
        if (!(r > 0.0f)) continue;
        l2r = __builtin_amdgcn_logf(r);
      }
      const uint32_t w = e == 0 ? w0 : e == 1 ? w1 : e == 2 ? w2 : w3;
      const float key = l2r - __builtin_amdgcn_logf(-__builtin_amdgcn_logf(word_to_uniform(w)));
      if (key > bv) { sv = bv; bv = key; bi = y; }
      else if (key > sv) sv = key;
    }
  }
  float vb = bv;
  int id = bi;
  block_argmax(vb, id, redv, redi);
  float s2 = (bi == id) ? sv : bv;
  s2 = block_max(s2, redv);
  if (threadIdx.x == 0) {
    VBonusPart r;
    r.best = vb;
    r.second = s2;
    r.idx = id;
    r.pad = 0;
    vp.bp[(size_t)it * vp.nchunks + ck] = r;
  }
}

// Resolve: one wave per item writes the accepted stage, or the bonus token.
template <typename TT>
__global__ __launch_bounds__(64) void verify_resolve_kernel(VerifyPass vp) {
  const int it = blockIdx.x;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  const VState v = verify_state<TT>(vp, item, it, TS_MAX_K + 1);
  const int lane = threadIdx.x;
  VerifyResult r;
  r.accepted = v.accepted;
  r.bonus = -1;
  r.margin = v.margin;
  r.pad = 0;
  if (v.accepted == 0) {
    const VBonusPart* bp = vp.bp + (size_t)it * vp.nchunks;
    float best = kNegInf, second = kNegInf;
    int idx = 0x7FFFFFFF;
    for (int k = lane; k < vp.nchunks; k += 64) {
      const VBonusPart b = bp[k];
      if (b.best > best || (b.best == best && b.idx < idx)) {
        second = fmaxf(second, best);
        best = b.best;
        idx = b.idx;
        second = fmaxf(second, b.second);
      } else {
        second = fmaxf(second, b.best);
      }
    }
    float vb = best;
    int id = idx;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(vb, o, 64);
      const int oi = __shfl_xor(id, o, 64);
      if (ov > vb || (ov == vb && oi < id)) { vb = ov; id = oi; }
    }
    const float s2 = wave_max(idx == id ? second : best);
    const float gap = (vb - s2) * kLn2 / fmaxf(1.0f, fabsf(vb * kLn2));
    r.bonus = id;
    r.margin = fminf(r.margin, gap);
  }
  if (lane == 0) vp.results[it] = r;
}

}  // namespace ts
