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

// Target values (as float) and draft logits of tokens b .. b+3.  A quad that
// lies wholly before y1 in rows whose length is a multiple of 4 (vec) is read
// with one vector load per row; otherwise token by token, and tokens at or
// past y1 read as 0 (the callers skip them).  zrow may be null (z reads 0).
template <bool HZ, typename TT>
__device__ __forceinline__ void load_quad_vec(const TT* trow, const float* zrow, int b, float (&t)[4],
                                              float (&z)[4]) {
  if constexpr (sizeof(TT) == 2) {
    const uint2 w = *reinterpret_cast<const uint2*>(trow + b);
    t[0] = __uint_as_float(w.x << 16);
    t[1] = __uint_as_float(w.x & 0xFFFF0000u);
    t[2] = __uint_as_float(w.y << 16);
    t[3] = __uint_as_float(w.y & 0xFFFF0000u);
  } else {
    const f32x4 v = *reinterpret_cast<const f32x4*>(trow + b);
    t[0] = v[0]; t[1] = v[1]; t[2] = v[2]; t[3] = v[3];
  }
  if constexpr (HZ) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(zrow + b);
    z[0] = v[0]; z[1] = v[1]; z[2] = v[2]; z[3] = v[3];
  } else {
    z[0] = z[1] = z[2] = z[3] = 0.0f;
  }
}
template <typename TT>
__device__ __forceinline__ void load_quad(const TT* trow, const float* zrow, int b, int y1, bool vec,
                                          float (&t)[4], float (&z)[4]) {
  if (vec && b + 4 <= y1) {
    if constexpr (sizeof(TT) == 2) {
      const uint2 w = *reinterpret_cast<const uint2*>(trow + b);
      t[0] = __uint_as_float(w.x << 16);
      t[1] = __uint_as_float(w.x & 0xFFFF0000u);
      t[2] = __uint_as_float(w.y << 16);
      t[3] = __uint_as_float(w.y & 0xFFFF0000u);
    } else {
      const f32x4 v = *reinterpret_cast<const f32x4*>(trow + b);
      t[0] = v[0]; t[1] = v[1]; t[2] = v[2]; t[3] = v[3];
    }
    if (zrow) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(zrow + b);
      z[0] = v[0]; z[1] = v[1]; z[2] = v[2]; z[3] = v[3];
    } else {
      z[0] = z[1] = z[2] = z[3] = 0.0f;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = b + e;
      t[e] = y < y1 ? target_at(trow, y) : 0.0f;
      z[e] = (zrow && y < y1) ? zrow[y] : 0.0f;
    }
  }
}

// One workgroup's pass over the tokens [y0, y1) of a target row and a draft
// row (zrow may be null): thread t takes the quad y0 + 4t + 1024 s in sweep
// s, in sweep order, and calls f(b, t[4], z[4], nv) with the quad's first
// token b and its nv tokens before y1.  Sweeps whose quads are all whole
// (vec: rows of a multiple of 4 tokens) are read four at a time, every load
// issued before any use, so a workgroup waits for memory about once per four
// sweeps.
template <bool HZ, typename TT, typename F>
__device__ __forceinline__ void sweep_rows(const TT* trow, const float* zrow, int y0, int y1, bool vec, F&& f) {
  constexpr int kQ = kVerifyThreads * 4;  // tokens per sweep
  const int b0 = y0 + 4 * threadIdx.x;
  const int nfull = vec ? (y1 - y0) / kQ : 0;
  int sw = 0;
  for (; sw + 4 <= nfull; sw += 4) {
    float t[4][4], z[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) load_quad_vec<HZ>(trow, zrow, b0 + (sw + u) * kQ, t[u], z[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u) f(b0 + (sw + u) * kQ, t[u], z[u], 4);
  }
  for (; sw < nfull; ++sw) {
    float t[4], z[4];
    load_quad_vec<HZ>(trow, zrow, b0 + sw * kQ, t, z);
    f(b0 + sw * kQ, t, z, 4);
  }
  for (int b = b0 + sw * kQ; b < y1; b += kQ) {
    float t[4], z[4];
    load_quad(trow, zrow, b, y1, vec, t, z);
    f(b, t, z, min(4, y1 - b));
  }
}
template <typename TT, typename F>
__device__ __forceinline__ void sweep_chunk(const TT* trow, const float* zrow, int y0, int y1, bool vec, F&& f) {
  if (zrow)
    sweep_rows<true>(trow, zrow, y0, y1, vec, f);
  else
    sweep_rows<false>(trow, zrow, y0, y1, vec, f);
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
  auto take = [&](float t, int y) {
    if (t > bv) { sv = bv; bv = t; bi = y; }
    else if (t > sv) sv = t;
  };
  // 16-byte groups of G tokens (rows 16-byte aligned: V a multiple of G),
  // four groups in flight per thread; each thread scans its tokens in
  // increasing order, so ties keep the smallest id
  constexpr int G = 16 / (int)sizeof(TT);
  constexpr int kStep = kVerifyThreads * G;
  int y0 = 0;
  if (V % G == 0 && (reinterpret_cast<uintptr_t>(target) & 15) == 0) {
    const int nfull = V / kStep;
    int sw = 0;
    for (; sw < nfull; sw += 4) {
      u32x4 w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (sw + u < nfull) w[u] = *reinterpret_cast<const u32x4*>(row + (sw + u) * kStep + G * threadIdx.x);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (sw + u >= nfull) break;
        const int yb = (sw + u) * kStep + G * threadIdx.x;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if constexpr (sizeof(TT) == 2) {
            take(__uint_as_float(w[u][k] << 16), yb + 2 * k);
            take(__uint_as_float(w[u][k] & 0xFFFF0000u), yb + 2 * k + 1);
          } else {
            take(__uint_as_float(w[u][k]), yb + k);
          }
        }
      }
    }
    y0 = nfull * kStep;
  }
  for (int y = y0 + threadIdx.x; y < V; y += kVerifyThreads) take(target_at(row, y), y);
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
  int32_t bonus;     // bonus token when accepted == 0, or at the accepted leaf (leaf_bonus)
  float margin;      // smallest |log u - log ratio| (or bonus key gap)
  int32_t leaf_bonus;  // 1: the accepted child has no children and bonus is its draw
};

// The children of a level item as the one-launch level needs them to carry
// on into an accepted child without children: its node, its path and whether
// it has children (pinned host memory, one per item).
struct VerifyNext {
  int32_t child_node[TS_MAX_K];
  uint64_t child_path[TS_MAX_K];
  uint32_t leaf_mask;  // bit s: child s (draw order) has no children
  int32_t pad;
};

// ---- T > 0: passes over (item, vocabulary chunk) workgroups ----------------
//
// One level of the walk is a fixed sequence of launches over the items (the
// requests still walking, each at its current node): pass A, stages
// 1..max(m_max, 1) and the resolve kernel.  No launch needs the host in
// between.  The bonus keys are taken by the sweep that already reads the
// residual they come from: pass A for a leaf, the last child's stage for a
// node whose children were all rejected.  The stage-1 launch turns the pass-A partials into the
// item's constants; each stage launch then advances the item's record (alpha,
// beta, the decision so far) by one stage from the previous launch's record
// and Z partials.  Every workgroup of an item computes that step in the same
// fixed order, so they agree bit for bit, and chunk 0 stores it.  All logits
// are handled in base-2 units (x = logit * log2(e) / T).

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

struct VConst;
struct VRec;

struct VerifyPass {
  const void* target;  // [R][cap][V]
  int cap, V;
  const VerifyItem* items;       // [nitems], device copy (staged by pass A)
  const VerifyItem* items_host;  // [nitems], pinned host memory: read by pass A only
  VerifyItem* items_w;           // the device copy, written by pass A
  int nitems;
  const float* zbuf;   // recomputed draft logits, row items[i].zrow
  float c;             // log2(e) / T
  PhiloxKeys keys;
  int nchunks, chunk;  // chunk: multiple of kVChunkQuantum
  VPartA* pa;          // [nitems][nchunks]
  double* zp;          // [TS_MAX_K][nitems][nchunks]: chunk shares of Z_j
  VBonusPart* bp;      // [nitems][nchunks]
  VConst* consts;      // [nitems]: written by the stage-1 launch
  VRec* recs;          // [TS_MAX_K][nitems]: record after the launch of stage j, at j - 1
  VerifyResult* results;  // [nitems], pinned host memory
};

// Rows can be read in aligned quads: a multiple of 4 tokens long, the target
// at a 4-token-aligned address (the logits live in the workspace).
template <typename TT>
__device__ __forceinline__ bool vector_rows(const VerifyPass& vp) {
  return (vp.V & 3) == 0 && (reinterpret_cast<uintptr_t>(vp.target) & (4 * sizeof(TT) - 1)) == 0;
}

// Wave-wide fp64 sum in the fixed order of wave_sum: DPP moves of both
// halves (pairs, quads, halves of a row, rows), then the four rows' sums in
// order.  Every lane gets the same value.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, 0xF, 0xF, true);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<0xB1>(v);
  v += dpp_f64<0x4E>(v);
  v += dpp_f64<0x141>(v);
  v += dpp_f64<0x140>(v);
  return ((lane_f64(v, 0) + lane_f64(v, 16)) + lane_f64(v, 32)) + lane_f64(v, 48);
}

// Per-item constants of one level, written by the stage-1 launch: the base-2
// log normalisers and, for each child s in draw order, log2 p(x_s), log2 qT(x_s),
// log2 R_s, 1/R_s and log2 u_s of its acceptance test.
struct VConst {
  float Lt, Lz;
  float lp[TS_MAX_K], lq[TS_MAX_K], lR[TS_MAX_K], invR[TS_MAX_K], lu[TS_MAX_K];
};

// Walk state after the launch of stage j.
enum : int32_t { kRejected = 0, kAccepted = 1, kExhausted = 2 };
struct VRec {
  float alpha, beta;  // residual p_s = max(alpha p - beta qT, 0) at the stage reached
  float betap;        // beta + 1 / R_s when status == kRejected (the Z_s pass uses it)
  float margin;       // smallest |log u - log ratio| of the tests run (natural log)
  int32_t status;     // kRejected at `stage` (Z_stage pending), kAccepted at `stage`, kExhausted
  int32_t stage;
};

// Acceptance test of child s with the residual (alpha, beta) (wave-uniform).
__device__ __forceinline__ VRec stage_test(float lp, float lq, float lR, float invR, float lu, int s,
                                           float alpha, float beta, float margin) {
  VRec r;
  float lpj;
  if (s == 1) {
    lpj = lp;
  } else {
    const float pj = alpha * exp2_fast(lp) - beta * exp2_fast(lq);
    lpj = pj > 0.0f ? __builtin_amdgcn_logf(pj) : kNegInf;
  }
  const float lr = lpj - (lq - lR);
  r.alpha = alpha;
  r.beta = beta;
  r.betap = beta + invR;
  r.margin = fminf(margin, fabsf(lu - lr) * kLn2);
  r.status = lu < lr ? kAccepted : kRejected;
  r.stage = s;
  return r;
}

// Constants of an item from its nc pass-A partials, pa_at(k) for chunk k (one
// whole wave): every lane gets the normalisers, lane s < m child s's terms
// (zero on the other lanes).
struct VConstLane {
  float Lt, Lz;
  float lp, lq, lR, invR, lu;
};
// Child `lane`'s target value and draft logit (times c), zero past the
// children.  Loaded on every lane from valid addresses (a lane past m reads
// token 0 of the item's rows, logit row 0 when there is none) and masked after.
struct VChildVals {
  float tv, wzl;
};
template <typename TT>
__device__ __forceinline__ VChildVals load_child_vals(const VerifyPass& vp, const VerifyItem& item) {
  const int lane = threadIdx.x & 63;
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const uint32_t mine = opaque_mask(lane < item.m);
  const int ctok = item.child_tok[min(lane, TS_MAX_K - 1)] & (int)mine;
  const float* zrow = vp.zbuf + (size_t)max(item.zrow, 0) * vp.V;
  VChildVals v;
  v.tv = keep_or_zero(target_at(trow, ctok), mine);
  v.wzl = keep_or_zero(zrow[ctok] * vp.c, mine);
  return v;
}
template <typename TT, typename PartAt>
__device__ VConstLane verify_consts_lane(const VerifyPass& vp, const VerifyItem& item, int nc, PartAt&& pa_at,
                                         const VChildVals& cv) {
  const int lane = threadIdx.x & 63;
  const int m = item.m;
  const uint32_t mine = opaque_mask(lane < m);
  const float tv = cv.tv, wzl = cv.wzl;
  float mt = kNegInf, mz = kNegInf;
  for (int k = lane; k < nc; k += 64) {
    const VPartA a = pa_at(k);
    mt = fmaxf(mt, a.mt);
    mz = fmaxf(mz, a.mz);
  }
  mt = wave_max(mt);
  mz = wave_max(mz);
  double st = 0.0, snc = 0.0;
  for (int k = lane; k < nc; k += 64) {
    const VPartA a = pa_at(k);
    st += a.st * (double)exp2_fast(a.mt - mt);
    if (m > 0) snc += a.snc * (double)exp2_fast(a.mz - mz);
  }
  st = wave_sum_f64(st);
  snc = wave_sum_f64(snc);
  VConstLane C;
  C.Lt = mt + (float)log2(st);
  C.Lz = 0.0f;
  C.lp = 0.0f; C.lq = 0.0f; C.lR = 0.0f; C.invR = 0.0f; C.lu = 0.0f;
  if (m == 0) return C;
  // suffix sums of the proposal mass, suf[s] = non-children + children s..m-1,
  // added in the fixed order s = m-1 .. 0 from the children's terms of every lane
  const double el = mine ? (double)exp2_fast(wzl - mz) : 0.0;
  const uint64_t elb = __builtin_bit_cast(uint64_t, el);
  double acc = snc, my_suf = snc;
#pragma unroll
  for (int s = TS_MAX_K - 1; s >= 0; --s) {
    if (s < m) {
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)elb, s);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(elb >> 32), s);
      acc += __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
      if (lane == s) my_suf = acc;
    }
  }
  const double suf0 = acc;
  C.Lz = mz + (float)log2(suf0);
  // lane s: child s's terms
  if (mine) {
    const double Rs = my_suf / suf0;
    C.lp = tv * vp.c - C.Lt;
    C.lq = wzl - C.Lz;
    C.lR = (float)log2(Rs);
    C.invR = (float)(1.0 / Rs);
    uint32_t w0 = (uint32_t)(lane + 1), w1 = (uint32_t)item.path, w2 = (uint32_t)(item.path >> 32),
             w3 = counter_word3(item.request, item.depth, 2u);
    philox10(w0, w1, w2, w3, vp.keys);
    C.lu = __builtin_amdgcn_logf(word_to_uniform(w0));
  }
  return C;
}
// The same constants gathered on every lane.
template <typename TT, typename PartAt>
__device__ VConst verify_consts_from(const VerifyPass& vp, const VerifyItem& item, int nc, PartAt&& pa_at) {
  // the children's values are loaded alongside the partials
  const VConstLane L = verify_consts_lane<TT>(vp, item, nc, pa_at, load_child_vals<TT>(vp, item));
  const int m = item.m;
  VConst C;
  C.Lt = L.Lt;
  C.Lz = L.Lz;
#pragma unroll
  for (int s = 0; s < TS_MAX_K; ++s) {
    C.lp[s] = 0.0f; C.lq[s] = 0.0f; C.lR[s] = 0.0f; C.invR[s] = 0.0f; C.lu[s] = 0.0f;
    if (s < m) {
      C.lp[s] = lane_f32(L.lp, s);
      C.lq[s] = lane_f32(L.lq, s);
      C.lR[s] = lane_f32(L.lR, s);
      C.invR[s] = lane_f32(L.invR, s);
      C.lu[s] = lane_f32(L.lu, s);
    }
  }
  return C;
}
// Constants of item `it` from the partials of the pass-A launch.
template <typename TT>
__device__ VConst verify_consts(const VerifyPass& vp, const VerifyItem& item, int it) {
  const VPartA* pa = vp.pa + (size_t)it * vp.nchunks;
  return verify_consts_from<TT>(vp, item, vp.nchunks, [&](int k) { return pa[k]; });
}

// Record after the launch of stage j >= 2 from the record of stage j - 1.
// Total Z of stage s for item it from its chunk partials (one whole wave; every
// lane gets it, summed in a fixed order).  The partials are read whatever the
// item's state, so the loads go out with the record's (unused unless the
// record is a pending rejection at stage s).
__device__ __forceinline__ double stage_z(const VerifyPass& vp, int it, int s) {
  const int lane = threadIdx.x & 63;
  const double* zs = vp.zp + ((size_t)(s - 1) * vp.nitems + it) * vp.nchunks;
  double Z = 0.0;
  for (int k = lane; k < vp.nchunks; k += 64) Z += zs[k];
  return wave_sum_f64(Z);
}

// Child j's acceptance constants (index j - 1 of the item's constants).
struct VChild {
  float lp, lq, lR, invR, lu;
};
__device__ __forceinline__ VChild child_consts(const VConst& C, int k) {
  return VChild{C.lp[k], C.lq[k], C.lR[k], C.invR[k], C.lu[k]};
}

// The record for stage j from the one after stage j - 1: a pending rejection
// divides alpha and beta by its stage's total Z and tests child j (or, past
// the last child, ends the walk with the residual); any other state carries
// over.
__device__ __forceinline__ VRec verify_advance(const VRec& prev, double Z, const VChild& c, int m, int j) {
  if (prev.status != kRejected) return prev;
  float alpha = prev.alpha, beta = prev.beta;
  if (Z > 0.0) {
    alpha = (float)(alpha / Z);
    beta = (float)(prev.betap / Z);
  }
  if (j <= m) return stage_test(c.lp, c.lq, c.lR, c.invR, c.lu, j, alpha, beta, prev.margin);
  VRec r = prev;
  r.alpha = alpha;
  r.beta = beta;
  r.status = kExhausted;
  r.stage = j;
  return r;
}

// Shares a value computed by wave 0 with the workgroup.
template <typename S>
__device__ __forceinline__ S share(const S& v, S* sh) {
  if (threadIdx.x == 0) *sh = v;
  __syncthreads();
  return *sh;
}

// Children of the item inside [y0, y1), first n of them, into LDS; returns the count.
__device__ __forceinline__ int chunk_children(const VerifyItem& item, int n, int y0, int y1, int* loc,
                                              int* cnt) {
  if (threadIdx.x == 0) {
    // every slot is loaded (the array is whole in each item) and stored, so
    // the loads are in flight together; slots at or past n do not count
    int x[TS_MAX_K];
#pragma unroll
    for (int s = 0; s < TS_MAX_K; ++s) x[s] = item.child_tok[s];
    int k = 0;
#pragma unroll
    for (int s = 0; s < TS_MAX_K; ++s) {
      loc[k] = x[s];
      k += (s < n && x[s] >= y0 && x[s] < y1) ? 1 : 0;
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

// Bonus draw (Gumbel-max over a residual r): the key of token y is
// log2 r(y) - log2(-log2 u_y), u_y from word y & 3 of the Philox call
// c0 = y >> 2 (tag 3).  Keys are only compared within one item, so r may be
// any fixed positive multiple of the residual; each chunk keeps its best key
// (ties: smallest token) and its second-best value.
struct BonusTop {
  float best = kNegInf, second = kNegInf;
  int idx = 0x7FFFFFFF;
  __device__ __forceinline__ void add(float key, int y) {
    if (key > best) { second = best; best = key; idx = y; }
    else if (key > second) second = key;
  }
};
__device__ __forceinline__ void bonus_words(uint32_t (&w)[4], int b, uint32_t pc1, uint32_t pc2, uint32_t c3,
                                            const PhiloxKeys& keys) {
  uint32_t w0 = (uint32_t)b >> 2, w1 = pc1, w2 = pc2, w3 = c3;
  philox10(w0, w1, w2, w3, keys);
  w[0] = w0; w[1] = w1; w[2] = w2; w[3] = w3;
}
__device__ __forceinline__ float gumbel_neg(uint32_t w) {  // -log2(-log2 u)
  return -__builtin_amdgcn_logf(-__builtin_amdgcn_logf(word_to_uniform(w)));
}
// The workgroup's best key, token and second-best value into the item's chunk slot.
__device__ __forceinline__ void store_bonus(const VerifyPass& vp, int it, int ck, const BonusTop& bt, float* redv,
                                            int* redi) {
  float vb = bt.best;
  int id = bt.idx;
  block_argmax(vb, id, redv, redi);
  float s2 = (bt.idx == id) ? bt.second : bt.best;
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

// Pass A: per-chunk maxima and sums of the target and draft rows.  For an
// item without children (a leaf: the walk ends with a bonus draw from the
// target itself) it also takes the bonus keys, with r = 2^(t c - mt).

template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_pass_a_kernel(VerifyPass vp) {
  __shared__ float red[4];
  __shared__ double redd[4];
  __shared__ int redi[4];
  __shared__ int loc[TS_MAX_K];
  __shared__ int cnt;
  __shared__ VerifyItem sitem;
  static_assert(sizeof(VerifyItem) % 4 == 0 && sizeof(VerifyItem) / 4 <= kVerifyThreads, "item words");
  const int it = blockIdx.x / vp.nchunks, ck = blockIdx.x % vp.nchunks;
  if (it >= vp.nitems) return;
  // the item from the host's pinned buffer; chunk 0 also stages it for the
  // level's later kernels
  if (threadIdx.x < (int)(sizeof(VerifyItem) / 4)) {
    const int32_t w = reinterpret_cast<const int32_t*>(vp.items_host + it)[threadIdx.x];
    reinterpret_cast<int32_t*>(&sitem)[threadIdx.x] = w;
    if (ck == 0) reinterpret_cast<int32_t*>(vp.items_w + it)[threadIdx.x] = w;
  }
  __syncthreads();
  const VerifyItem& item = sitem;
  const int y0 = ck * vp.chunk, y1 = min(vp.V, y0 + vp.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)item.request * vp.cap + item.node) * vp.V;
  const float* zrow = item.m > 0 ? vp.zbuf + (size_t)item.zrow * vp.V : nullptr;
  const int nloc = item.m > 0 ? chunk_children(item, item.m, y0, y1, loc, &cnt) : 0;
  const bool vec = vector_rows<TT>(vp);
  // one sweep: running maxima, and sums relative to them (rescaled when a
  // maximum rises); the draft sum leaves the children out, its maximum does not
  float mt = kNegInf, mz = kNegInf, st = 0.0f, snc = 0.0f;
  const bool leaf = item.m == 0;  // uniform over the workgroup
  if (leaf) {
    const uint32_t pc1 = (uint32_t)item.path, pc2 = (uint32_t)(item.path >> 32);
    const uint32_t c3 = counter_word3(item.request, item.depth, 3u);
    BonusTop bt;
    sweep_chunk(trow, zrow, y0, y1, vec, [&](int b, const float(&tq)[4], const float(&zq)[4], int nv) {
      uint32_t w[4];
      bonus_words(w, b, pc1, pc2, c3, vp.keys);
      float qt = kNegInf;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < nv) qt = fmaxf(qt, tq[e] * vp.c);
      if (qt > mt) {
        if (st > 0.0f) st *= exp2_fast(mt - qt);
        mt = qt;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < nv) {
          st += exp2_fast(tq[e] * vp.c - mt);
          bt.add(tq[e] * vp.c + gumbel_neg(w[e]), b + e);
        }
      }
    });
    store_bonus(vp, it, ck, bt, red, redi);
  } else {
  sweep_chunk(trow, zrow, y0, y1, vec, [&](int b, const float(&tq)[4], const float(&zq)[4], int nv) {
    float qt = kNegInf, qz = kNegInf;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e < nv) {
        qt = fmaxf(qt, tq[e] * vp.c);
        if (zrow) qz = fmaxf(qz, zq[e] * vp.c);
      }
    }
    if (qt > mt) {
      if (st > 0.0f) st *= exp2_fast(mt - qt);
      mt = qt;
    }
    if (qz > mz) {
      if (snc > 0.0f) snc *= exp2_fast(mz - qz);
      mz = qz;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e < nv) {
        st += exp2_fast(tq[e] * vp.c - mt);
        if (zrow && !(nloc && is_listed(b + e, loc, nloc))) snc += exp2_fast(zq[e] * vp.c - mz);
      }
    }
  });
  }
  // to the workgroup's maxima
  const float Mt = block_max(mt, red), Mz = block_max(mz, red);
  st = st > 0.0f ? st * exp2_fast(mt - Mt) : 0.0f;
  snc = snc > 0.0f ? snc * exp2_fast(mz - Mz) : 0.0f;
  mt = Mt;
  mz = Mz;
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

// Stage j: advances the item's record by one stage (the stage-1 launch also
// builds the constants); if child j is rejected, this workgroup adds its
// chunk's share of Z_j = sum max(alpha_j p - beta'_j qT, 0) over tokens not
// drawn up to j.  When j is the item's last child, that same residual (up to
// the factor 1 / Z_j) is the one the bonus token is drawn from, so the sweep
// also takes the bonus keys.  Chunk 0 stores the record for the next launch.
template <typename TT>
__global__ __launch_bounds__(kVerifyThreads) void verify_stage_kernel(VerifyPass vp, int j) {
  __shared__ VRec shr;
  __shared__ float shL[2];
  __shared__ double redd[4];
  __shared__ float redv[4];
  __shared__ int redi[4];
  __shared__ int loc[TS_MAX_K];
  __shared__ int cnt;
  __shared__ VerifyItem sitem;
  const int it = blockIdx.x / vp.nchunks, ck = blockIdx.x % vp.nchunks;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  constexpr int kItemWords = (int)(sizeof(VerifyItem) / 4);
  VRec rec;
  if (j == 1) {
    if (threadIdx.x < kItemWords)
      reinterpret_cast<int32_t*>(&sitem)[threadIdx.x] = reinterpret_cast<const int32_t*>(vp.items + it)[threadIdx.x];
    VConst C;
    if (threadIdx.x < 64) {
      C = verify_consts<TT>(vp, item, it);
      if (item.m == 0) {
        rec.alpha = 1.0f; rec.beta = 0.0f; rec.betap = 1.0f;
        rec.margin = __builtin_huge_valf();
        rec.status = kExhausted;
        rec.stage = 1;
      } else {
        rec = stage_test(C.lp[0], C.lq[0], C.lR[0], C.invR[0], C.lu[0], 1, 1.0f, 0.0f,
                         __builtin_huge_valf());
      }
      if (ck == 0 && threadIdx.x == 0) vp.consts[it] = C;
      if (threadIdx.x == 0) {
        shL[0] = C.Lt;
        shL[1] = C.Lz;
      }
    }
    rec = share(rec, &shr);
  } else {
    // Wave 0 issues every load of the scalar step before using any (one
    // round trip): a word of the item, the previous record, stage j - 1's Z
    // partials (at clamped indices, masked after), child j's constants and
    // the normalisers.  The empty asm consumes them all at one point, so
    // none of the loads is moved behind a use.
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      const int nc = vp.nchunks;
      constexpr int kZq = 4;  // partials per lane loaded up front (256 chunks)
      const int32_t iw = reinterpret_cast<const int32_t*>(vp.items + it)[min(lane, kItemWords - 1)];
      const VRec prev = vp.recs[(size_t)(j - 2) * vp.nitems + it];
      const double* zs = vp.zp + ((size_t)(j - 2) * vp.nitems + it) * nc;
      double zq[kZq];
#pragma unroll
      for (int q = 0; q < kZq; ++q) zq[q] = zs[min(lane + 64 * q, nc - 1)];
      const VConst& C = vp.consts[it];
      const VChild c = child_consts(C, j - 1);
      const float Lt = C.Lt, Lz = C.Lz;
      asm volatile("" ::"v"(iw), "v"(prev.alpha), "v"(prev.beta), "v"(prev.betap), "v"(prev.margin),
                   "v"(prev.status), "v"(prev.stage), "v"(zq[0]), "v"(zq[1]), "v"(zq[2]), "v"(zq[3]),
                   "v"(c.lp), "v"(c.lq), "v"(c.lR), "v"(c.invR), "v"(c.lu), "v"(Lt), "v"(Lz));
      if (lane < kItemWords) reinterpret_cast<int32_t*>(&sitem)[lane] = iw;
      // stage j - 1's total Z, in the order chunk k = lane, lane + 64, ...
      double Z = 0.0;
#pragma unroll
      for (int q = 0; q < kZq; ++q) Z += lane + 64 * q < nc ? zq[q] : 0.0;
      for (int k = lane + 64 * kZq; k < nc; k += 64) Z += zs[k];
      Z = wave_sum_f64(Z);
      if (lane == 0) {
        shL[0] = Lt;
        shL[1] = Lz;
      }
      const int m = __builtin_amdgcn_readlane(iw, (int)(offsetof(VerifyItem, m) / 4));  // the item's child count
      rec = verify_advance(prev, Z, c, m, j);
    }
    rec = share(rec, &shr);
  }
  if (ck == 0 && threadIdx.x == 0) vp.recs[(size_t)(j - 1) * vp.nitems + it] = rec;
  if (rec.status != kRejected || rec.stage != j) return;
  const int y0 = ck * vp.chunk, y1 = min(vp.V, y0 + vp.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)sitem.request * vp.cap + sitem.node) * vp.V;
  const float* zrow = vp.zbuf + (size_t)sitem.zrow * vp.V;
  const int nloc = chunk_children(sitem, j, y0, y1, loc, &cnt);
  const float Lt = shL[0], Lz = shL[1];
  const bool vec = vector_rows<TT>(vp);
  float acc = 0.0f;
  if (j == sitem.m) {  // the last child: the sweep also takes the bonus keys
    const uint32_t pc1 = (uint32_t)sitem.path, pc2 = (uint32_t)(sitem.path >> 32);
    const uint32_t c3 = counter_word3(sitem.request, sitem.depth, 3u);
    BonusTop bt;
    sweep_chunk(trow, zrow, y0, y1, vec, [&](int b, const float(&tq)[4], const float(&zq)[4], int nv) {
      uint32_t w[4];
      bonus_words(w, b, pc1, pc2, c3, vp.keys);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < nv && !(nloc && is_listed(b + e, loc, nloc))) {
          const float p = exp2_fast(tq[e] * vp.c - Lt);
          const float q = exp2_fast(zq[e] * vp.c - Lz);
          const float r = rec.alpha * p - rec.betap * q;
          if (r > 0.0f) {
            acc += r;
            bt.add(__builtin_amdgcn_logf(r) + gumbel_neg(w[e]), b + e);
          }
        }
      }
    });
    store_bonus(vp, it, ck, bt, redv, redi);
  } else {
    sweep_chunk(trow, zrow, y0, y1, vec, [&](int b, const float(&tq)[4], const float(&zq)[4], int nv) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < nv && !(nloc && is_listed(b + e, loc, nloc))) {
          const float p = exp2_fast(tq[e] * vp.c - Lt);
          const float q = exp2_fast(zq[e] * vp.c - Lz);
          acc += fmaxf(rec.alpha * p - rec.betap * q, 0.0f);
        }
      }
    });
  }
  const double z = block_sum_f64((double)acc, redd);
  if (threadIdx.x == 0) vp.zp[((size_t)(j - 1) * vp.nitems + it) * vp.nchunks + ck] = z;
}

// Final record of an item after the last stage launch (stage J): a pending
// rejection at J is folded into the residual.
// Every item has at most J children, so the fold never tests a child.
__device__ __forceinline__ VRec verify_final(const VerifyPass& vp, const VerifyItem& item, int it, int J) {
  const VRec prev = vp.recs[(size_t)(J - 1) * vp.nitems + it];
  const double Z = stage_z(vp, it, J);
  return verify_advance(prev, Z, VChild{}, item.m, J + 1);
}

// An item's result from its final record and, when no child was accepted,
// the nc chunk bests of the bonus keys, bp_at(k) for chunk k (one whole wave).
template <typename BonusAt>
__device__ VerifyResult verify_result(const VRec& v, int nc, BonusAt&& bp_at) {
  const int lane = threadIdx.x & 63;
  VerifyResult r;
  r.accepted = v.status == kAccepted ? v.stage : 0;
  r.bonus = -1;
  r.margin = v.margin;
  r.leaf_bonus = 0;
  if (v.status != kAccepted) {
    float best = kNegInf, second = kNegInf;
    int idx = 0x7FFFFFFF;
    for (int k = lane; k < nc; k += 64) {
      const VBonusPart b = bp_at(k);
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
  return r;
}

// Resolve: one wave per item writes the accepted stage, or the bonus token.
template <typename TT>
__global__ __launch_bounds__(64) void verify_resolve_kernel(VerifyPass vp, int J) {
  const int it = blockIdx.x;
  if (it >= vp.nitems) return;
  const VerifyItem& item = vp.items[it];
  const VRec v = verify_final(vp, item, it, J);
  const VBonusPart* bp = vp.bp + (size_t)it * vp.nchunks;
  const VerifyResult r = verify_result(v, vp.nchunks, [&](int k) { return bp[k]; });
  // pinned host memory, read by the host after it synchronises the stream
  if (threadIdx.x == 0) vp.results[it] = r;
}

}  // namespace ts
