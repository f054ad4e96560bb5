// Kernels of the parent-conditioned expansion (ts_expand).
//
// For a frontier parent p (token x, depth d, request q) the drafter logits are
//   z[y] = U[q][d][y] + <E[x], W2[y]>                     (§1 Eq. 1; §3.2 item 1)
// and one node evaluation needs log-sum-exp of z and of z/T, the top-k of z
// (greedy children, and the pre-draw bound at T > 0) and, at T > 0, the top-k
// of the Gumbel-perturbed keys z/T + G (k draws without replacement from
// q_T, the residual-proposal draws of §3.3).
//
// Pass 1 (expand_eval) streams the vocabulary once.  The P x r x V contraction
// runs on MFMA (16x16x32 bf16 or 16x16x4 f32): rows are 16 tokens, columns are
// 16 parents, K is the rank r.  The accumulator starts from the U values, so
// the MFMA output is z itself.  Each lane then owns one parent and 16
// contiguous tokens per 64-token step and keeps:
//   - an online log-sum-exp (running max and scaled sums for z and z/T);
//   - "run" maxima for exact top-k: a run is the 16 tokens one lane sees in
//     one step; per (parent, chunk) the kernel keeps the best run maximum,
//     its run index and the best maximum of the other runs.
// Pass 2 (expand_merge) merges the per-chunk partials in a fixed order and
// finds the exact top-k: with L = the k-th largest chunk maximum, every
// top-k token lies in a chunk whose maximum is >= L, inside that chunk's
// best run unless the chunk's second-best run maximum is also >= L.  Only
// those runs are recomputed, with the same MFMA sequence as pass 1 (so the
// recomputed z are bit-identical, which the kernel checks), and the exact
// top-k is taken by (value desc, id asc).
#pragma once

#include "device_common.hpp"

namespace ts {

struct ExpandParams {
  const void* U;
  const void* E;
  const void* W2;
  int R, D, V, r;
  const ts_parent* parents;
  int P;
  int Vc;         // tokens per chunk, multiple of 64
  int S;          // number of chunks
  int n_pblocks;  // parent blocks of 16 * NB parents (one wave each)
  int wpg;        // waves (parent blocks) per workgroup
  int n_pgroups;  // workgroups per chunk
  float cT;       // log2(e) / T  (T > 0)
  int need_T;     // T > 0 and T != 1: keep a separate sum for log-sum-exp of z/T
  PhiloxKeys keys;
  float* part_m;   // [P][S] running max of z
  float* part_s0;  // [P][S] sum exp(z - m)
  float* part_sT;  // [P][S] sum exp((z - m) / T)
  float* zb1;      // [P][S] best run maximum of z
  float* zb2;      // [P][S] best maximum of the other runs
  int* zrun;       // [P][S] run index of zb1 (step * 4 + lane group)
  float* gb1;      // same three for the Gumbel keys (T > 0)
  float* gb2;
  int* grun;
  float* z_out;    // optional [P][V]: the logits themselves (verification recompute)
};

struct MergeParams {
  const void* U;
  const void* E;
  const void* W2;
  int R, D, V, r;
  const ts_parent* parents;
  int P;
  int Vc, S;
  int K;
  float T, cT;
  int need_T;
  float calib_a, calib_b;
  PhiloxKeys keys;
  const float* part_m;
  const float* part_s0;
  const float* part_sT;
  const float* zb1;
  const float* zb2;
  const int* zrun;
  const float* gb1;
  const float* gb2;
  const int* grun;
  ts_expand_out out;
};

// ---------------------------------------------------------------- fragments

template <typename TE>
struct Frag;

// bf16: 16x16x32 MFMA; a lane holds 8 consecutive K values of one row/column.
template <>
struct Frag<uint16_t> {
  typedef bf16x8 type;
  static constexpr int kPerStep = 32;
  __device__ static __forceinline__ type load(const uint16_t* row, int k0, int kb) {
    const uint4 v = *reinterpret_cast<const uint4*>(row + k0 + kb * 8);
    return __builtin_bit_cast(type, v);
  }
  __device__ static __forceinline__ type zero() {
    uint4 v = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(type, v);
  }
  __device__ static __forceinline__ f32x4 mma(type a, type b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }
};

// f32: 16x16x4 MFMA; a lane holds one K value of one row/column.
template <>
struct Frag<float> {
  typedef float type;
  static constexpr int kPerStep = 4;
  __device__ static __forceinline__ type load(const float* row, int k0, int kb) {
    return row[k0 + kb];
  }
  __device__ static __forceinline__ type zero() { return 0.0f; }
  __device__ static __forceinline__ f32x4 mma(type a, type b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ float to_f32(float v) { return v; }
};

// 16 consecutive logits U[row][t .. t+16) as fp32; tokens >= V read as -inf.
template <typename TE>
__device__ __forceinline__ void load_u16(const TE* row, int t, int V, bool vec_ok, float (&u)[16]) {
  if (vec_ok && t + 16 <= V) {
    if constexpr (sizeof(TE) == 2) {
      const uint4* p = reinterpret_cast<const uint4*>(row + t);
      const uint4 a = p[0], b = p[1];
      const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        u[2 * i] = __uint_as_float(w[i] << 16);
        u[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      }
    } else {
      const float4* p = reinterpret_cast<const float4*>(row + t);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 v = p[i];
        u[4 * i] = v.x; u[4 * i + 1] = v.y; u[4 * i + 2] = v.z; u[4 * i + 3] = v.w;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      u[i] = (t + i < V) ? Frag<TE>::to_f32(row[t + i]) : kNegInf;
  }
}

// Order of (max, second, run) bucket summaries: larger max wins, ties go to
// the smaller run index; the loser's max joins the second-best.
__device__ __forceinline__ void bucket_combine(float& b1, float& b2, int& run, float o1, float o2,
                                               int orun) {
  if (o1 > b1 || (o1 == b1 && orun < run)) {
    b2 = fmaxf(o2, b1);
    b1 = o1;
    run = orun;
  } else {
    b2 = fmaxf(b2, o1);
  }
}

// ---------------------------------------------------------------- pass 1

template <typename TE, int KS, int NB, bool SAMPLE>
__global__ __launch_bounds__(256) void expand_eval_kernel(const ExpandParams p) {
  typedef Frag<TE> F;
  typedef typename F::type FT;
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int n = lane & 15;  // parent column / token row inside a 16x16 tile
  const int g = lane >> 4;  // lane group: K sub-block for A/B, row block for C

  // Workgroups are dispatched round-robin over the 8 XCDs (block b on XCD
  // b % 8).  Chunks are dealt to XCDs the same way so that every workgroup
  // working on a chunk shares one XCD's L2 for that chunk's W2 rows.
  const int b = blockIdx.x;
  const int kx = b >> 3;
  const int chunk = (b & 7) + 8 * (kx / p.n_pgroups);
  const int pgroup = kx % p.n_pgroups;
  if (chunk >= p.S) return;
  const int pb = pgroup * p.wpg + wv;
  if (pb >= p.n_pblocks) return;

  const TE* U = static_cast<const TE*>(p.U);
  const TE* E = static_cast<const TE*>(p.E);
  const TE* W2 = static_cast<const TE*>(p.W2);
  const int V = p.V, r = p.r;
  const bool vec_ok = (V % (16 / (int)sizeof(TE))) == 0;

  // Per-column parent state (this lane's parent in each of the NB blocks).
  const TE* urow[NB];
  FT bfrag[NB][KS];
  uint32_t pc1[NB], pc2[NB], pc3[NB];
  int pidx[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    pidx[nb] = (pb * NB + nb) * 16 + n;
    int tok = 0, dep = 0, req = 0;
    uint64_t path = 0;
    if (pidx[nb] < p.P) {
      const ts_parent par = p.parents[pidx[nb]];
      if (par.token >= 0 && par.token < V && par.depth >= 0 && par.depth < p.D &&
          par.request >= 0 && par.request < p.R) {
        tok = par.token; dep = par.depth; req = par.request; path = par.path;
      }
    }
    urow[nb] = U + ((size_t)req * p.D + dep) * (size_t)V;
    const TE* erow = E + (size_t)tok * r;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) bfrag[nb][kk] = F::load(erow, kk * F::kPerStep, g);
    pc1[nb] = (uint32_t)path;
    pc2[nb] = (uint32_t)(path >> 32);
    pc3[nb] = counter_word3(req, dep, 1u);
  }

  float m0[NB], s0[NB], sT[NB], zb1[NB], zb2[NB], gb1[NB], gb2[NB];
  int zr[NB], gr[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m0[nb] = kNegInf; s0[nb] = 0.0f; sT[nb] = 0.0f;
    zb1[nb] = kNegInf; zb2[nb] = kNegInf; zr[nb] = -1;
    gb1[nb] = kNegInf; gb2[nb] = kNegInf; gr[nb] = -1;
  }

  const int tbeg = chunk * p.Vc;
  const int tend = min(tbeg + p.Vc, V);
  int step = 0;
  for (int t0 = tbeg; t0 < tend; t0 += 64, ++step) {
    // A: row n of M-block bb is token t0 + (n/4)*16 + bb*4 + n%4, so that the
    // C layout gives lane group g the 16 contiguous tokens t0 + g*16 + [0,16).
    FT afrag[4][KS];
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const int tA = min(t0 + (n >> 2) * 16 + bb * 4 + (n & 3), V - 1);
      const TE* wrow = W2 + (size_t)tA * r;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) afrag[bb][kk] = F::load(wrow, kk * F::kPerStep, g);
    }
    f32x4 acc[4][NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float u[16];
      load_u16<TE>(urow[nb], t0 + g * 16, V, vec_ok, u);
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
        acc[bb][nb] = f32x4{u[bb * 4], u[bb * 4 + 1], u[bb * 4 + 2], u[bb * 4 + 3]};
    }
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[bb][nb] = F::mma(afrag[bb][kk], bfrag[nb][kk], acc[bb][nb]);

    const int run = step * 4 + g;
    const int tl = t0 + g * 16;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float v[16];
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[bb * 4 + e] = acc[bb][nb][e];
      if (p.z_out != nullptr && pidx[nb] < p.P) {
        float* zo = p.z_out + (size_t)pidx[nb] * V;
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (tl + j < V) zo[tl + j] = v[j];
      }
      float bm = v[0];
#pragma unroll
      for (int j = 1; j < 16; ++j) bm = fmaxf(bm, v[j]);
      const float mn = fmaxf(m0[nb], bm);
      const float mref = fmaxf(mn, -1e30f);
      const float ml = mref * kLog2e;
      float a0 = 0.0f;
#pragma unroll
      for (int j = 0; j < 16; ++j) a0 += exp2_fast(__builtin_fmaf(v[j], kLog2e, -ml));
      s0[nb] = __builtin_fmaf(s0[nb], exp2_fast(__builtin_fmaf(m0[nb], kLog2e, -ml)), a0);
      if (SAMPLE && p.need_T) {
        const float mlT = mref * p.cT;
        float aT = 0.0f;
#pragma unroll
        for (int j = 0; j < 16; ++j) aT += exp2_fast(__builtin_fmaf(v[j], p.cT, -mlT));
        sT[nb] = __builtin_fmaf(sT[nb], exp2_fast(__builtin_fmaf(m0[nb], p.cT, -mlT)), aT);
      }
      m0[nb] = mn;
      if (bm > zb1[nb]) {
        zb2[nb] = zb1[nb];
        zb1[nb] = bm;
        zr[nb] = run;
      } else {
        zb2[nb] = fmaxf(zb2[nb], bm);
      }
      if constexpr (SAMPLE) {
        float gm = kNegInf;
        const uint32_t cbase = (uint32_t)tl >> 2;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint32_t c0 = cbase + i, c1 = pc1[nb], c2 = pc2[nb], c3 = pc3[nb];
          philox10(c0, c1, c2, c3, p.keys);
          const uint32_t w[4] = {c0, c1, c2, c3};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int j = i * 4 + q;
            const float key = (tl + j < V) ? gumbel_key2(v[j], p.cT, w[q]) : kNegInf;
            gm = fmaxf(gm, key);
          }
        }
        if (gm > gb1[nb]) {
          gb2[nb] = gb1[nb];
          gb1[nb] = gm;
          gr[nb] = run;
        } else {
          gb2[nb] = fmaxf(gb2[nb], gm);
        }
      }
    }
  }

  // Combine the four lane groups of each parent (lanes n, n+16, n+32, n+48).
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float M = m0[nb];
    M = fmaxf(M, __shfl_xor(M, 16, 64));
    M = fmaxf(M, __shfl_xor(M, 32, 64));
    const float Mref = fmaxf(M, -1e30f);
    float s = s0[nb] * exp2_fast(__builtin_fmaf(m0[nb], kLog2e, -Mref * kLog2e));
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    float st = 0.0f;
    if (SAMPLE && p.need_T) {
      st = sT[nb] * exp2_fast(__builtin_fmaf(m0[nb], p.cT, -Mref * p.cT));
      st += __shfl_xor(st, 16, 64);
      st += __shfl_xor(st, 32, 64);
    }
    float b1 = zb1[nb], b2 = zb2[nb];
    int rr = zr[nb];
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float o1 = __shfl_xor(b1, o, 64), o2 = __shfl_xor(b2, o, 64);
      const int orr = __shfl_xor(rr, o, 64);
      bucket_combine(b1, b2, rr, o1, o2, orr);
    }
    float h1 = gb1[nb], h2 = gb2[nb];
    int hr = gr[nb];
    if constexpr (SAMPLE) {
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float o1 = __shfl_xor(h1, o, 64), o2 = __shfl_xor(h2, o, 64);
        const int orr = __shfl_xor(hr, o, 64);
        bucket_combine(h1, h2, hr, o1, o2, orr);
      }
    }
    if (g == 0 && pidx[nb] < p.P) {
      const size_t o = (size_t)pidx[nb] * p.S + chunk;
      p.part_m[o] = M;
      p.part_s0[o] = s;
      if (p.part_sT) p.part_sT[o] = st;
      p.zb1[o] = b1;
      p.zb2[o] = b2;
      p.zrun[o] = rr;
      if constexpr (SAMPLE) {
        p.gb1[o] = h1;
        p.gb2[o] = h2;
        p.grun[o] = hr;
      }
    }
  }
}

// ---------------------------------------------------------------- pass 2

// Recompute the logits of 16 consecutive tokens [t, t+16) for one parent with
// the MFMA sequence of pass 1 (same operands in the same K positions, same
// accumulator start).  The parent sits in column 0; lanes 0, 16, 32, 48 get
// tokens t + g*4 + [0, 4).
template <typename TE, int KS>
__device__ __forceinline__ f32x4 recompute_run(const TE* W2, const TE* urow, int V, int r, int t,
                                               const typename Frag<TE>::type (&bcol)[KS]) {
  typedef Frag<TE> F;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, g = lane >> 4;
  const int tA = min(t + n, V - 1);
  const TE* wrow = W2 + (size_t)tA * r;
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if (n == 0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int tok = t + g * 4 + e;
      acc[e] = tok < V ? F::to_f32(urow[tok]) : kNegInf;
    }
  }
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) acc = F::mma(F::load(wrow, kk * F::kPerStep, g), bcol[kk], acc);
  return acc;
}

// Insert (v, id) into a list sorted by (value desc, id asc) holding at most K entries.
__device__ __forceinline__ void topk_insert(float* val, int* ids, float* aux, int& cnt, int K,
                                            float v, int id, float a) {
  if (cnt == K && !(v > val[K - 1] || (v == val[K - 1] && id < ids[K - 1]))) return;
  int pos = cnt < K ? cnt : K - 1;
  while (pos > 0 && (v > val[pos - 1] || (v == val[pos - 1] && id < ids[pos - 1]))) {
    val[pos] = val[pos - 1];
    ids[pos] = ids[pos - 1];
    aux[pos] = aux[pos - 1];
    --pos;
  }
  val[pos] = v;
  ids[pos] = id;
  aux[pos] = a;
  if (cnt < K) ++cnt;
}

struct MergeLds {
  float zval[TS_MAX_K];
  int zid[TS_MAX_K];
  float zaux[TS_MAX_K];
  float gval[TS_MAX_K];
  int gid[TS_MAX_K];
  float gz[TS_MAX_K];  // z of the drawn tokens
  float buf_z[16];
  float buf_g[16];
  int zcnt, gcnt;
};

// Select the chunks that can hold a top-K element of one key (z or Gumbel) and
// rescan their candidate runs; fills the sorted list in LDS (lane 0 inserts).
template <typename TE, int KS, bool GUMBEL>
__device__ int select_and_rescan(const MergeParams& p, const float* b1, const float* b2,
                                  const int* brun, size_t pbase, const TE* urow,
                                  const typename Frag<TE>::type (&bcol)[KS], uint32_t pc1,
                                  uint32_t pc2, uint32_t pc3, MergeLds& L, float* val, int* ids,
                                  float* aux, int& cnt_lds) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int S = p.S, K = p.K, V = p.V;
  // threshold: the K-th largest chunk maximum (ties by chunk index)
  uint32_t taken = 0u;  // bit i: chunk lane + 64 i already picked
  float thr = kNegInf;
  int picked = 0;
  for (; picked < K; ++picked) {
    float bv = kNegInf;
    int bc = 0x7FFFFFFF;
    for (int c = lane, i = 0; c < S; c += 64, ++i) {
      if (taken & (1u << i)) continue;
      const float v = b1[pbase + c];
      if (v > bv || (v == bv && c < bc)) { bv = v; bc = c; }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oc = __shfl_xor(bc, o, 64);
      if (ov > bv || (ov == bv && oc < bc)) { bv = ov; bc = oc; }
    }
    if (bc == 0x7FFFFFFF) break;
    if ((bc & 63) == lane) taken |= 1u << (bc >> 6);
    thr = bv;
  }
  if (picked < K) thr = kNegInf;  // fewer than K chunks: every token is a candidate

  if (lane == 0) cnt_lds = 0;
  int cnt = 0;  // lane 0's view of the list length
  int mismatches = 0;
  for (int c = 0; c < S; ++c) {
    const float cm = b1[pbase + c];
    if (!(cm >= thr)) continue;
    const bool whole = b2[pbase + c] >= thr;
    const int best = brun[pbase + c];
    const int cbeg = c * p.Vc;
    const int nruns = ((min(cbeg + p.Vc, V) - cbeg + 63) / 64) * 4;
    for (int ri = 0; ri < nruns; ++ri) {
      const int run = whole ? ri : best;
      if (!whole && ri > 0) break;
      const int t = cbeg + (run >> 2) * 64 + (run & 3) * 16;
      if (t >= V) continue;
      const f32x4 z4 = recompute_run<TE, KS>(static_cast<const TE*>(p.W2), urow, V, p.r, t, bcol);
      float k4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) k4[e] = z4[e];
      if constexpr (GUMBEL) {
        // lanes 0/16/32/48 hold tokens t + g*4 + [0,4): one Philox call each
        uint32_t c0 = (uint32_t)(t + g * 4) >> 2, c1 = pc1, c2 = pc2, c3 = pc3;
        philox10(c0, c1, c2, c3, p.keys);
        const uint32_t w[4] = {c0, c1, c2, c3};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          k4[e] = (t + g * 4 + e < V) ? gumbel_key2(z4[e], p.cT, w[e]) : kNegInf;
      }
      if ((lane & 15) == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          L.buf_z[g * 4 + e] = z4[e];
          L.buf_g[g * 4 + e] = k4[e];
        }
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      if (lane == 0) {
        float rm = kNegInf;
        for (int j = 0; j < 16; ++j) {
          const float kv = L.buf_g[j];
          rm = fmaxf(rm, kv);
          if (kv >= thr && t + j < V) topk_insert(val, ids, aux, cnt, K, kv, t + j, L.buf_z[j]);
        }
        if (run == best && rm != cm) ++mismatches;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
  if (lane == 0) cnt_lds = cnt;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  return mismatches;
}

template <typename TE, int KS, bool SAMPLE>
__global__ __launch_bounds__(256) void expand_merge_kernel(const MergeParams p) {
  typedef Frag<TE> F;
  typedef typename F::type FT;
  __shared__ MergeLds lds[4];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int pidx = blockIdx.x * 4 + wv;
  if (pidx >= p.P) return;
  MergeLds& L = lds[wv];
  const int K = p.K, V = p.V, S = p.S;
  const ts_parent par = p.parents[pidx];
  const bool ok = par.token >= 0 && par.token < V && par.depth >= 0 && par.depth < p.D &&
                  par.request >= 0 && par.request < p.R;
  const size_t ob = (size_t)pidx * K;
  if (!ok) {
    const float nan = __builtin_nanf("");
    if (lane < K) {
      p.out.child_token[ob + lane] = -1;
      p.out.child_log_q0[ob + lane] = nan;
      p.out.child_log_surv[ob + lane] = nan;
      p.out.slot_key[ob + lane] = nan;
      if (p.out.child_log_qT) p.out.child_log_qT[ob + lane] = nan;
      if (p.out.rank_token) p.out.rank_token[ob + lane] = -1;
      if (p.out.rank_log_q0) p.out.rank_log_q0[ob + lane] = nan;
    }
    if (lane == 0) {
      if (p.out.lse0) p.out.lse0[pidx] = nan;
      if (p.out.lseT) p.out.lseT[pidx] = nan;
      if (p.out.diag) p.out.diag[pidx] = 0;
    }
    return;
  }
  const size_t pbase = (size_t)pidx * S;

  // log-sum-exp over chunks: each lane folds its chunks in index order, then a fixed butterfly.
  float M = kNegInf;
  for (int c = lane; c < S; c += 64) M = fmaxf(M, p.part_m[pbase + c]);
  M = wave_max(M);
  const float Mref = fmaxf(M, -1e30f);
  float s = 0.0f, st = 0.0f;
  for (int c = lane; c < S; c += 64) {
    const float mc = p.part_m[pbase + c];
    s += p.part_s0[pbase + c] * exp2_fast(__builtin_fmaf(mc, kLog2e, -Mref * kLog2e));
    if (SAMPLE && p.need_T)
      st += p.part_sT[pbase + c] * exp2_fast(__builtin_fmaf(mc, p.cT, -Mref * p.cT));
  }
  s = wave_sum(s);
  st = wave_sum(st);
  const float lse0 = M + logf(s);
  float lseT = __builtin_nanf("");
  if (SAMPLE) lseT = p.need_T ? M / p.T + logf(st) : lse0;

  const TE* urow = static_cast<const TE*>(p.U) + ((size_t)par.request * p.D + par.depth) * (size_t)V;
  const TE* erow = static_cast<const TE*>(p.E) + (size_t)par.token * p.r;
  FT bcol[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) bcol[kk] = (n == 0) ? F::load(erow, kk * F::kPerStep, g) : F::zero();
  const uint32_t pc1 = (uint32_t)par.path, pc2 = (uint32_t)(par.path >> 32);
  const uint32_t pc3 = counter_word3(par.request, par.depth, 1u);

  int mism = select_and_rescan<TE, KS, false>(p, p.zb1, p.zb2, p.zrun, pbase, urow, bcol, pc1,
                                              pc2, pc3, L, L.zval, L.zid, L.zaux, L.zcnt);
  if constexpr (SAMPLE)
    mism += select_and_rescan<TE, KS, true>(p, p.gb1, p.gb2, p.grun, pbase, urow, bcol, pc1, pc2,
                                            pc3, L, L.gval, L.gid, L.gz, L.gcnt);

  // Child scoring: lane j handles slot j + 1 (Algorithm 1; §3.2 pre-draw bound; Eq. 3).
  if (lane < K) {
    const int j = lane;
    const float lsp = par.log_surv;
    const float a = p.calib_a, bb = p.calib_b;
    const float zpi = L.zval[j];
    if (p.out.rank_token) p.out.rank_token[ob + j] = L.zid[j];
    if (p.out.rank_log_q0) p.out.rank_log_q0[ob + j] = zpi - lse0;
    if constexpr (!SAMPLE) {
      const float lq0 = zpi - lse0;
      const float ls = lsp + log_phat(lq0, a, bb);
      p.out.child_token[ob + j] = L.zid[j];
      p.out.child_log_q0[ob + j] = lq0;
      p.out.child_log_surv[ob + j] = ls;
      p.out.slot_key[ob + j] = ls;
      if (p.out.child_log_qT) p.out.child_log_qT[ob + j] = __builtin_nanf("");
    } else {
      const int tok = L.gid[j];
      const float zc = L.gz[j];
      const float lq0 = zc - lse0;
      // bound: the first of the greedy order not drawn before j
      int bi = 0;
      for (; bi < K; ++bi) {
        bool used = false;
        for (int s2 = 0; s2 < j; ++s2) used |= (L.gid[s2] == L.zid[bi]);
        if (!used) break;
      }
      const float zb = L.zval[bi < K ? bi : K - 1];
      p.out.child_token[ob + j] = tok;
      p.out.child_log_q0[ob + j] = lq0;
      p.out.child_log_surv[ob + j] = lsp + log_phat(lq0, a, bb);
      p.out.slot_key[ob + j] = lsp + log_phat(zb - lse0, a, bb);
      if (p.out.child_log_qT) p.out.child_log_qT[ob + j] = zc / p.T - lseT;
    }
  }
  if (lane == 0) {
    if (p.out.lse0) p.out.lse0[pidx] = lse0;
    if (p.out.lseT) p.out.lseT[pidx] = lseT;
    if (p.out.diag) p.out.diag[pidx] = mism;
  }
}

}  // namespace ts
