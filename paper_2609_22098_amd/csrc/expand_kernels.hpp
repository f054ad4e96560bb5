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
//     one step; per (parent, chunk) the kernel keeps the kTopRuns best run
//     keys (the maximum with the run index in its low bits) and the best key
//     of the other runs.
// Pass 2 (expand_merge, in merge_kernels.hpp) merges the per-chunk partials
// in a fixed order and finds the exact top-k: with L = the k-th largest
// recorded run key, lowered by the keys' slack, every top-k token lies in a
// recorded run whose key is >= L, or in a chunk whose other runs reach L
// (then the whole chunk is rescanned).  Those runs are recomputed with the same MFMA
// sequence as pass 1 (so the recomputed z are bit-identical, which the
// kernel checks), and the exact top-k is taken by (value desc, id asc).
//
// Sequential draws (the residual-proposal draws of §3.3 taken one after
// another) replace the Gumbel keys by one number per (parent, 64-token block):
// the base-2 log of the block's q_T mass.  The merge then makes each draw by
// picking a 4096-token segment, a block in it and a token in it in proportion
// to the remaining mass, recomputing only the chosen block.
#pragma once
#include <type_traits>

#include "device_common.hpp"

namespace ts {

constexpr int kTopRuns = 4;  // best runs recorded per (parent, chunk)

// Per-(parent, chunk) run summaries: m is [P][S][kTopRuns] run keys, rest is [P][S].
struct RunSummaryPtr {
  float* m;
  float* rest;
};

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
  float hr;       // headroom of the streaming pass's lazily raised reference, in logit units:
                  // 60 / max(log2(e), cT), so that no term of a sum exceeds 2^60
  int need_T;     // T > 0 and T != 1: keep a separate sum for log-sum-exp of z/T
  PhiloxKeys keys;
  float* part_m;   // [P][S] running max of z
  float* part_s0;  // [P][S] sum exp(z - m)
  float* part_sT;  // [P][S] sum exp((z - m) / T)
  RunSummaryPtr zs;  // per (parent, chunk): the two best runs of z and the rest
  RunSummaryPtr gs;  // the same for the Gumbel keys (Gumbel draws)
  float* blk;      // [P][blk_ld]: base-2 log of the q_T mass of each 64-token block (sequential
                   // draws); rows padded to whole 64-byte lines
  int nblk;        // ceil(V / 64)
  int blk_ld;      // row stride of blk: nblk rounded up to a multiple of 16
  float* z_out;    // optional [P][V]: the logits themselves (verification recompute)
  const int* P_dev;  // optional: the parent count in device memory (device-resident
                     // tree waves); the grid and P are then an upper bound
};

// Parents of a launch: P, or the count the device holds (<= P).
template <typename Params>
__device__ __forceinline__ int launch_parents(const Params& p) {
  return p.P_dev ? min(*p.P_dev, p.P) : p.P;
}

// Sampling modes of a launch: greedy (T = 0), Gumbel-top-k draws, sequential draws.
// The LDS streaming kernel also takes kModeNeedT in its mode (T != 1: a second
// sum for log-sum-exp of z / T), so that both sums are computed together.
enum : int { kModeGreedy = 0, kModeGumbel = 1, kModeSeq = 2, kModeNeedT = 4 };
constexpr int kSegTokens = 4096;  // tokens per segment of the sequential draws
constexpr int kBlkTokens = 64;    // tokens per block


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

// The 16 logits U[row][t .. t+16) one lane needs for one parent in a step,
// kept in their storage format until the accumulator is seeded.  Tokens >= V
// read as -inf.  U is streamed once, so its loads are non-temporal.
template <typename TE>
struct URun;

template <>
struct URun<uint16_t> {
  uint32_t w[8];
  __device__ __forceinline__ void load(const uint16_t* row, int t) {
    const u32x4* p = reinterpret_cast<const u32x4*>(row + t);
    const u32x4 a = __builtin_nontemporal_load(p);
    const u32x4 b = __builtin_nontemporal_load(p + 1);
    w[0] = a[0]; w[1] = a[1]; w[2] = a[2]; w[3] = a[3];
    w[4] = b[0]; w[5] = b[1]; w[6] = b[2]; w[7] = b[3];
  }
  // Tokens at or past V read as bf16 -inf (0xFF80).  Every load reads a
  // clamped index and the tail is masked after, so the loads are in flight
  // together.
  __device__ __forceinline__ void load_masked(const uint16_t* row, int t, int V) {
    uint32_t raw[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) raw[i] = row[min(t + i, V - 1)];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t m0 = opaque_mask(t + 2 * i < V), m1 = opaque_mask(t + 2 * i + 1 < V);
      const uint32_t lo = (raw[2 * i] & m0) | (0xFF80u & ~m0);
      const uint32_t hi = (raw[2 * i + 1] & m1) | (0xFF80u & ~m1);
      w[i] = lo | (hi << 16);
    }
  }
  __device__ __forceinline__ float get(int i) const {
    return (i & 1) ? __uint_as_float(w[i >> 1] & 0xFFFF0000u) : __uint_as_float(w[i >> 1] << 16);
  }
};

template <>
struct URun<float> {
  float f[16];
  __device__ __forceinline__ void load(const float* row, int t) {
    const f32x4* p = reinterpret_cast<const f32x4*>(row + t);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 v = __builtin_nontemporal_load(p + i);
      f[4 * i] = v[0]; f[4 * i + 1] = v[1]; f[4 * i + 2] = v[2]; f[4 * i + 3] = v[3];
    }
  }
  __device__ __forceinline__ void load_masked(const float* row, int t, int V) {
    float raw[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) raw[i] = row[min(t + i, V - 1)];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t m = opaque_mask(t + i < V);
      f[i] = __uint_as_float((__float_as_uint(raw[i]) & m) | (0xFF800000u & ~m));
    }
  }
  __device__ __forceinline__ float get(int i) const { return f[i]; }
};

// A run's maximum is recorded as a key that carries the run index (step * 4
// + lane group within the chunk, < 256) in its 8 low bits: the top lists then
// keep the index without selects.  The value is first clamped to finite
// values (an infinity with low bits set would be a NaN).  In the order of
// the float bit patterns a key lies within kRunSlack / 2 units of the
// clamped maximum, so the merge's threshold tests allow kRunSlack.
constexpr int kRunSlack = 512;
__device__ __forceinline__ float run_key(float v, int run) {
  const float c = __builtin_amdgcn_fmed3f(v, -3.40282347e38f, 3.40282347e38f);
  return __uint_as_float((__float_as_uint(c) & ~0xFFu) | (uint32_t)run);
}
__device__ __forceinline__ int run_of(float key) { return (int)(__float_as_uint(key) & 0xFFu); }
// v lowered by n units in the order of the float bit patterns (v is -inf or
// a finite key); a result at or below -FLT_MAX, the lowest key, is -inf.
__device__ __forceinline__ float key_lowered(float v, int n) {
  if (v == kNegInf) return kNegInf;
  const uint32_t b = __float_as_uint(v);
  const int o = (b & 0x80000000u) ? -(int)(b & 0x7FFFFFFFu) : (int)b;
  const int lo = o - n;
  if (lo <= -0x7F7FFFFF) return kNegInf;
  return lo < 0 ? __uint_as_float(0x80000000u | (uint32_t)(-lo)) : __uint_as_float((uint32_t)lo);
}

// Summary of a set of runs for one key: the kTopRuns largest run keys
// (sorted, larger first; keys of different runs never tie; empty entries are
// -inf) and the largest key of every other run.
struct RunTop {
  float m[kTopRuns];
  float rest;
};

// (value desc, index asc): the order of the exact top-k lists
__device__ __forceinline__ bool run_before(float v, int r, float w, int s) {
  return v > w || (v == w && r < s);
}

__device__ __forceinline__ void top_init(RunTop& t) {
#pragma unroll
  for (int i = 0; i < kTopRuns; ++i) t.m[i] = kNegInf;
  t.rest = kNegInf;
}

// Add one run key.  With the list sorted (m[0] >= .. >= m[3] >= rest), the
// new i-th entry is the median of m[i-1], m[i] and v, and the new rest that
// of m[3], rest and v.
__device__ __forceinline__ void top_add(RunTop& t, float v) {
  static_assert(kTopRuns == 4, "unrolled for four entries");
  t.rest = __builtin_amdgcn_fmed3f(t.m[3], t.rest, v);
#pragma unroll
  for (int i = kTopRuns - 1; i >= 1; --i) t.m[i] = __builtin_amdgcn_fmed3f(t.m[i - 1], t.m[i], v);
  t.m[0] = max2_med3(t.m[0], v);
}

// Merge two summaries of disjoint run sets (symmetric in its arguments):
// the top kTopRuns of the union by a bitonic split, then a bitonic sort.
__device__ __forceinline__ void top_combine(RunTop& a, const RunTop& b) {
  float c[kTopRuns];
  float rest = fmaxf(a.rest, b.rest);
#pragma unroll
  for (int k = 0; k < kTopRuns; ++k) {
    const float x = a.m[k], y = b.m[kTopRuns - 1 - k];
    c[k] = fmaxf(x, y);
    rest = fmaxf(rest, fminf(x, y));
  }
  auto cs = [](float& u, float& w) {
    const float hi = fmaxf(u, w), lo = fminf(u, w);
    u = hi;
    w = lo;
  };
  cs(c[0], c[2]);
  cs(c[1], c[3]);
  cs(c[0], c[1]);
  cs(c[2], c[3]);
#pragma unroll
  for (int k = 0; k < kTopRuns; ++k) a.m[k] = c[k];
  a.rest = rest;
}

__device__ __forceinline__ RunTop top_shfl_xor(const RunTop& t, int o) {
  RunTop u;
#pragma unroll
  for (int k = 0; k < kTopRuns; ++k) u.m[k] = __shfl_xor(t.m[k], o, 64);
  u.rest = __shfl_xor(t.rest, o, 64);
  return u;
}

__device__ __forceinline__ void top_store(const RunSummaryPtr& d, size_t o, const RunTop& t) {
#pragma unroll
  for (int k = 0; k < kTopRuns; ++k) d.m[o * kTopRuns + k] = t.m[k];
  d.rest[o] = t.rest;
}

// ---------------------------------------------------------------- pass 1

// Base-2 log of the q_T mass of this step's 64-token block for the lane's
// parent: a is the lane's run sum relative to 2^ml; the four lane groups of a
// parent (lanes n, n+16, n+32, n+48) hold the block's four runs.
// sum over j of 2^(v[j] * c - ref), as four interleaved partial sums
// (short dependency chains), combined in a fixed order.
__device__ __forceinline__ float sum16_exp2(const float (&v)[16], float c, float ref) {
  float a[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) a[q] = exp2_fast(__builtin_fmaf(v[q], c, -ref));
#pragma unroll
  for (int j = 4; j < 16; ++j) a[j & 3] += exp2_fast(__builtin_fmaf(v[j], c, -ref));
  return (a[0] + a[1]) + (a[2] + a[3]);
}

// The two sums of one run (scales c0, c1; references r0, r1) interleaved:
// eight independent chains, each summed in the order of sum16_exp2.
__device__ __forceinline__ void sum16_exp2_x2(const float (&v)[16], float c0, float r0, float c1, float r1,
                                              float& s0, float& s1) {
  float a[4], b[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a[q] = exp2_fast(__builtin_fmaf(v[q], c0, -r0));
    b[q] = exp2_fast(__builtin_fmaf(v[q], c1, -r1));
  }
#pragma unroll
  for (int j = 4; j < 16; ++j) {
    a[j & 3] += exp2_fast(__builtin_fmaf(v[j], c0, -r0));
    b[j & 3] += exp2_fast(__builtin_fmaf(v[j], c1, -r1));
  }
  s0 = (a[0] + a[1]) + (a[2] + a[3]);
  s1 = (b[0] + b[1]) + (b[2] + b[3]);
}

// a: this lane's run sum relative to 2^ref (ref finite); the run holding
// the block's largest ref has a >= 1 unless the whole block is masked.
__device__ __forceinline__ float block_log_mass(float a, float ref) {
  const float m = cross_row_max(ref);
  const float s = cross_row_sum(a * exp2_fast(ref - m));
  return s > 0.0f ? m + __builtin_amdgcn_logf(s) : kNegInf;
}

// Block-table stores of the streaming pass.  Blocks are grouped in windows of
// 16 (one 64-byte line of a parent's row); lane group g keeps blocks 4g..4g+3
// of the current window in registers, and at the window's end (or the chunk's)
// the four lane groups of a parent store the line as four 16-byte pieces.  A
// window cut by a chunk boundary stores only its own blocks, one by one.
struct BlkWindow {
  float h[4];
  __device__ __forceinline__ void put(int bi, int g, float lb) {
    const bool mine = g == ((bi >> 2) & 3);
#pragma unroll
    for (int q = 0; q < 4; ++q) h[q] = (mine && q == (bi & 3)) ? lb : h[q];
  }
  // bi: the block just put; bfirst, blast: the chunk's first and last block
  __device__ __forceinline__ void flush(float* row, int bi, int bfirst, int blast, int g) const {
    if ((bi & 15) != 15 && bi != blast) return;
    const int wb = bi & ~15;
    float* dst = row + wb + 4 * g;
    if (wb >= bfirst && (bi & 15) == 15) {
      *reinterpret_cast<f32x4*>(dst) = f32x4{h[0], h[1], h[2], h[3]};
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int b = wb + 4 * g + q;
        if (b >= bfirst && b <= bi) dst[q] = h[q];
      }
    }
  }
};

template <typename TE, int KS, int NB, int MODE, bool STORE_Z>
__global__ __launch_bounds__(256) void expand_eval_kernel(const ExpandParams p) {
  typedef Frag<TE> F;
  typedef typename F::type FT;
  const int lane = threadIdx.x & 63;
  constexpr bool SAMPLE = MODE != kModeGreedy;  // T > 0: lse of z/T and K draws
  constexpr bool GUMBEL = MODE == kModeGumbel;
  constexpr bool SEQ = MODE == kModeSeq;
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
  const int P = launch_parents(p);
  const int pb = pgroup * p.wpg + wv;
  if (pb * 16 * NB >= P) return;

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
    if (pidx[nb] < P) {
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

  float m0[NB], s0[NB], sT[NB];
  RunTop zt[NB], gt[NB];
  BlkWindow bw[NB];
  const int bfirst = chunk * (p.Vc >> 6);
  const int blast = (min(chunk * p.Vc + p.Vc, V) - 1) >> 6;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m0[nb] = kNegInf; s0[nb] = 0.0f; sT[nb] = 0.0f;
    top_init(zt[nb]);
    top_init(gt[nb]);
  }

  // One 64-token step: 16 tokens per lane group, each lane owns one parent
  // per block.  u holds this step's U values (prefetched one step ahead).
  // A: row n of M-block bb is token t0 + (n/4)*16 + bb*4 + n%4, so that the
  // C layout gives lane group g the 16 contiguous tokens t0 + g*16 + [0,16).
  auto load_a = [&](FT (&afrag)[4][KS], int t0) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const int tA = min(t0 + (n >> 2) * 16 + bb * 4 + (n & 3), V - 1);
      const TE* wrow = W2 + (size_t)tA * r;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) afrag[bb][kk] = F::load(wrow, kk * F::kPerStep, g);
    }
  };

  auto do_step = [&](const URun<TE> (&u)[NB], const FT (&afrag)[4][KS], int t0, int step) {
    f32x4 acc[4][NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
        acc[bb][nb] = f32x4{u[nb].get(bb * 4), u[nb].get(bb * 4 + 1), u[nb].get(bb * 4 + 2),
                            u[nb].get(bb * 4 + 3)};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[bb][nb] = F::mma(afrag[bb][kk], bfrag[nb][kk], acc[bb][nb]);

    const int run = step * 4 + g;
    const int tl = t0 + g * 16;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float v[16];
#pragma unroll
      for (int bb = 0; bb < 4; ++bb)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[bb * 4 + e] = acc[bb][nb][e];
      if constexpr (STORE_Z) {
        if (pidx[nb] < P) {
          float* zo = p.z_out + (size_t)pidx[nb] * V;
          if ((V & 3) == 0 && tl + 16 <= V) {  // 16-byte aligned: four vector stores
#pragma unroll
            for (int j = 0; j < 16; j += 4)
              *reinterpret_cast<f32x4*>(zo + tl + j) = f32x4{v[j], v[j + 1], v[j + 2], v[j + 3]};
          } else {
#pragma unroll
            for (int j = 0; j < 16; ++j)
              if (tl + j < V) zo[tl + j] = v[j];
          }
        }
      }
      float bm = max2_med3(v[0], v[1]);
#pragma unroll
      for (int j = 2; j < 16; ++j) bm = fmaxf(bm, v[j]);
      // run sums are taken relative to the run's own maximum (a run far below
      // the running maximum keeps its mass), then folded into the running
      // sums, which are relative to the running maximum: of the two terms the
      // one with the lower reference is scaled down (one exponential)
      const float m0c = fmaxf(m0[nb], -1e30f);
      const float bref = fmaxf(bm, -1e30f);
      const bool run_high = bref > m0c;
      const float gap = -__builtin_fabsf(m0c - bref);
      const float bl = bref * kLog2e;
      float a0 = sum16_exp2(v, kLog2e, bl);
      const float f0 = exp2_fast(gap * kLog2e);
      s0[nb] = run_high ? __builtin_fmaf(s0[nb], f0, a0) : __builtin_fmaf(a0, f0, s0[nb]);
      const float blT = bref * p.cT;
      float aT = 0.0f;
      if (SAMPLE && p.need_T) {
        aT = sum16_exp2(v, p.cT, blT);
        const float fT = exp2_fast(gap * p.cT);
        sT[nb] = run_high ? __builtin_fmaf(sT[nb], fT, aT) : __builtin_fmaf(aT, fT, sT[nb]);
      }
      m0[nb] = fmaxf(m0[nb], bm);
      top_add(zt[nb], run_key(bm, run));
      if constexpr (SEQ) {
        const float lb = p.need_T ? block_log_mass(aT, blT) : block_log_mass(a0, bl);
        const int bi = t0 >> 6;
        bw[nb].put(bi, g, lb);
        if (pidx[nb] < P) bw[nb].flush(p.blk + (size_t)pidx[nb] * p.blk_ld, bi, bfirst, blast, g);
      }
      if constexpr (GUMBEL) {
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
        top_add(gt[nb], run_key(gm, run));
      }
    }
  };

  auto load_u = [&](URun<TE> (&u)[NB], int t0) {
    if (vec_ok && t0 + 64 <= V) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) u[nb].load(urow[nb], t0 + g * 16);
    } else {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) u[nb].load_masked(urow[nb], t0 + g * 16, V);
    }
  };

  // Steps alternate between two buffers of U values and W2 fragments: the
  // next step's loads are in flight while the current step computes.
  const int tbeg = chunk * p.Vc;
  const int tend = min(tbeg + p.Vc, V);
  URun<TE> ua[NB], ub[NB];
  FT aa[4][KS], ab[4][KS];
  int t0 = tbeg, step = 0;
  load_u(ua, t0);
  load_a(aa, t0);
  for (;;) {
    const bool more1 = t0 + 64 < tend;
    if (more1) { load_u(ub, t0 + 64); load_a(ab, t0 + 64); }
    do_step(ua, aa, t0, step);
    if (!more1) break;
    t0 += 64; ++step;
    const bool more2 = t0 + 64 < tend;
    if (more2) { load_u(ua, t0 + 64); load_a(aa, t0 + 64); }
    do_step(ub, ab, t0, step);
    if (!more2) break;
    t0 += 64; ++step;
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
    RunTop zc = zt[nb], gc = gt[nb];
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      top_combine(zc, top_shfl_xor(zc, o));
      if constexpr (GUMBEL) top_combine(gc, top_shfl_xor(gc, o));
    }
    if (g == 0 && pidx[nb] < P) {
      const size_t o = (size_t)pidx[nb] * p.S + chunk;
      p.part_m[o] = M;
      p.part_s0[o] = s;
      if (p.part_sT) p.part_sT[o] = st;
      top_store(p.zs, o, zc);
      if constexpr (GUMBEL) top_store(p.gs, o, gc);
    }
  }
}

// Streaming pass, bf16, staged through LDS.  The four waves of a workgroup
// work on one chunk with different parent blocks.  Each 64-token step needs a
// W2 tile (64 rows of r bf16, shared by the four waves) and one U tile per
// wave; both are brought in with direct global->LDS loads one step ahead, in
// two buffers used alternately, so no registers hold prefetched data.  The W2
// tile is laid out in 16-byte pieces in the exact order the A fragments are
// read (piece (bb*KS + kk)*64 + lane), so every fragment read is one
// conflict-free ds_read_b128.  Requires V % 8 == 0 and chunks of a multiple of
// 256 tokens.
//
// Per (parent, token) the pass spends an FMA, an exp2 and an add on each sum
// it keeps; everything else is amortised over a lane's 16-token run or over
// four steps:
//   - the log-sum-exp sums are taken against a reference per parent that is
//     raised only when a run maximum passes it by more than the headroom (one
//     wave-wide vote per run; the raise itself is rare), instead of rescaling
//     at every run;
//   - with sequential draws, the q_T sum of each run is taken against the
//     run's own maximum instead (the draws need every block's mass, however
//     small next to the parent's largest), the block masses are combined over
//     four steps at a time with one exchange across the lane groups and
//     stored a 64-byte line per 16 blocks; the merge takes log-sum-exp of
//     z / T from the block masses, so no separate sum of z / T is kept.
__device__ __forceinline__ void lds_dma16(const void* src, u32x4* dst_wave_base) {
  typedef __attribute__((address_space(3))) void* lds_ptr;
  __builtin_amdgcn_global_load_lds(src, (lds_ptr)dst_wave_base, 16, 0, 0);
}
// Buffer resource word 3 of a raw (unswizzled, byte-addressed) buffer on gfx9.
constexpr int kRawBufferFlags = 0x00020000;
// 16 bytes per lane from a raw buffer at voff + soff into LDS at
// dst_wave_base + 16 * lane; out-of-range bytes read as zero.  Issued as
// inline assembly: the kernel orders its LDS tiles with explicit vmcnt waits,
// and the compiler, which does not see these as writes to LDS, inserts no
// wait of its own before the LDS reads of other tiles (with the builtin, in a
// loop it cannot tell which tile a queued load writes, and waits for all of
// them).  The kernel's waits must cover every read of the tile.  M0 holds the
// wave's LDS destination (no other instruction of the kernel uses M0); rsrc
// is the buffer resource as four scalar words.
__device__ __forceinline__ void lds_buf16_asm(u32x4 rsrc, uint32_t voff, int soff, const u32x4* dst_wave_base) {
  typedef __attribute__((address_space(3))) const void* lds_ptr;
  const uint32_t m0 = (uint32_t)(uintptr_t)(lds_ptr)dst_wave_base;
  asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :: "v"(voff), "s"(rsrc), "s"(soff), "s"(m0) : "memory", "m0");
}
// Raw buffer resource of n bytes at base, as four scalar words.
__device__ __forceinline__ u32x4 raw_rsrc(const void* base, uint32_t n) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xFFFFu, n, (uint32_t)kRawBufferFlags};
}

// s_waitcnt immediate that waits until at most n vector memory operations of
// the wave are outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt in 6:4, lgkmcnt in 11:8; the counters not waited on hold their
// maxima).  Vector memory operations complete in issue order.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// A mass held as x * 2^r (x >= 0, r finite): the sum of two, against the
// larger reference.  Equal references keep the order x1 + x2.
struct Mass {
  float x, r;
};
__device__ __forceinline__ Mass mass_add(Mass a, Mass b) {
  const float e = exp2_fast(-__builtin_fabsf(a.r - b.r));
  const bool ahi = a.r >= b.r;
  return Mass{ahi ? __builtin_fmaf(b.x, e, a.x) : __builtin_fmaf(a.x, e, b.x), ahi ? a.r : b.r};
}
__device__ __forceinline__ Mass swap16_pair(Mass& a, Mass& b) {  // see quad_block_masses
  const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(a.x), __float_as_uint(b.x), false, false);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a.r), __float_as_uint(b.r), false, false);
  return mass_add(Mass{__uint_as_float(x[0]), __uint_as_float(r[0])}, Mass{__uint_as_float(x[1]), __uint_as_float(r[1])});
}

// Block masses of a quad of steps.  m_j is this lane's 16-token share of the
// quad's block j (step j), against its own run maximum; the four lane groups
// of a parent (lanes n, n+16, n+32, n+48) hold the four quarters of every
// block.  Lane group g gets the mass of block g: one swap across row pairs
// halves the values a lane holds (rows 0 and 2 keep blocks 0 and 2, rows 1
// and 3 blocks 1 and 3), a swap across the halves of the wave finishes the
// sums.  Every block is combined in the same order, (q0 + q1) + (q2 + q3)
// over its quarters, and each partial sum is taken against the larger of
// its references, so no block underflows however far below the parent's
// largest logit it lies.
__device__ __forceinline__ Mass quad_block_masses(Mass m0, Mass m1, Mass m2, Mass m3) {
  const Mass A = swap16_pair(m0, m1);  // row g: block (g & 1), its row pair
  const Mass B = swap16_pair(m2, m3);  // row g: block 2 + (g & 1)
  const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(A.x), __float_as_uint(B.x), false, false);
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(A.r), __float_as_uint(B.r), false, false);
  return mass_add(Mass{__uint_as_float(x[0]), __uint_as_float(r[0])}, Mass{__uint_as_float(x[1]), __uint_as_float(r[1])});
}

// 4 x 4 transpose across lane groups: in, lane group g holds h[k] = block
// 4k + g of a 16-block window; out, it holds h[k] = block 4g + k.
__device__ __forceinline__ void window_transpose(float (&h)[4]) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(h[0]), __float_as_uint(h[1]), false, false);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(h[2]), __float_as_uint(h[3]), false, false);
  const auto c = __builtin_amdgcn_permlane32_swap(a[0], b[0], false, false);
  const auto d = __builtin_amdgcn_permlane32_swap(a[1], b[1], false, false);
  h[0] = __uint_as_float(c[0]);
  h[1] = __uint_as_float(d[0]);
  h[2] = __uint_as_float(c[1]);
  h[3] = __uint_as_float(d[1]);
}

// At rank <= 64 with two parent blocks per wave the kernel must fit three
// waves per SIMD (168 VGPRs), four with eight-wave workgroups (128 VGPRs): a
// few registers more halve the waves that hide its latencies.  WPG waves per
// workgroup share each W2 tile (loaded by the first four).
template <int KS, int NB, int MODE, int WPG>
__global__ __launch_bounds__(64 * WPG) __attribute__((amdgpu_waves_per_eu(KS <= 2 && NB == 2 ? (WPG == 8 ? 4 : 3) : 1)))
void expand_eval_lds_kernel(const ExpandParams p) {
  typedef Frag<uint16_t> F;
  typedef typename F::type FT;
  constexpr int kW = 4 * KS * 64;  // 16-byte pieces of one W2 tile
  constexpr int kU = NB * 2 * 64;  // 16-byte pieces of one wave's U tile
  // W2 tiles (from L2, mostly: every parent group reads them) one step
  // ahead, in two buffers; U tiles (from HBM: each is read once) two steps
  // ahead, in two buffers per wave: step t reads U buffer t % 2 into
  // registers, then queues step t + 2's pieces into it
  __shared__ __attribute__((aligned(16))) u32x4 w0[kW];
  __shared__ __attribute__((aligned(16))) u32x4 w1[kW];
  __shared__ __attribute__((aligned(16))) u32x4 ub0[WPG * kU];
  __shared__ __attribute__((aligned(16))) u32x4 ub1[WPG * kU];
  const int lane = threadIdx.x & 63;
  constexpr int BASE = MODE & 3;
  constexpr bool SAMPLE = BASE != kModeGreedy;  // T > 0: lse of z/T and K draws
  constexpr bool GUMBEL = BASE == kModeGumbel;
  constexpr bool SEQ = BASE == kModeSeq;
  constexpr bool NT = SAMPLE && (MODE & kModeNeedT) != 0;  // T != 1: a separate sum for z/T
  // the wave index is uniform: kept scalar, the LDS destinations of the
  // direct loads need no per-step readfirstlane
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15;
  const int g = lane >> 4;

  const int b = blockIdx.x;
  const int kx = b >> 3;
  const int chunk = (b & 7) + 8 * (kx / p.n_pgroups);
  const int pgroup = kx % p.n_pgroups;
  if (chunk >= p.S) return;  // uniform over the workgroup
  const int P = launch_parents(p);
  if (pgroup * WPG * 16 * NB >= P) return;  // uniform: no parent in this workgroup
  const int pb = pgroup * WPG + wv;
  const bool active = pb * 16 * NB < P;  // idle waves still load W2 and join the barriers

  const uint16_t* U = static_cast<const uint16_t*>(p.U);
  const uint16_t* E = static_cast<const uint16_t*>(p.E);
  const uint16_t* W2 = static_cast<const uint16_t*>(p.W2);
  const int V = p.V, r = p.r;

  // Byte offsets of this lane's U pieces from the step's first token of row
  // 0: its parent's row plus its lane group's 16 tokens (U is under 4 GiB).
  // A step's loads add them to a scalar base.
  uint32_t uoff[NB];
  FT bfrag[NB][KS];
  uint32_t pc1[NB], pc2[NB], pc3[NB];
  int pidx[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    pidx[nb] = (pb * NB + nb) * 16 + n;
    int tok = 0, dep = 0, req = 0;
    uint64_t path = 0;
    if (active && pidx[nb] < P) {
      const ts_parent par = p.parents[pidx[nb]];
      if (par.token >= 0 && par.token < V && par.depth >= 0 && par.depth < p.D &&
          par.request >= 0 && par.request < p.R) {
        tok = par.token; dep = par.depth; req = par.request; path = par.path;
      }
    }
    uoff[nb] = ((uint32_t)(req * p.D + dep) * (uint32_t)V + (uint32_t)g * 16u) * 2u;
    const uint16_t* erow = E + (size_t)tok * r;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) bfrag[nb][kk] = F::load(erow, kk * F::kPerStep, g);
    pc1[nb] = (uint32_t)path;
    pc2[nb] = (uint32_t)(path >> 32);
    pc3[nb] = counter_word3(req, dep, 1u);
  }
  // the E fragments are in registers before the first tile load is queued:
  // the compiler does not count the queued loads (inline assembly), so its
  // own waits for these registers inside the loop would otherwise stall on
  // them
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) asm volatile("" ::"v"(bfrag[nb][kk]));

  // Per parent (shared by its four lane groups): the reference of the sums,
  // in logit units, the level that triggers a raise, and the FMA offsets
  // reference * log2(e) and reference * cT.  It starts below every finite
  // logit, so the first run with a finite maximum raises it before any term
  // is summed.
  float ref[NB], lim[NB], off0[NB], offT[NB], s0[NB], sT[NB];
  RunTop zt[NB], gt[NB];
  // sequential draws: the q_T sum of the lane's run j of the open quad, as
  // qx * 2^qr with qr the run maximum times c (c = cT, or log2(e) at T = 1)
  float qx[NB][4], qr[NB][4];
  float hw[NB][4];  // sequential draws: the open window's block log-masses, hw[k] = block 4k + g
  // sequential draws keep no sum of z / T, and at T = 1 no sum at all: the
  // merge takes those log-sum-exps from the block masses
  constexpr bool SUM0 = !SEQ || NT;
  constexpr bool SUMT = NT && !SEQ;
  const float cX = NT ? p.cT : kLog2e;  // scale of the block masses
  const int bfirst = chunk * (p.Vc >> 6);
  const int blast = (min(chunk * p.Vc + p.Vc, V) - 1) >> 6;
  // the vocabulary's last chunk may write its last window whole (the row is padded to 16 blocks)
  const int bstore = blast == p.nblk - 1 ? p.blk_ld - 1 : blast;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    ref[nb] = -1e30f; lim[nb] = -1e30f;
    off0[nb] = -1e30f * kLog2e; offT[nb] = -1e30f * p.cT;
    s0[nb] = 0.0f; sT[nb] = 0.0f;
    top_init(zt[nb]);
    top_init(gt[nb]);
#pragma unroll
    for (int k = 0; k < 4; ++k) { qx[nb][k] = 0.0f; qr[nb][k] = -1e30f; hw[nb][k] = kNegInf; }
  }

  // W2: this wave loads pieces (wv*KS + j)*64 + lane of the tile: row
  // (n >> 2)*16 + bb*4 + (n & 3) of the step, 16 bytes at k = kk*32 + g*8.
  // U: tokens t0 + g*16 + 8h + [0, 8) of this lane's parent in block nb.
  // Both are raw buffer loads: a per-lane byte offset fixed for the whole
  // chunk plus a scalar offset per step, so a step's loads cost no vector
  // instruction.  Rows past the vocabulary read as zeros (W2, U's last row)
  // or as the next row's first tokens (U): the last step masks them.
  uint32_t woff[KS];
#pragma unroll
  for (int j = 0; j < KS; ++j) {
    const int bb = ((wv & 3) * KS + j) / KS, kk = ((wv & 3) * KS + j) % KS;
    woff[j] = (uint32_t)((((n >> 2) * 16 + bb * 4 + (n & 3)) * r + kk * 32 + g * 8) * 2);
  }
  const u32x4 wsrc = raw_rsrc(W2, (uint32_t)V * r * 2);
  const u32x4 usrc = raw_rsrc(U, (uint32_t)p.R * p.D * V * 2);
  auto issue_w = [&](u32x4* wb, int t0) {
    if (wv < 4) {
#pragma unroll
      for (int j = 0; j < KS; ++j) lds_buf16_asm(wsrc, woff[j], t0 * r * 2, wb + (wv * KS + j) * 64);
    }
  };
  typedef u32x4 UPieces[NB][2];
  auto issue_u = [&](u32x4* ub, int t0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h) lds_buf16_asm(usrc, uoff[nb], t0 * 2 + 16 * h, ub + wv * kU + (nb * 2 + h) * 64);
  };

  // The vocabulary's last step when V % 64 != 0: with V % 8 == 0 every 8-token
  // piece of U lies wholly before V or wholly at or past it; the latter (their
  // loads read the next row, or zeros past the array) become bf16 -inf, so
  // those logits are -inf.
  auto mask_tail = [&](UPieces& pu, int t0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (t0 + g * 16 + 8 * h >= V) {
          const uint32_t ninf2 = 0xFF80FF80u;
          pu[nb][h] = u32x4{ninf2, ninf2, ninf2, ninf2};
        }
  };

  // Raise the reference of every parent of block nb to the largest of its
  // lane groups' references and run maxima (all of them agree afterwards);
  // the sums and the open quad's shares are scaled to it.
  auto raise = [&](int nb, float bm) {
    const float nr = fmaxf(cross_row_max(max2_med3(ref[nb], bm)), -1e30f);
    const float d = ref[nb] - nr;
    s0[nb] *= exp2_fast(d * kLog2e);
    if constexpr (SUMT) sT[nb] *= exp2_fast(d * p.cT);
    ref[nb] = nr;
    lim[nb] = nr + p.hr;
    off0[nb] = nr * kLog2e;
    offT[nb] = nr * p.cT;
  };

  // z of the parents of block nb for one step: the accumulator starts at U
  // (seed), then takes the rank-r product on the matrix core (logits).
  auto seed = [&](const UPieces& pu, int nb, f32x4 (&acc)[4]) {
    const u32x4 pa = pu[nb][0];
    const u32x4 pc = pu[nb][1];
    URun<uint16_t> u;
    u.w[0] = pa[0]; u.w[1] = pa[1]; u.w[2] = pa[2]; u.w[3] = pa[3];
    u.w[4] = pc[0]; u.w[5] = pc[1]; u.w[6] = pc[2]; u.w[7] = pc[3];
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
      acc[bb] = f32x4{u.get(bb * 4), u.get(bb * 4 + 1), u.get(bb * 4 + 2), u.get(bb * 4 + 3)};
  };
  // the step's W2 fragments (shared by the NB blocks), read from LDS at once
  typedef FT AFrags[4][KS];
  auto read_a = [&](const u32x4* wb, AFrags& af) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) af[bb][kk] = __builtin_bit_cast(FT, wb[(bb * KS + kk) * 64 + lane]);
  };
  auto logits = [&](const AFrags& af, int nb, f32x4 (&acc)[4]) {
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[bb] = F::mma(af[bb][kk], bfrag[nb][kk], acc[bb]);
  };

  // The run's sums (a0 of z against the parent's reference; ax of z times c
  // against the run maximum for the block masses, or aT of z / T against the
  // parent's reference); returns the run maximum.
  auto run_sums = [&](int nb, const f32x4 (&acc)[4], float (&v)[16], float& a0, float& ax, float& br) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[bb * 4 + e] = acc[bb][e];
    float bm = max2_med3(v[0], v[1]);
#pragma unroll
    for (int i = 2; i < 16; ++i) bm = fmaxf(bm, v[i]);
    if constexpr (SUM0)
      if (__builtin_expect(__ballot(bm > lim[nb]) != 0, 0)) raise(nb, bm);
    a0 = 0.0f; ax = 0.0f; br = 0.0f;
    if constexpr (SEQ) {
      // the run's q_T sum against its own maximum (finite: an all -inf run sums to 0)
      br = max2_med3(bm, -1e30f) * cX;
      if constexpr (NT)
        sum16_exp2_x2(v, kLog2e, off0[nb], p.cT, br, a0, ax);
      else
        ax = sum16_exp2(v, kLog2e, br);
    } else {
      if constexpr (SUMT)
        sum16_exp2_x2(v, kLog2e, off0[nb], p.cT, offT[nb], a0, ax);
      else
        a0 = sum16_exp2(v, kLog2e, off0[nb]);
    }
    return bm;
  };

  // One 64-token step; j is the step's place in its quad (known at compile time).
  auto compute = [&](const AFrags& af, f32x4 (&accs)[NB][4], int t0, int step, auto jtag) {
    constexpr int j = decltype(jtag)::value;
    const int tl = t0 + g * 16;
    const int run = step * 4 + g;
    auto epilogue = [&](int nb, f32x4 (&acc)[4]) {
      float v[16], a0, ax, br;
      const float bm = run_sums(nb, acc, v, a0, ax, br);
      if constexpr (SUM0) s0[nb] += a0;
      if constexpr (SUMT) sT[nb] += ax;
      if constexpr (SEQ) {
        qx[nb][j] = ax;
        qr[nb][j] = br;
      }
      top_add(zt[nb], run_key(bm, run));
      if constexpr (GUMBEL) {
        float gm = kNegInf;
        const uint32_t cbase = (uint32_t)tl >> 2;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint32_t c0 = cbase + i, c1 = pc1[nb], c2 = pc2[nb], c3 = pc3[nb];
          philox10(c0, c1, c2, c3, p.keys);
          const uint32_t w[4] = {c0, c1, c2, c3};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float key = gumbel_key2(v[i * 4 + q], p.cT, w[q]);  // -inf past the vocabulary
            gm = fmaxf(gm, key);
          }
        }
        top_add(gt[nb], run_key(gm, run));
      }
    };
    // block by block: block nb + 1's products run on the matrix core while
    // block nb's epilogue runs on the vector ALUs
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      logits(af, nb, accs[nb]);
      epilogue(nb, accs[nb]);
    }
  };

  // End of a quad (or of the chunk inside one): the quad's block totals as
  // base-2 log-masses into the open window; at the window's last quad, or the
  // chunk's, the window goes to the block table, a 16-byte piece per lane
  // group (single entries where the window reaches outside the chunk).
  auto end_quad = [&](int qb) {  // qb: the quad's first block (a multiple of 4)
    const int k = (qb >> 2) & 3;
    const int wfirst = qb & ~15;
    const bool flush = k == 3 || qb + 4 > blast;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const Mass tot = quad_block_masses(Mass{qx[nb][0], qr[nb][0]}, Mass{qx[nb][1], qr[nb][1]},
                                         Mass{qx[nb][2], qr[nb][2]}, Mass{qx[nb][3], qr[nb][3]});
      const float lb = tot.x > 0.0f ? tot.r + __builtin_amdgcn_logf(tot.x) : kNegInf;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        hw[nb][i] = k == i ? lb : hw[nb][i];
        qx[nb][i] = 0.0f;
        qr[nb][i] = -1e30f;
      }
      if (flush) {
        window_transpose(hw[nb]);
        if (pidx[nb] < P) {
          float* dst = p.blk + (size_t)pidx[nb] * p.blk_ld + wfirst + 4 * g;
          if (wfirst >= bfirst && wfirst + 15 <= bstore) {
            *reinterpret_cast<f32x4*>(dst) = f32x4{hw[nb][0], hw[nb][1], hw[nb][2], hw[nb][3]};
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int bi = wfirst + 4 * g + i;
              if (bi >= bfirst && bi <= bstore) dst[i] = hw[nb][i];
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) hw[nb][i] = kNegInf;
      }
    }
  };

  const int tbeg = chunk * p.Vc;
  const int tend = min(tbeg + p.Vc, V);
  // Issue priority falls as the wave walks its chunk (3 in the first quarter,
  // then 2, 1, 0), so that on a SIMD the waves that are behind are served
  // first.  With equal priorities the oldest wave wins every arbitration:
  // the waves of a SIMD finish one after another and the last one runs
  // alone, with nothing to hide its latencies.
  const int nsteps = (tend - tbeg + 63) >> 6;
  int prio_next = (nsteps + 3) >> 2, prio_q = 0;
  __builtin_amdgcn_s_setprio(3);
  auto lower_priority = [&](int done) {
    if (done < prio_next) return;
    ++prio_q;
    prio_next = (nsteps * (prio_q + 1) + 3) >> 2;
    if (prio_q == 1) __builtin_amdgcn_s_setprio(2);
    else if (prio_q == 2) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
  };

  // One step: wait for its tiles, queue the next ones, compute.  Returns
  // false after the chunk's last step.  Step j of a quad reads the buffers
  // j & 1.  A U load has two steps' compute to land (one step ahead it
  // waited out most of its latency under load).
  int t0 = tbeg, step = 0;
  auto do_step = [&](auto jtag) -> bool {
    constexpr int j = decltype(jtag)::value;
    u32x4* wcur = (j & 1) ? w1 : w0;
    u32x4* wnext = (j & 1) ? w0 : w1;
    u32x4* ucur = (j & 1) ? ub1 : ub0;
    const bool more = t0 + 64 < tend;
    const bool more2 = t0 + 128 < tend;
    // this step's tiles are in LDS once at most the next step's U pieces
    // (2 NB per lane, queued last) are outstanding; stores issued since only
    // make the wait longer
    if (more && active)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * NB));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    // the waits above order the tiles' arrival; a barrier with the usual
    // workgroup fences would wait for every queued load as well
    asm volatile("s_barrier" ::: "memory");
    lower_priority(step);
    if (more) issue_w(wnext, t0 + 64);
    if (active) {
      UPieces pu;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int h = 0; h < 2; ++h) pu[nb][h] = ucur[wv * kU + (nb * 2 + h) * 64 + lane];
      AFrags af;
      read_a(wcur, af);
      // the pieces are in registers before the loads two steps ahead overwrite
      // them (and no LDS read of the step comes after those loads)
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
      if (more2) issue_u(ucur, t0 + 128);
      if (t0 + 64 > V) mask_tail(pu, t0);
      f32x4 accs[NB][4];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) seed(pu, nb, accs[nb]);
      compute(af, accs, t0, step, jtag);
      if (SEQ && (j == 3 || !more)) end_quad((t0 >> 6) & ~3);
    }
    if (!more) return false;
    // the step position is the same in every lane: keep it scalar
    t0 = __builtin_amdgcn_readfirstlane(t0 + 64);
    step = __builtin_amdgcn_readfirstlane(step + 1);
    return true;
  };
  issue_w(w0, t0);
  if (active) {
    issue_u(ub0, t0);
    if (t0 + 64 < tend) issue_u(ub1, t0 + 64);
  }
  for (;;) {
    if (!do_step(std::integral_constant<int, 0>{})) break;
    if (!do_step(std::integral_constant<int, 1>{})) break;
    if (!do_step(std::integral_constant<int, 2>{})) break;
    if (!do_step(std::integral_constant<int, 3>{})) break;
  }
  if (!active) return;

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    // the four lane groups of a parent share its reference: their sums add
    float s = s0[nb];
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    float st = 0.0f;
    if constexpr (SUMT) {
      st = sT[nb];
      st += __shfl_xor(st, 16, 64);
      st += __shfl_xor(st, 32, 64);
    }
    RunTop zc = zt[nb], gc = gt[nb];
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      top_combine(zc, top_shfl_xor(zc, o));
      if constexpr (GUMBEL) top_combine(gc, top_shfl_xor(gc, o));
    }
    if (g == 0 && pidx[nb] < P) {
      const size_t o = (size_t)pidx[nb] * p.S + chunk;
      if constexpr (SUM0) {
        p.part_m[o] = ref[nb];
        p.part_s0[o] = s;
      }
      if constexpr (SUMT) p.part_sT[o] = st;
      top_store(p.zs, o, zc);
      if constexpr (GUMBEL) top_store(p.gs, o, gc);
    }
  }
}

}  // namespace ts
