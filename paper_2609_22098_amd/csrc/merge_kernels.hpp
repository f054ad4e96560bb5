// Pass 2 of the parent-conditioned expansion (ts_expand): merge of the
// per-chunk partials of pass 1, exact top-k, the sequential draws and child
// scoring.  The pass-1 kernels, the shared parameter blocks and the MFMA
// fragment helpers are in expand_kernels.hpp.
#pragma once
#include "expand_kernels.hpp"

namespace ts {

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
  RunSummaryPtr zs;
  RunSummaryPtr gs;
  float* blk;  // per-parent block table [P][blk_ld]; the draws update their own parent's rows
  int nblk, blk_ld;
  ts_expand_out out;
  const int* P_dev;  // optional device-held parent count (<= P), as in ExpandParams
};

// ---------------------------------------------------------------- pass 2

constexpr int kMaxChunks = 256;                              // chunks per parent
constexpr int kEntrySlots = kMaxChunks * kTopRuns / 64;      // recorded runs per lane
constexpr int kRestSlots = kMaxChunks / 64;                  // chunk rests per lane
constexpr int kBatch = 8;                                    // runs recomputed together
constexpr int kItemCap = 256;                                // candidate items per parent

struct MergeLds {
  float bz[kBatch][16];  // logits of a batch of recomputed runs
  float bk[kBatch][16];  // their keys (z, or the Gumbel keys)
  int item_t[kItemCap];  // run start token, or -(chunk+1) for a whole chunk
  int item_k[kItemCap];  // key kind: 0 = z, 1 = Gumbel
  float item_e[kItemCap];  // expected run key (NaN if unknown)
  uint32_t whole[kMaxChunks / 32];
};

// Sequential draws run on a wave of their own (the parent's second wave):
// its scratch, and the draws it hands to the scoring wave.
constexpr int kLdsSegs = 40;  // segments whose block table is kept in LDS (one per lane)
static_assert(kLdsSegs <= 64, "one segment per lane");
struct DrawLds {
  alignas(16) float seg_blk[kLdsSegs * 64];  // the parent's block table when V <= 40 * 4096
  int id[TS_MAX_K];              // draw j's token and logit at j - 1
  float z[TS_MAX_K];
  float lmass;                   // base-2 log of the parent's whole q_T mass (before the draws)
};

// Workgroup LDS of the merge: four parents of one wave each, or, for
// sequential draws, one parent of two waves.
template <bool SEQ>
struct MergeShared {
  MergeLds l[4];
};
template <>
struct MergeShared<true> {
  MergeLds l[1];
  DrawLds d;
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int wave_sum_int(int v) { return wave_sum_i32(v); }

// A sorted list of at most K (key, token, aux) entries kept in registers:
// lane j < cnt holds entry j; order: key desc, token asc.
struct RegList {
  float val;
  int id;
  float aux;
  int cnt;
};

__device__ __forceinline__ void reglist_init(RegList& l) {
  l.val = kNegInf; l.id = 0x7FFFFFFF; l.aux = 0.0f; l.cnt = 0;
}

// Insert a candidate (uniform across the wave).
__device__ __forceinline__ void reglist_insert(RegList& l, int K, float v, int id, float a) {
  const int lane = threadIdx.x & 63;
  // entry before the candidate: key desc, token asc (run_before, without
  // the short-circuit branches)
  const bool ahead = (lane < l.cnt) & ((l.val > v) | ((l.val == v) & (l.id < id)));
  const int pos = __popcll(__ballot(ahead));
  if (pos >= K) return;
  // the entries from pos on move up one lane (DPP wave_shr:1)
  const float pv = dpp_f32<0x138>(l.val);
  const int pid = dpp_i32<0x138>(l.id);
  const float pa = dpp_f32<0x138>(l.aux);
  const bool at = lane == pos;
  const bool up = (lane > pos) & (lane < K);
  l.val = at ? v : (up ? pv : l.val);
  l.id = at ? id : (up ? pid : l.id);
  l.aux = at ? a : (up ? pa : l.aux);
  l.cnt = min(l.cnt + 1, K);
}

// The accumulator seeds of a lane's four tokens tok0 + [0, 4): their U
// values, -inf at or past V.  Every load reads a clamped index inside the
// row and none sits under a condition, so all of a batch's loads are in
// flight together (a conditional load becomes a branch that waits for its
// own value); the tail select comes afterwards.
template <typename TE>
__device__ __forceinline__ void u_seeds(const TE* urow, int tok0, int V, float (&u)[4]) {
  TE raw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) raw[e] = urow[min(tok0 + e, V - 1)];
#pragma unroll
  for (int e = 0; e < 4; ++e) u[e] = tok0 + e < V ? Frag<TE>::to_f32(raw[e]) : kNegInf;
}
// The same four seeds with one vector load, for a group that starts at a
// multiple of 4 inside a row of V % 4 == 0 tokens (the row then starts 8-byte
// aligned for bf16, 16-byte for f32) and ends at or before V.
__device__ __forceinline__ void u_seeds4(const uint16_t* p, float (&u)[4]) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  u[0] = __uint_as_float(w.x << 16);
  u[1] = __uint_as_float(w.x & 0xFFFF0000u);
  u[2] = __uint_as_float(w.y << 16);
  u[3] = __uint_as_float(w.y & 0xFFFF0000u);
}
__device__ __forceinline__ void u_seeds4(const float* p, float (&u)[4]) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  u[0] = v.x;
  u[1] = v.y;
  u[2] = v.z;
  u[3] = v.w;
}

// Recompute up to kBatch runs of 16 tokens [t, t+16) for one parent with the
// MFMA sequence of pass 1 (same operands in the same K positions, same
// accumulator start), so the values are bit-identical to the streaming pass.
// The parent sits in column 0; lanes 0, 16, 32, 48 get tokens t + g*4 + [0,4).
// Runs of kind 1 also get their Gumbel keys.  All lanes then check the keys
// against the kind's threshold; candidates go into the kind's list.  A run
// whose expected maximum is known counts a mismatch if the recomputed one differs.
template <typename TE, int KS, bool SAMPLE, int PARTS>
__device__ __forceinline__ void rescan_batch(const MergeParams& p, const TE* urow,
                                             const typename Frag<TE>::type (&bcol)[KS],
                                             uint32_t pc1, uint32_t pc2, uint32_t pc3,
                                             const int (&t)[kBatch], const int (&kind)[kBatch],
                                             const float (&expect)[kBatch], int nrun,
                                             const float (&thr)[2], MergeLds& L, RegList& zl,
                                             RegList& gl, int& mism) {
  typedef Frag<TE> F;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, g = lane >> 4;
  const int V = p.V;
  const TE* W2 = static_cast<const TE*>(p.W2);
  f32x4 acc[kBatch];
  const uint32_t col0 = opaque_mask(n == 0);
  // whole aligned runs take vector seed loads (uniform over the wave)
  bool vec = (V & 3) == 0;
#pragma unroll
  for (int b = 0; b < kBatch; ++b) {
    const int tb = b < nrun ? t[b] : 0;
    vec = vec && (tb & 3) == 0 && tb + 16 <= V;
  }
  // in PARTS parts: all loads of a part first (one round trip), then its MFMAs
  constexpr int kHalf = kBatch / PARTS;
#pragma unroll
  for (int h = 0; h < PARTS; ++h) {
    typename F::type wf[kHalf][KS];
    float u[kHalf][4];
#pragma unroll
    for (int i = 0; i < kHalf; ++i) {
      const int b = h * kHalf + i;
      const int tb = b < nrun ? t[b] : 0;
      const TE* wrow = W2 + (size_t)min(tb + n, V - 1) * p.r;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) wf[i][kk] = F::load(wrow, kk * F::kPerStep, g);
    }
    if (vec) {
#pragma unroll
      for (int i = 0; i < kHalf; ++i) {
        const int b = h * kHalf + i;
        u_seeds4(urow + (b < nrun ? t[b] : 0) + g * 4, u[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < kHalf; ++i) {
        const int b = h * kHalf + i;
        u_seeds(urow, (b < nrun ? t[b] : 0) + g * 4, V, u[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < kHalf; ++i) {
      const int b = h * kHalf + i;
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[b][e] = keep_or_zero(u[i][e], col0);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) acc[b] = F::mma(wf[i][kk], bcol[kk], acc[b]);
    }
  }
  if (n == 0) {
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int tb = b < nrun ? t[b] : 0;
      float k4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) k4[e] = acc[b][e];
      if constexpr (SAMPLE) {
        if (b < nrun && kind[b] == 1) {
          // tokens tb + g*4 + [0,4) are exactly one Philox call
          uint32_t c0 = (uint32_t)(tb + g * 4) >> 2, c1 = pc1, c2 = pc2, c3 = pc3;
          philox10(c0, c1, c2, c3, p.keys);
          const uint32_t w[4] = {c0, c1, c2, c3};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            k4[e] = (tb + g * 4 + e < V) ? gumbel_key2(acc[b][e], p.cT, w[e]) : kNegInf;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        L.bz[b][g * 4 + e] = acc[b][e];
        L.bk[b][g * 4 + e] = k4[e];
      }
    }
  }
  wave_sync_lds();
#ifdef TS_DEBUG_RUNS
  mism += nrun * 1000;
#endif
  // lane l checks key j = l + 64 h of the batch (run j / 16, token j % 16)
#pragma unroll
  for (int h = 0; h < kBatch / 4; ++h) {
    const int j = lane + 64 * h;
    const int b = j >> 4, e = j & 15;
    const float kv = L.bk[b][e];
    int tb = 0, kd = 0;
    float ex = 0.0f;
#pragma unroll
    for (int q = 0; q < kBatch; ++q)
      if (q == b) { tb = t[q]; kd = kind[q]; ex = expect[q]; }
    const bool live = b < nrun && tb + e < V;
    float rm = live ? kv : kNegInf;
    rm = row_max(rm);  // the run's 16 keys sit in one row of 16 lanes
    mism += __popcll(__ballot(live && e == 0 && !__builtin_isnan(ex) && run_key(rm, (tb % p.Vc) >> 4) != ex));
    const float th = kd ? thr[1] : thr[0];
    uint64_t mask = __ballot(live && kv >= th);
    while (mask) {
      const int src = __ffsll((unsigned long long)mask) - 1;
      mask &= mask - 1;
      const float cv = lane_f32(kv, src);
      const float cz = lane_f32(L.bz[b][e], src);
      const int ct = lane_i32(tb + e, src);
      const int ck = lane_i32(kd, src);
      if (ck == 0)
        reglist_insert(zl, p.K, cv, ct, cz);
      else
        reglist_insert(gl, p.K, cv, ct, cz);
    }
  }
  wave_sync_lds();
}

// Descending bitonic sort of N values in registers (N a power of two).
template <int N>
__device__ __forceinline__ void sort_desc(float (&x)[N]) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          const float hi = fmaxf(x[i], x[l]), lo = fminf(x[i], x[l]);
          const bool desc = (i & k) == 0;
          x[i] = desc ? hi : lo;
          x[l] = desc ? lo : hi;
        }
      }
}

// The LL largest of the lane's list a (descending) and b (descending), in
// descending order: max(a[k], b[LL-1-k]) is a bitonic sequence holding
// them, and a half-cleaner cascade sorts it.  The result does not depend on
// which list is a.
template <int LL>
__device__ __forceinline__ void merge_top(float (&a)[LL], const float (&b)[LL]) {
#pragma unroll
  for (int k = 0; k < LL; ++k) a[k] = fmaxf(a[k], b[LL - 1 - k]);
#pragma unroll
  for (int j = LL >> 1; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < LL; ++i) {
      const int l = i ^ j;
      if (l > i) {
        const float hi = fmaxf(a[i], a[l]), lo = fminf(a[i], a[l]);
        a[i] = hi;
        a[l] = lo;
      }
    }
}

// The K-th largest (K <= LL) of the wave's entries, NE per lane, equal
// values counted separately; -inf when fewer than K are finite.  Each lane
// sorts its entries and keeps LL of them; six exchange steps then merge the
// lists of partner lanes (lanes i^1, i^2, the mirrored lane in its group of
// 8 and of 16, i^16, i^32), after which every lane holds the wave's top LL.
template <int LL, int NE>
__device__ __forceinline__ float wave_kth_largest(const float (&v)[NE], int K) {
  float x[NE];
#pragma unroll
  for (int i = 0; i < NE; ++i) x[i] = v[i];
  sort_desc<NE>(x);
  float a[LL], b[LL];
#pragma unroll
  for (int k = 0; k < LL; ++k) a[k] = k < NE ? x[k] : kNegInf;
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = dpp_f32<0xB1>(a[k]);
  merge_top<LL>(a, b);
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = dpp_f32<0x4E>(a[k]);
  merge_top<LL>(a, b);
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = dpp_f32<0x141>(a[k]);
  merge_top<LL>(a, b);
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = dpp_f32<0x140>(a[k]);
  merge_top<LL>(a, b);
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = xor16_f32(a[k]);
  merge_top<LL>(a, b);
#pragma unroll
  for (int k = 0; k < LL; ++k) b[k] = xor32_f32(a[k]);
  merge_top<LL>(a, b);
  float r = kNegInf;
#pragma unroll
  for (int k = 0; k < LL; ++k) r = k == K - 1 ? a[k] : r;
  return r;
}

// Threshold and candidate items for one key kind.  Let L be the K-th
// largest recorded run key: those are keys of K distinct runs, whose maxima
// lie within kRunSlack / 2 units of their keys, so the K-th largest token
// key over the vocabulary is at least L lowered by kRunSlack / 2 units, and
// a run holding such a token has a key of at least L lowered by kRunSlack
// units (the returned threshold).  Such a run is one of its chunk's recorded
// runs, or, when the chunk's rest key reaches the threshold too, anywhere in
// the chunk (a whole-chunk item).
// NE, NR: recorded-run and chunk-rest slots per lane (NE = 4 NR; S <= 64 NR).
template <int NE, int NR>
__device__ __forceinline__ float select_items_n(const MergeParams& p, const RunSummaryPtr& sm,
                                                int pidx, int kind, MergeLds& L, int& nitems) {
  constexpr int kEntrySlots = NE, kRestSlots = NR;
  const int lane = threadIdx.x & 63;
  const int S = p.S, K = p.K;
  const size_t pb = (size_t)pidx * S;
  float ev[kEntrySlots];
  float rv[kRestSlots];
  // Every load reads a clamped index, so all are in flight together.  A slot
  // past the last chunk holds a copy of a real entry: it starts out taken in
  // the threshold rounds below, and every later use checks the chunk range.
  float live[kEntrySlots];
#pragma unroll
  for (int i = 0; i < kEntrySlots; ++i) {
    const int e = i * 64 + lane;
    const size_t ec = pb * kTopRuns + min(e, S * kTopRuns - 1);
    ev[i] = sm.m[ec];
    live[i] = (e >> 2) < S ? ev[i] : kNegInf;
  }
#pragma unroll
  for (int i = 0; i < kRestSlots; ++i) rv[i] = sm.rest[pb + min(i * 64 + lane, S - 1)];
  // fewer than K runs recorded: -inf, every token is a candidate
  float thr = K <= 8 ? wave_kth_largest<8, kEntrySlots>(live, K) : wave_kth_largest<16, kEntrySlots>(live, K);
  thr = key_lowered(thr, kRunSlack);

  // whole chunks
#pragma unroll
  for (int i = 0; i < kRestSlots; ++i) {
    const uint64_t wm = __ballot(rv[i] >= thr);
    if (lane == 0) {
      L.whole[2 * i] = (uint32_t)wm;
      L.whole[2 * i + 1] = (uint32_t)(wm >> 32);
    }
  }
  wave_sync_lds();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int base = nitems;
  // recorded runs of chunks that are not whole
#pragma unroll
  for (int i = 0; i < kEntrySlots; ++i) {
    const int e = i * 64 + lane;
    const int c = e >> 2;
    const bool in = c < S;
    const bool wh = in && ((L.whole[c >> 5] >> (c & 31)) & 1u);
    const bool cand = in && !wh && ev[i] >= thr;
    const uint64_t mask = __ballot(cand);
    const int off = base + __popcll(mask & lt);
    if (cand && off < kItemCap) {
      const int run = run_of(ev[i]);
      L.item_t[off] = c * p.Vc + (run >> 2) * 64 + (run & 3) * 16;
      L.item_k[off] = kind;
      L.item_e[off] = ev[i];
    }
    base += __popcll(mask);
  }
#pragma unroll
  for (int i = 0; i < kRestSlots; ++i) {
    const int c = i * 64 + lane;
    const bool cand = c < S && rv[i] >= thr;
    const uint64_t mask = __ballot(cand);
    const int off = base + __popcll(mask & lt);
    if (cand && off < kItemCap) {
      L.item_t[off] = -(c + 1);
      L.item_k[off] = kind;
      L.item_e[off] = __builtin_nanf("");
    }
    base += __popcll(mask);
  }
  if (base > kItemCap) {
    // too many candidates (heavy ties): rescan every chunk of this kind
    base = nitems;
    for (int c0 = 0; c0 < S; c0 += 64) {
      const int c = c0 + lane;
      if (c < S && base + c - c0 < kItemCap) {
        L.item_t[base + c - c0] = -(c + 1);
        L.item_k[base + c - c0] = kind;
        L.item_e[base + c - c0] = __builtin_nanf("");
      }
      base += min(64, S - c0);
    }
    thr = kNegInf;
  }
  nitems = min(base, kItemCap);
  wave_sync_lds();
  return thr;
}

__device__ __forceinline__ float select_items(const MergeParams& p, const RunSummaryPtr& sm,
                                              int pidx, int kind, MergeLds& L, int& nitems) {
  if (p.S <= 64) return select_items_n<4, 1>(p, sm, pidx, kind, L, nitems);
  return select_items_n<kMaxChunks * kTopRuns / 64, kMaxChunks / 64>(p, sm, pidx, kind, L, nitems);
}

// ---------------------------------------------------------------- sequential draws

constexpr int kSegSlots = (TS_MAX_V + 64 * kSegTokens - 1) / (64 * kSegTokens);  // segments per lane

// One categorical pick over items laid out as item = 64 * slot + lane with
// masses m >= 0: the first item whose inclusive cumulative mass exceeds
// u * total (never a zero-mass item); rounding at the top end falls back to
// the last item with mass.  Returns -1 only if every mass is zero.
template <int NS>
__device__ __forceinline__ int wave_pick(const float (&m)[NS], float u) {
  float c[NS];
  float base = 0.0f;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const float x = wave_incl_scan(m[i]);
    c[i] = base + x;
    base += lane_f32(x, 63);
  }
  const float t = u * base;
  int cnt = 0, last = -1;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    cnt += __popcll(__ballot(c[i] <= t));
    const uint64_t pos = __ballot(m[i] > 0.0f);
    if (pos) last = 64 * i + 63 - __clzll((long long)pos);
  }
  return cnt > last ? last : cnt;
}

// K draws without replacement from q_T, one after another (§3.3 residual
// proposal): draw j picks a segment, a block in it and a token in it, each in
// proportion to its remaining mass, from the words of one Philox call
// (c0 = j, tag 4).  Masses are kept as base-2 logs: the segment pick scales
// them by the largest segment, the block and token picks by the segment's
// and the block's own log-mass (no member exceeds it), and a block's mass
// after a removal is summed relative to the largest token left, so removing
// drawn tokens never underflows the rest.
// The parent's block table lives in LDS when it fits (V <= 40 * 4096), else
// in its rows of the workspace; a drawn token's block is rewritten in place.
// Draw j lands in lane j - 1 of gl (token, z); a draw after every token with
// a finite logit has been drawn is empty (token -1, z = -inf).  Every value
// here is finite or -inf for finite or -inf logits, so maxima take the median
// form; whatever the logits hold, every load stays inside the parent's rows.

template <typename TE, int KS, int NSEG>
__device__ __forceinline__ void seq_draws_n(const MergeParams& p, int pidx, const TE* urow,
                                          const typename Frag<TE>::type (&erow_all)[KS], uint32_t pc1,
                                          uint32_t pc2, uint32_t pc3, DrawLds& L, RegList& gl) {
  typedef Frag<TE> F;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, g = lane >> 4;
  const int V = p.V, nblk = p.nblk;
  const TE* W2 = static_cast<const TE*>(p.W2);
  float* gblk = p.blk + (size_t)pidx * p.blk_ld;
  constexpr int kBps = kSegTokens / kBlkTokens;  // blocks per segment (64)
  const int nseg = (nblk + kBps - 1) / kBps;
  const bool in_lds = nseg <= kLdsSegs;

  // Segment log-masses (lane l owns segment l + 64 i).  The wave reads the
  // table one segment per load (lane = block offset, coalesced); every load
  // is issued before the first reduction (a global round trip costs about
  // as much as all the arithmetic here).  The table is kept in LDS when it
  // fits, and segments are reduced eight at a time.
  float segL[NSEG];
#pragma unroll
  for (int i = 0; i < NSEG; ++i) segL[i] = kNegInf;
  auto reduce8 = [&](int s0, const float (&xs)[8]) {
    float m[8], e[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) m[k] = xs[k];
    wave_max8(m);
#pragma unroll
    for (int k = 0; k < 8; ++k) e[k] = m[k] == kNegInf ? 0.0f : exp2_fast(xs[k] - m[k]);
    wave_sum8(e);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int sg = s0 + k;
      const float l = m[k] == kNegInf ? kNegInf : m[k] + __builtin_amdgcn_logf(e[k]);
#pragma unroll
      for (int i = 0; i < NSEG; ++i)
        if (sg < nseg && sg == 64 * i + lane) segL[i] = l;
    }
  };
  // the row goes straight to LDS (no registers): each direct load moves 256
  // entries, 16 bytes per lane; a piece past the row's stride reads its last
  // 16 bytes instead, and every entry at or past nblk (the last segment's
  // tail) is set to -inf once the loads have landed
  const int nent = nseg * kBps;
  if (in_lds) {
    const int npc = (nent + 255) / 256;
    for (int pc = 0; pc < npc; ++pc)
      lds_dma16(gblk + min(pc * 256 + lane * 4, p.blk_ld - 4), reinterpret_cast<u32x4*>(L.seg_blk + pc * 256));
  }
  // the words of every draw (lane j - 1 computes draw j's Philox call), while
  // the table loads are in flight
  uint32_t dw0 = (uint32_t)(lane + 1), dw1 = pc1, dw2 = pc2, dw3 = pc3;
  philox10(dw0, dw1, dw2, dw3, p.keys);
  if (in_lds) {
    __builtin_amdgcn_s_waitcnt(0);
    for (int b = nblk + lane; b < nent; b += 64) L.seg_blk[b] = kNegInf;
    wave_sync_lds();
    // lane l reduces segment l from LDS (no cross-lane steps); the 16-byte
    // pieces of its row are read in a lane-rotated order
    if (lane < nseg) {
      const f32x4* row = reinterpret_cast<const f32x4*>(L.seg_blk + lane * kBps);
      f32x4 xv[kBps / 4];
#pragma unroll
      for (int i = 0; i < kBps / 4; ++i) xv[i] = row[(i + lane) & (kBps / 4 - 1)];
      float m = kNegInf;
#pragma unroll
      for (int i = 0; i < kBps / 4; ++i)
        m = max2_med3(max2_med3(m, max2_med3(xv[i][0], xv[i][1])), max2_med3(xv[i][2], xv[i][3]));
      if (m != kNegInf) {
        float a[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < kBps / 4; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) a[e] += exp2_fast(xv[i][e] - m);
        segL[0] = m + __builtin_amdgcn_logf((a[0] + a[1]) + (a[2] + a[3]));
      }
    }
  } else {
#pragma unroll 1
    for (int s0 = 0; s0 < nseg; s0 += 8) {
      float xs[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int b = (s0 + k) * kBps + lane;
        xs[k] = keep_or(gblk[min(b, nblk - 1)], opaque_mask(s0 + k < nseg && b < nblk), kNegInf);
      }
      reduce8(s0, xs);
    }
  }
  // the parent's whole q_T mass (base-2 log), from the segments before any
  // draw: the log-sum-exp of z / T is ln 2 times it
  {
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < NSEG; ++i) mx = fmaxf(mx, segL[i]);
    mx = wave_max_fin(mx);
    float e = 0.0f;
#pragma unroll
    for (int i = 0; i < NSEG; ++i) e += segL[i] == kNegInf ? 0.0f : exp2_fast(segL[i] - mx);
    e = wave_sum(e);
    if (lane == 0) L.lmass = mx == kNegInf ? kNegInf : mx + __builtin_amdgcn_logf(e);
  }
  gl.cnt = 0;
#pragma unroll 1
  for (int j = 1; j <= p.K; ++j) {
    const uint32_t w0 = (uint32_t)lane_i32((int)dw0, j - 1);
    const uint32_t w1 = (uint32_t)lane_i32((int)dw1, j - 1);
    const uint32_t w2 = (uint32_t)lane_i32((int)dw2, j - 1);
    // level 1: segment
    float ms[NSEG];
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < NSEG; ++i) mx = fmaxf(mx, segL[i]);
    mx = wave_max_fin(mx);
#pragma unroll
    for (int i = 0; i < NSEG; ++i) ms[i] = segL[i] == kNegInf ? 0.0f : exp2_fast(segL[i] - mx);
    const int sg = wave_pick(ms, word_to_uniform(w0));
    // level 2: block within the segment (lane = block offset)
    // The masses are taken relative to the segment's own log-mass, which no
    // block of it exceeds (a common scale, so no reduction for a maximum).
    const int b = sg * kBps + lane;
    const bool bin = sg >= 0 && b < nblk;
    const float lb = bin ? (in_lds ? L.seg_blk[b] : gblk[b]) : kNegInf;
    float sref = 0.0f;
#pragma unroll
    for (int i = 0; i < NSEG; ++i)
      if (sg >= 0 && (sg >> 6) == i) sref = lane_f32(segL[i], sg & 63);
    float m2[1];
    m2[0] = lb == kNegInf ? 0.0f : exp2_fast(lb - sref);
    const int bo = wave_pick(m2, word_to_uniform(w1));
    const int bsel = sg * kBps + bo;
    // level 3: token within the block; recompute its 64 logits (four runs of
    // 16).  The operands are the streaming pass's with their roles swapped:
    // E in every row of A, the run's W2 rows as the columns of B, so run q's
    // logit of token t0 + 16 q + n lands in lane n + 16 i for every row
    // group i (the matrix core gives the same values bit for bit either
    // way).  Lane y takes run y / 16 and so holds token t0 + y; its seed is
    // that token's U (-inf past V), the other runs' results on it are unused.
    // Every load is issued before the MFMAs (one round trip).
    // with no mass left (fewer than j tokens have finite logits) both picks
    // are -1: the loads then read block 0, no lane is live and the draw is empty
    const int t0 = max(bsel, 0) * kBlkTokens;
    const int y = t0 + lane;
    typename F::type wf[4][KS];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const TE* wrow = W2 + (size_t)min(t0 + 16 * q + n, V - 1) * p.r;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) wf[q][kk] = F::load(wrow, kk * F::kPerStep, g);
    }
    const float useed = keep_or(F::to_f32(urow[min(y, V - 1)]), opaque_mask(y < V), kNegInf);
    // while the block's rows are in flight: the log-mass of the segment's
    // other blocks, so that its new mass after the draw takes no reduction
    const float lo = lane == bo ? kNegInf : lb;
    const float mo = wave_max_fin(lo);
    const float so = wave_sum(lo == kNegInf ? 0.0f : exp2_fast(lo - mo));
    f32x4 acc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = f32x4{useed, useed, useed, useed};
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) acc[q] = F::mma(erow_all[kk], wf[q][kk], acc[q]);
    // the four registers of a run's result hold the same value (every row of
    // A is E); all four are read, so none of them is handed to another value
    // while the matrix core may still be writing it (with only one register
    // read, the compiler reused the other three a few wait states after the
    // MFMA and the loaded W2 row came from a clobbered address)
    float zq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      zq[q] = max2_med3(__builtin_amdgcn_fmed3f(acc[q][0], acc[q][1], acc[q][2]), acc[q][3]);
    const float zy = g == 0 ? zq[0] : g == 1 ? zq[1] : g == 2 ? zq[2] : zq[3];
    // tokens drawn before are out: lanes of gl not drawn yet hold id
    // 0x7FFFFFFF (an empty draw -1), which no y matches
    bool live = y < V && bo >= 0 && sg >= 0;
#pragma unroll
    for (int k = 0; k < 7; ++k) live &= lane_i32(gl.id, k) != y;
    if (p.K > 8) {
#pragma unroll
      for (int k = 7; k < TS_MAX_K - 1; ++k) live &= lane_i32(gl.id, k) != y;
    }
    // relative to the block's log-mass, which no live token of it exceeds
    const float xy = live ? zy * p.cT : kNegInf;
    const float bref = bo >= 0 ? lane_f32(lb, bo) : 0.0f;
    float m3[1];
    m3[0] = live ? exp2_fast(xy - bref) : 0.0f;
    const int to = wave_pick(m3, word_to_uniform(w2));
    const int tsel = t0 + to;
    const float zsel = lane_f32(zy, to < 0 ? 0 : to);
    if (lane == j - 1) {
      gl.id = to < 0 ? -1 : tsel;
      gl.aux = to < 0 ? kNegInf : zsel;
      gl.val = 0.0f;
    }
    // the block and the segment lose the drawn token's mass; both sums are
    // taken relative to the largest value left, so nothing underflows
    const bool left = live && lane != to;
    const float mt2 = wave_max_fin(left ? xy : kNegInf);
    const float rest3 = wave_sum(left ? exp2_fast(xy - mt2) : 0.0f);
    const float lnew = mt2 == kNegInf ? kNegInf : mt2 + __builtin_amdgcn_logf(rest3);
    if (lane == bo && bin) {
      if (in_lds)
        L.seg_blk[bsel] = lnew;
      else
        gblk[bsel] = lnew;
    }
    if (in_lds) {
      wave_sync_lds();
    } else {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    // the segment: its other blocks (mo, so) and the block's new mass
    const float M = max2_med3(mo, lnew);
    const float tot = (mo == kNegInf ? 0.0f : so * exp2_fast(mo - M)) + (lnew == kNegInf ? 0.0f : exp2_fast(lnew - M));
    const float snew = M == kNegInf ? kNegInf : M + __builtin_amdgcn_logf(tot);
#pragma unroll
    for (int i = 0; i < NSEG; ++i)
      if (sg == 64 * i + lane) segL[i] = snew;
  }
  gl.cnt = p.K;
}

// The draws with NSEG segment slots per lane: one when the vocabulary has at
// most 64 segments (V <= 64 * 4096), so level 1 is a single scan.
template <typename TE, int KS>
__device__ __forceinline__ void seq_draws(const MergeParams& p, int pidx, const TE* urow,
                                          const typename Frag<TE>::type (&erow_all)[KS], uint32_t pc1,
                                          uint32_t pc2, uint32_t pc3, DrawLds& L, RegList& gl) {
  const int nseg = (p.nblk + kSegTokens / kBlkTokens - 1) / (kSegTokens / kBlkTokens);
  if (nseg <= 64)
    seq_draws_n<TE, KS, 1>(p, pidx, urow, erow_all, pc1, pc2, pc3, L, gl);
  else
    seq_draws_n<TE, KS, kSegSlots>(p, pidx, urow, erow_all, pc1, pc2, pc3, L, gl);
}

template <typename TE, int KS, int MODE>
__global__ __launch_bounds__(256) void expand_merge_kernel(const MergeParams p) {
  typedef Frag<TE> F;
  typedef typename F::type FT;
  constexpr bool SAMPLE = MODE != kModeGreedy;
  constexpr bool GUMBEL = MODE == kModeGumbel;
  constexpr bool SEQ = MODE == kModeSeq;
  // Sequential draws: one parent per workgroup; wave 1 draws while wave 0
  // finds the greedy top-K, then wave 0 scores the children.
  __shared__ MergeShared<SEQ> sh;
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int pidx = SEQ ? blockIdx.x : blockIdx.x * 4 + wv;
  if (pidx >= launch_parents(p)) return;  // uniform over the workgroup when SEQ
#ifdef TS_DEBUG_RUNS
  const long long t_start = clock64();
#endif
  MergeLds& L = sh.l[SEQ ? 0 : wv];
  const int K = p.K, V = p.V, S = p.S;
  const ts_parent par = p.parents[pidx];
  const bool ok = par.token >= 0 && par.token < V && par.depth >= 0 && par.depth < p.D &&
                  par.request >= 0 && par.request < p.R;
  const size_t ob = (size_t)pidx * K;
  if (!ok) {
    if (SEQ && wv != 0) return;
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
  const TE* urow = static_cast<const TE*>(p.U) + ((size_t)par.request * p.D + par.depth) * (size_t)V;
  const TE* erow = static_cast<const TE*>(p.E) + (size_t)par.token * p.r;
  FT bcol[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) bcol[kk] = (n == 0) ? F::load(erow, kk * F::kPerStep, g) : F::zero();
  const uint32_t pc1 = (uint32_t)par.path, pc2 = (uint32_t)(par.path >> 32);
  const uint32_t pc3 = counter_word3(par.request, par.depth, 1u);

  if constexpr (SEQ) {
    if (wv == 1) {
      // the draws are the longer of the two chains: their wave issues first
      // when both waves of a SIMD are ready
      __builtin_amdgcn_s_setprio(2);
      // the parent's E fragment on every lane: the A operand of the draws'
      // block recompute
      FT eall[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) eall[kk] = F::load(erow, kk * F::kPerStep, g);
      RegList dl;
      reglist_init(dl);
      seq_draws<TE, KS>(p, pidx, urow, eall, pc1, pc2, counter_word3(par.request, par.depth, 4u), sh.d, dl);
      if (lane < K) {
        sh.d.id[lane] = dl.id;
        sh.d.z[lane] = dl.aux;
      }
      __syncthreads();
      return;
    }
  }
  const size_t pbase = (size_t)pidx * S;

  // log-sum-exp over chunks: each lane folds its chunks in index order, then a
  // fixed butterfly.  The chunks' sums are against their own references.
  // With sequential draws the log-sum-exp of z / T (and of z at T = 1) comes
  // from the block masses instead, once the draws' wave has them.
  constexpr bool kPartsT = SAMPLE && !SEQ;  // the streaming pass kept sums of z / T
  const bool parts0 = !SEQ || p.need_T;     // ... and sums of z
  float lse0 = __builtin_nanf(""), lseT = __builtin_nanf("");
  if (parts0) {
    float pm[kRestSlots], ps[kRestSlots], pt[kRestSlots];
#pragma unroll
    for (int i = 0; i < kRestSlots; ++i) {
      const int c = i * 64 + lane;
      // clamped loads, masked after: all of them in flight together (without
      // the z/T sums, their loads read the z sums and are masked out)
      const size_t cc = pbase + min(c, S - 1);
      const uint32_t in = opaque_mask(c < S);
      const bool has_T = kPartsT && p.need_T;
      pm[i] = keep_or(p.part_m[cc], in, kNegInf);
      ps[i] = keep_or_zero(p.part_s0[cc], in);
      pt[i] = keep_or_zero((has_T ? p.part_sT : p.part_s0)[cc], in & opaque_mask(has_T));
    }
    float M = kNegInf;
#pragma unroll
    for (int i = 0; i < kRestSlots; ++i) M = fmaxf(M, pm[i]);
    M = wave_max(M);
    const float Mref = fmaxf(M, -1e30f);
    float s = 0.0f, st = 0.0f;
#pragma unroll
    for (int i = 0; i < kRestSlots; ++i) {
      s += ps[i] * exp2_fast(__builtin_fmaf(pm[i], kLog2e, -Mref * kLog2e));
      if (kPartsT && p.need_T) st += pt[i] * exp2_fast(__builtin_fmaf(pm[i], p.cT, -Mref * p.cT));
    }
    s = wave_sum(s);
    st = wave_sum(st);
    lse0 = M + logf(s);
    if (kPartsT) lseT = p.need_T ? M / p.T + logf(st) : lse0;
  }

  int nitems = 0;
  float thr[2];
  thr[0] = select_items(p, p.zs, pidx, 0, L, nitems);
  thr[1] = kNegInf;
  if constexpr (GUMBEL) thr[1] = select_items(p, p.gs, pidx, 1, L, nitems);

  RegList zl, gl;
  reglist_init(zl);
  reglist_init(gl);
  int mism = 0;
  const float nan = __builtin_nanf("");
  // a batch's loads in one round trip at rank <= 64; in two with sequential
  // draws (beside the draws, which are the longer chain, the wave keeps to
  // the registers that leave four waves per SIMD) or at higher ranks
  constexpr int kRescanParts = (SEQ || KS > 2) ? 2 : 1;
  int it = 0, sub = 0;
#pragma unroll 1
  while (it < nitems) {
    int qt[kBatch], qk[kBatch];
    float qe[kBatch];
#pragma unroll
    for (int q = 0; q < kBatch; ++q) { qt[q] = 0; qk[q] = 0; qe[q] = nan; }
    int nr = 0;
    // the leading single-run items of the batch in one read by all lanes
    // (lane i reads item it + i); they fill the arrays as the loop below
    // would, the last one read in slot 0
    if (sub == 0) {
      const int cnt = min(kBatch, nitems - it);
      const int li = it + min(lane, cnt - 1);
      const int code = L.item_t[li];
      const int kd = L.item_k[li];
      const float e = L.item_e[li];
      const uint64_t whole = __ballot(lane < cnt && code < 0);
      const int m = whole ? min(cnt, __ffsll((unsigned long long)whole) - 1) : cnt;
#pragma unroll
      for (int q = 0; q < kBatch; ++q)
        if (q < m) {
          qt[q] = lane_i32(code, m - 1 - q);
          qk[q] = lane_i32(kd, m - 1 - q);
          qe[q] = lane_f32(e, m - 1 - q);
        }
      nr = m;
      it += m;
    }
#pragma unroll 1
    while (nr < kBatch && it < nitems) {
      const int code = L.item_t[it];
      const int kd = L.item_k[it];
      int t;
      float e;
      if (code < 0) {
        const int cc = -code - 1;
        const int cbeg = cc * p.Vc;
        const int nruns = ((min(cbeg + p.Vc, V) - cbeg + 63) / 64) * 4;
        t = cbeg + (sub >> 2) * 64 + (sub & 3) * 16;
        e = nan;
        if (++sub == nruns) { sub = 0; ++it; }
        if (t >= V) continue;
      } else {
        t = code;
        e = L.item_e[it];
        ++it;
      }
#pragma unroll
      for (int q = kBatch - 1; q > 0; --q) { qt[q] = qt[q - 1]; qk[q] = qk[q - 1]; qe[q] = qe[q - 1]; }
      qt[0] = t;
      qk[0] = kd;
      qe[0] = e;
      ++nr;
    }
    if (nr > 0)
      rescan_batch<TE, KS, GUMBEL, kRescanParts>(p, urow, bcol, pc1, pc2, pc3, qt, qk, qe, nr, thr, L, zl, gl,
                                                 mism);
  }
  if constexpr (SEQ) {
    __syncthreads();  // the draws of wave 1
    if (lane < K) {
      gl.id = sh.d.id[lane];
      gl.aux = sh.d.z[lane];
      gl.val = 0.0f;
    }
    gl.cnt = K;
    lseT = sh.d.lmass * kLn2;
    if (!p.need_T) lse0 = lseT;  // T = 1
  }

  // Child scoring: lane j handles slot j + 1 (Algorithm 1; §3.2 pre-draw bound; Eq. 3).
  const float lsp = par.log_surv;
  const float a = p.calib_a, bb = p.calib_b;
  float zb = 0.0f;
  if constexpr (SAMPLE) {
    // bound of slot j: the first of the greedy order not drawn before j.
    // Lane i < K first finds the first draw s < K - 1 that took greedy entry
    // i (K if none); slot j's bound is then the first entry with drawn_at >= j.
    int drawn_at = K;
#pragma unroll
    for (int s2 = TS_MAX_K - 2; s2 >= 0; --s2)
      if (s2 < K - 1 && lane_i32(gl.id, s2) == zl.id) drawn_at = s2;
    int bi = K - 1;
#pragma unroll
    for (int i = TS_MAX_K - 1; i >= 0; --i)
      if (i < K && lane_i32(drawn_at, i) >= lane) bi = i;
    zb = __shfl(zl.val, bi, 64);
  }
  if (lane < K) {
    const int j = lane;
    const float zpi = zl.val;
    if (p.out.rank_token) p.out.rank_token[ob + j] = zl.id;
    if (p.out.rank_log_q0) p.out.rank_log_q0[ob + j] = zpi - lse0;
    if constexpr (!SAMPLE) {
      const float lq0 = zpi - lse0;
      const float ls = lsp + log_phat(lq0, a, bb);
      p.out.child_token[ob + j] = zl.id;
      p.out.child_log_q0[ob + j] = lq0;
      p.out.child_log_surv[ob + j] = ls;
      p.out.slot_key[ob + j] = ls;
      if (p.out.child_log_qT) p.out.child_log_qT[ob + j] = __builtin_nanf("");
    } else {
      const float zc = gl.aux;
      const float lq0 = zc - lse0;
      p.out.child_token[ob + j] = gl.id;
      p.out.child_log_q0[ob + j] = lq0;
      p.out.child_log_surv[ob + j] = lsp + log_phat(lq0, a, bb);
      p.out.slot_key[ob + j] = lsp + log_phat(zb - lse0, a, bb);
      if (p.out.child_log_qT) p.out.child_log_qT[ob + j] = zc / p.T - lseT;
    }
  }
  if (lane == 0) {
    if (p.out.lse0) p.out.lse0[pidx] = lse0;
    if (p.out.lseT) p.out.lseT[pidx] = lseT;
#ifdef TS_DEBUG_RUNS
    if (p.out.rank_log_q0) p.out.rank_log_q0[ob + K - 1] = (float)(clock64() - t_start);
#endif
    if (p.out.diag) p.out.diag[pidx] = mism;
  }
}

}  // namespace ts
