// One launch per level of the T > 0 walk (§3.3, Proposition 1) with the
// rows held in registers.
//
// The per-stage launches read an item's target and draft rows once for pass A
// and again for every rejected child, so a node whose children are all
// rejected costs 1 + m sweeps of both rows.  Here each workgroup (item,
// chunk) loads its chunk of the two rows into registers once and keeps it for
// the whole walk at that node: pass A, the Z_j reductions of every rejected
// stage and the bonus keys all read registers.
//
// The chunks of an item meet between the walk's steps through tagged slots
// in global memory: a workgroup stores its partial result for a step as
// 64-bit words holding the value and the launch's epoch, with agent-scope
// relaxed stores (coherent across the XCDs' L2 caches); wave 0 of every
// workgroup that needs the step's total polls the item's slots of that step
// with agent-scope loads until every chunk's words carry the epoch, and reduces
// them in the same fixed order, so all workgroups take the same decisions.
// The slots are cleared once per ts_verify call and each launch of the call
// has its own epoch, so no stale word matches.  The host sizes the grid to
// what the device holds at once, so every workgroup is resident and every wait
// ends; each wait is also bounded, and one that runs out sets a flag (device
// and pinned host copies) that ends the other waits early: the host then runs
// the level again through the per-stage launches.
#pragma once

#include "verify_kernels.hpp"

namespace ts {

// Quads of four tokens each thread holds: 40 tokens of a bf16 target (20 KB
// of LDS per workgroup for the target, 40 VGPRs for the draft), 24 of a
// float target (24 KB of LDS).
constexpr int kFusedQuadsBf16 = 10;
constexpr int kFusedQuadsF32 = 6;
// Most chunks an item is split into (more only when the chunk would not fit).
constexpr int kFusedMaxChunks = 32;

// Words of an item's slots, each [cpi] long: pass A (maxima and sums of
// both rows), the Z_j partial of each stage, the bonus keys' best, second
// best and token.
constexpr int kSlotPA = 0, kSlotZ = 4, kSlotB = 4 + TS_MAX_K, kSlotWords = 7 + TS_MAX_K;
// Most chunks of an item in one launch (one polling lane per chunk), and
// most workgroups of one launch (the slots are sized for that many).
constexpr int kFusedMaxCpi = 64;
constexpr int kFusedMaxGrid = 4096;

struct VFused {
  int cpi;           // chunks per item (<= kFusedMaxCpi)
  int chunk;         // tokens per chunk, a multiple of 4
  uint64_t* slots;   // [nitems][kSlotWords][cpi]: value bits | epoch << 32
  uint32_t epoch;    // this launch's tag (slots start the call at zero)
  int* err;          // device flag: a wait ran out
  int32_t* herr;     // the flag's pinned host copy
  int spin_limit;    // polls before a wait gives up
  const VerifyNext* next_host;  // [nitems], pinned host memory
};

// Quad of target values as loaded: four bf16 in two words, or four floats.
template <typename TT>
struct TQuad;
template <>
struct TQuad<uint16_t> {
  using type = uint2;
};
template <>
struct TQuad<float> {
  using type = f32x4;
};
__device__ __forceinline__ float tquad_at(const uint2& w, int e) {
  const uint32_t x = (e < 2) ? w.x : w.y;
  return __uint_as_float((e & 1) ? (x & 0xFFFF0000u) : (x << 16));
}
__device__ __forceinline__ float tquad_at(const f32x4& v, int e) { return v[e]; }

// Tokens b .. b+3 of both rows (z only when zrow is set); tokens at or past
// y1 read as -inf, which no maximum, sum or key takes up.  Quad loads when
// the rows hold a multiple of 4 tokens (every quad of a chunk, a multiple of
// 4 long, then lies wholly inside or outside it), token loads otherwise.
template <typename TT>
__device__ __forceinline__ void load_quad_vec(const TT* trow, const float* zrow, int b, int y1,
                                              typename TQuad<TT>::type& t, f32x4& z) {
  if (b < y1) {
    if constexpr (sizeof(TT) == 2)
      t = *reinterpret_cast<const uint2*>(trow + b);
    else
      t = *reinterpret_cast<const f32x4*>(trow + b);
    if (zrow) z = *reinterpret_cast<const f32x4*>(zrow + b);
    else z = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
  } else {
    if constexpr (sizeof(TT) == 2)
      t = uint2{0xFF80FF80u, 0xFF80FF80u};
    else
      t = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
    z = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
  }
}
template <typename TT>
__device__ __forceinline__ void load_quad_tok(const TT* trow, const float* zrow, int b, int y1,
                                              typename TQuad<TT>::type& t, f32x4& z) {
  uint32_t tw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int y = b + e;
    if constexpr (sizeof(TT) == 2)
      tw[e] = y < y1 ? (uint32_t)trow[y] : 0xFF80u;
    else
      tw[e] = y < y1 ? __float_as_uint(trow[y]) : 0xFF800000u;
    z[e] = (zrow && y < y1) ? zrow[y] : kNegInf;
  }
  if constexpr (sizeof(TT) == 2)
    t = uint2{tw[0] | (tw[1] << 16), tw[2] | (tw[3] << 16)};
  else
    t = f32x4{__uint_as_float(tw[0]), __uint_as_float(tw[1]), __uint_as_float(tw[2]), __uint_as_float(tw[3])};
}

// Agent-scope relaxed accesses of 64-bit words.
__device__ __forceinline__ void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t pack_f32x2(float lo, float hi) {
  return (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32);
}
__device__ __forceinline__ float lo_f32(uint64_t w) { return __uint_as_float((uint32_t)w); }
__device__ __forceinline__ float hi_f32(uint64_t w) { return __uint_as_float((uint32_t)(w >> 32)); }

// Thread 0: the workgroup's word w of a step, tagged with the launch's epoch.
__device__ __forceinline__ void put_slot(const VFused& f, int it, int ck, int w, uint32_t bits) {
  st_agent(f.slots + ((size_t)it * kSlotWords + w) * f.cpi + ck, ((uint64_t)f.epoch << 32) | bits);
}

// Wave 0: lane k < cpi waits until words w0 .. w0 + NW - 1 of chunk k carry
// the launch's epoch and returns their values in out.  False when the wait
// ran out (the flag is then set) or another wait did.
template <int NW>
__device__ __forceinline__ bool poll_slots(const VFused& f, int it, int w0, uint32_t (&out)[NW]) {
  const int lane = threadIdx.x & 63;
  const bool mine = lane < f.cpi;
  const uint64_t* base = f.slots + ((size_t)it * kSlotWords + w0) * f.cpi + (mine ? lane : 0);
  bool ready = !mine;
#pragma unroll
  for (int i = 0; i < NW; ++i) out[i] = 0u;
  for (int n = 1;; ++n) {
    if (!ready) {
      uint64_t v[NW];
#pragma unroll
      for (int i = 0; i < NW; ++i) v[i] = ld_agent(base + (size_t)i * f.cpi);
      bool ok = true;
#pragma unroll
      for (int i = 0; i < NW; ++i) ok = ok && (uint32_t)(v[i] >> 32) == f.epoch;
      if (ok) {
#pragma unroll
        for (int i = 0; i < NW; ++i) out[i] = (uint32_t)v[i];
        ready = true;
      }
    }
    if (__all(ready)) return true;
    if ((n & 63) == 0) {
      if (__hip_atomic_load(f.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return false;
      if (n >= f.spin_limit) {
        if (lane == 0) {
          __hip_atomic_store(f.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(f.herr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        return false;
      }
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Bonus keys of a node without children over the thread's quads of its
// target row (r = 2^(t c - const): the draw comes from the target itself),
// reduced over the workgroup; thread 0 stores the chunk's best, second best
// and token in the bonus slots.
template <typename Q, int NQ>
__device__ __forceinline__ void leaf_keys(const Q (&tq)[NQ], int b0, int y1, float c, uint64_t path, uint32_t c3,
                                          const VerifyPass& vp, const VFused& f, int it, int ck, float* redv,
                                          int* redi) {
  const uint32_t pc1 = (uint32_t)path, pc2 = (uint32_t)(path >> 32);
  BonusTop bt;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (b0 + 1024 * q >= y1) break;
    // one quad's Philox words at a time: tied to the keys taken so far, the
    // next quad's words are not computed ahead (register pressure)
    int bq = b0 + 1024 * q;
    asm volatile("" : "+v"(bq) : "v"(bt.best));
    uint32_t w[4];
    bonus_words(w, bq, pc1, pc2, c3, vp.keys);
#pragma unroll
    for (int e = 0; e < 4; ++e) bt.add(tquad_at(tq[q], e) * c + gumbel_neg(w[e]), b0 + 1024 * q + e);
  }
  float vb = bt.best;
  int id = bt.idx;
  block_argmax(vb, id, redv, redi);
  float s2 = (bt.idx == id) ? bt.second : bt.best;
  s2 = block_max(s2, redv);
  if (threadIdx.x == 0) {
    put_slot(f, it, ck, kSlotB, __float_as_uint(vb));
    put_slot(f, it, ck, kSlotB + 1, __float_as_uint(s2));
    put_slot(f, it, ck, kSlotB + 2, (uint32_t)id);
  }
}

template <typename TT, int NQ>
__global__ __launch_bounds__(kVerifyThreads) __attribute__((amdgpu_waves_per_eu(4))) void verify_fused_kernel(
    VerifyPass vp, VFused f) {
  using Q = typename TQuad<TT>::type;
  static_assert(4 * NQ <= 64, "a thread's tokens fit the 64-bit child mask");
  __shared__ Q tl[NQ * kVerifyThreads];  // each thread's target quads, [q][thread]
  __shared__ VerifyItem sitem;
  __shared__ VerifyNext snext;
  __shared__ VConst sC;
  __shared__ VRec shr;
  __shared__ float redv[4];
  __shared__ int redi[4];
  __shared__ double redd[4];
  __shared__ int loc[TS_MAX_K];   // children inside the chunk: token
  __shared__ int locj[TS_MAX_K];  // and its place in the draw order (1-based)
  __shared__ int sh_n, sh_ok;
  const int it = blockIdx.x / f.cpi, ck = blockIdx.x % f.cpi;
  if (it >= vp.nitems) return;  // never: the grid is nitems * cpi
  const int tid = threadIdx.x;
  constexpr int kItemWords = (int)(sizeof(VerifyItem) / 4);
  constexpr int kNextWords = (int)(sizeof(VerifyNext) / 4);
  static_assert(kItemWords + kNextWords <= kVerifyThreads, "item and next words");
  if (tid < kItemWords)
    reinterpret_cast<int32_t*>(&sitem)[tid] = reinterpret_cast<const int32_t*>(vp.items_host + it)[tid];
  else if (tid < kItemWords + kNextWords)
    reinterpret_cast<int32_t*>(&snext)[tid - kItemWords] =
        reinterpret_cast<const int32_t*>(f.next_host + it)[tid - kItemWords];
  __syncthreads();
  const int m = sitem.m;
  const int y0 = ck * f.chunk, y1 = min(vp.V, y0 + f.chunk);
  const TT* trow = static_cast<const TT*>(vp.target) + ((size_t)sitem.request * vp.cap + sitem.node) * vp.V;
  const float* zrow = m > 0 ? vp.zbuf + (size_t)sitem.zrow * vp.V : nullptr;
  if (tid == 0) {
    int k = 0;
    for (int s = 0; s < m; ++s) {
      const int x = sitem.child_tok[s];
      if (x >= y0 && x < y1) {
        loc[k] = x;
        locj[k] = s + 1;
        ++k;
      }
    }
    sh_n = k;
  }
  // thread t holds the quads y0 + 4 t + 1024 q, q < NQ
  const int b0 = y0 + 4 * tid;
  Q tq[NQ];
  f32x4 zq[NQ];
  if (vector_rows<TT>(vp)) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) load_quad_vec<TT>(trow, zrow, b0 + 1024 * q, y1, tq[q], zq[q]);
  } else {
#pragma unroll
    for (int q = 0; q < NQ; ++q) load_quad_tok<TT>(trow, zrow, b0 + 1024 * q, y1, tq[q], zq[q]);
  }
  __syncthreads();
  const int nloc = sh_n;
  const float c = vp.c;
  const uint32_t pc1 = (uint32_t)sitem.path, pc2 = (uint32_t)(sitem.path >> 32);
  const uint32_t c3 = counter_word3(sitem.request, sitem.depth, 3u);
  bool alive = true;
  bool bonus = false;  // the walk ended without an accepted child: chunk 0 draws the bonus
  VRec rec;
  rec.status = kExhausted;  // a leaf: the bonus comes from the target itself
  rec.stage = 1;
  rec.alpha = 1.0f; rec.beta = 0.0f; rec.betap = 1.0f;
  rec.margin = __builtin_huge_valf();

  if (m == 0) {
    // leaf: bonus keys from the target row
    leaf_keys(tq, b0, y1, c, sitem.path, c3, vp, f, it, ck, redv, redi);
    bonus = true;
  } else {
    // an item with children holds the level's longest chain of steps: its
    // waves go first when leaves' bonus keys share the SIMDs
    __builtin_amdgcn_s_setprio(2);
    // the children's values, for the constants, on their way during pass A
    VChildVals cv{0.0f, 0.0f};
    if (tid < 64) cv = load_child_vals<TT>(vp, sitem);
    // pass A: the chunk's maxima, then its sums relative to them; the draft
    // sum leaves every child out.  The target quads then move to LDS.
    float mt = kNegInf, mz = kNegInf;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mt = fmaxf(mt, tquad_at(tq[q], e) * c);
        mz = fmaxf(mz, zq[q][e] * c);
      }
    mt = block_max(mt, redv);
    mz = block_max(mz, redv);
    const float mts = mt > kNegInf ? mt : 0.0f, mzs = mz > kNegInf ? mz : 0.0f;
    float st = 0.0f, snc = 0.0f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
      for (int e = 0; e < 4; ++e) st += exp2_fast(tquad_at(tq[q], e) * c - mts);
      tl[q * kVerifyThreads + tid] = tq[q];
    }
    if (nloc == 0) {
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) snc += exp2_fast(zq[q][e] * c - mzs);
    } else {
      // bit 4 q + e: the thread's token (q, e) is a child, left out of the sum
      uint64_t cmask = 0;
      for (int k = 0; k < nloc; ++k) {
        const int at = loc[k] - b0;
        if (at >= 0 && at < 1024 * NQ && (at & 1023) < 4) cmask |= 1ull << (4 * (at >> 10) + (at & 3));
      }
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = exp2_fast(zq[q][e] * c - mzs);
          snc += ((cmask >> (4 * q + e)) & 1) ? 0.0f : x;
        }
    }
    const double dst = block_sum_f64((double)st, redd);
    const double dsnc = block_sum_f64((double)snc, redd);
    if (tid == 0) {
      put_slot(f, it, ck, kSlotPA, __float_as_uint(mt));
      put_slot(f, it, ck, kSlotPA + 1, __float_as_uint(mz));
      put_slot(f, it, ck, kSlotPA + 2, __float_as_uint((float)dst));
      put_slot(f, it, ck, kSlotPA + 3, __float_as_uint((float)dsnc));
    }
    // every workgroup: the item's constants and the test of child 1
    if (tid < 64) {
      const int lane = tid;
      uint32_t w[4];
      const bool ok = poll_slots<4>(f, it, kSlotPA, w);
      if (ok) {
        const VConstLane C = verify_consts_lane<TT>(vp, sitem, f.cpi, [&](int) {
          VPartA a;
          a.mt = __uint_as_float(w[0]);
          a.mz = __uint_as_float(w[1]);
          a.st = (double)__uint_as_float(w[2]);
          a.snc = (double)__uint_as_float(w[3]);
          return a;
        }, cv);
        if (lane < m) {
          sC.lp[lane] = C.lp;
          sC.lq[lane] = C.lq;
          sC.lR[lane] = C.lR;
          sC.invR[lane] = C.invR;
          sC.lu[lane] = C.lu;
        }
        if (lane == 0) {
          sC.Lt = C.Lt;
          sC.Lz = C.Lz;
          shr = stage_test(C.lp, C.lq, C.lR, C.invR, C.lu, 1, 1.0f, 0.0f, __builtin_huge_valf());
        }
      }
      if (lane == 0) sh_ok = ok ? 1 : 0;
    }
    __syncthreads();
    alive = sh_ok != 0;
    if (alive) {
      rec = shr;
      const float Lt = sC.Lt, Lz = sC.Lz;
      // the draft quads become q = 2^(z c - Lz) (zero outside the chunk); p =
      // 2^(t c - Lt) is taken from the LDS quads in each sweep
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) zq[q][e] = exp2_fast(zq[q][e] * c - Lz);
      // stage j rejected: Z_j over the tokens not drawn up to j; at the last
      // child the same residual also gives the bonus keys
      for (int j = 1; rec.status == kRejected; ++j) {
        if (nloc) {
          for (int k = 0; k < nloc; ++k) {
            if (locj[k] != j) continue;
            // the drawn child leaves the sums: q = 0 and t = -inf
            const int at = loc[k] - b0;
#pragma unroll
            for (int q = 0; q < NQ; ++q)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (1024 * q + e == at) {
                  zq[q][e] = 0.0f;
                  Q t = tl[q * kVerifyThreads + tid];
                  if constexpr (sizeof(TT) == 2) {
                    uint32_t& x = (e < 2) ? t.x : t.y;
                    x = (e & 1) ? ((x & 0xFFFFu) | 0xFF800000u) : ((x & 0xFFFF0000u) | 0xFF80u);
                  } else {
                    t[e] = kNegInf;
                  }
                  tl[q * kVerifyThreads + tid] = t;
                }
          }
        }
        const float a = rec.alpha, bb = rec.betap;
        if (j == m) {
          BonusTop bt;
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            if (b0 + 1024 * q >= y1) break;
            const Q t = tl[q * kVerifyThreads + tid];
            int bq = b0 + 1024 * q;
            asm volatile("" : "+v"(bq) : "v"(bt.best));
            uint32_t w[4];
            bonus_words(w, bq, pc1, pc2, c3, vp.keys);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float r = a * exp2_fast(tquad_at(t, e) * c - Lt) - bb * zq[q][e];
              if (r > 0.0f) bt.add(__builtin_amdgcn_logf(r) + gumbel_neg(w[e]), b0 + 1024 * q + e);
            }
          }
          float vb = bt.best;
          int id = bt.idx;
          block_argmax(vb, id, redv, redi);
          float s2 = (bt.idx == id) ? bt.second : bt.best;
          s2 = block_max(s2, redv);
          if (tid == 0) {
            put_slot(f, it, ck, kSlotB, __float_as_uint(vb));
            put_slot(f, it, ck, kSlotB + 1, __float_as_uint(s2));
            put_slot(f, it, ck, kSlotB + 2, (uint32_t)id);
          }
          rec.status = kExhausted;
          rec.stage = j + 1;
          bonus = true;
          break;
        }
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const Q t = tl[q * kVerifyThreads + tid];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc += fmaxf(a * exp2_fast(tquad_at(t, e) * c - Lt) - bb * zq[q][e], 0.0f);
        }
        const double z = block_sum_f64((double)acc, redd);
        if (tid == 0) put_slot(f, it, ck, kSlotZ + j - 1, __float_as_uint((float)z));
        if (tid < 64) {
          uint32_t w[1];
          const bool ok = poll_slots<1>(f, it, kSlotZ + j - 1, w);
          if (ok) {
            const double Z = wave_sum_f64(tid < f.cpi ? (double)__uint_as_float(w[0]) : 0.0);
            const VRec nr = verify_advance(rec, Z, child_consts(sC, j), m, j + 1);
            if (tid == 0) shr = nr;
          }
          if (tid == 0) sh_ok = ok ? 1 : 0;
        }
        __syncthreads();
        alive = sh_ok != 0;
        if (!alive) break;
        rec = shr;
      }
    }
  }
  // an accepted child without children ends the walk there: its bonus comes
  // from its own target row, drawn here instead of at the next level
  bool leaf_next = false;
  if (alive && m > 0 && rec.status == kAccepted && ((snext.leaf_mask >> (rec.stage - 1)) & 1u)) {
    leaf_next = true;
    const int cn = snext.child_node[rec.stage - 1];
    const TT* crow = static_cast<const TT*>(vp.target) + ((size_t)sitem.request * vp.cap + cn) * vp.V;
    Q cq[NQ];
    f32x4 unused[NQ];
    if (vector_rows<TT>(vp)) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) load_quad_vec<TT>(crow, nullptr, b0 + 1024 * q, y1, cq[q], unused[q]);
    } else {
#pragma unroll
      for (int q = 0; q < NQ; ++q) load_quad_tok<TT>(crow, nullptr, b0 + 1024 * q, y1, cq[q], unused[q]);
    }
    leaf_keys(cq, b0, y1, c, snext.child_path[rec.stage - 1], counter_word3(sitem.request, sitem.depth + 1, 3u),
              vp, f, it, ck, redv, redi);
    bonus = true;
  }
  // chunk 0 writes the item's result: the accepted child, or the bonus token
  // from the chunks' best keys, or both
  if (ck == 0 && alive && tid < 64) {
    uint32_t w[3] = {0u, 0u, 0u};
    const bool ok = bonus ? poll_slots<3>(f, it, kSlotB, w) : true;
    if (ok) {
      VRec rr = rec;
      if (leaf_next) rr.status = kExhausted;  // the bonus part of the result
      VerifyResult r = verify_result(rr, f.cpi, [&](int) {
        VBonusPart b;
        b.best = __uint_as_float(w[0]);
        b.second = __uint_as_float(w[1]);
        b.idx = (int32_t)w[2];
        b.pad = 0;
        return b;
      });
      if (leaf_next) {
        r.accepted = rec.stage;
        r.leaf_bonus = 1;
      }
      // pinned host memory, read by the host after it synchronises the stream
      if (tid == 0) vp.results[it] = r;
    }
  }
}

}  // namespace ts
