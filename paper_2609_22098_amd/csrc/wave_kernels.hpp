// Device-resident waves of ts_build_tree: best-first control on the GPU.
//
// The branch-and-bound waves of Algorithm 1 (§3.2; the price stop of §3.5)
// run without host round trips.  After a wave's expansion, one workgroup per
// request merges the wave's children into the request's list of its best N
// known slots (pop order: key desc, child depth asc, child path asc) and
// appends to the next wave's frontier the children that may still become
// nodes: key >= log(theta), rank strictly above the request's N-th known
// slot (any rank while fewer than N are known), depth < D.  A slot that
// misses this never qualifies later, since ranks only grow as slots become
// known, so a wave's frontier is always children of the previous wave.
// Every node of the final tree descends from such a child, because a slot's
// key never exceeds the key of the slot whose pop created it.
//
// The frontier is appended per request at an offset taken with one atomic
// add; the order of requests in a frontier may change from run to run, but
// no result does, since every draw is keyed by the parent's path (not its
// row).  At the end one workgroup per request writes its tree: the list in
// pop order, each node's parent found by its path prefix.
#pragma once

#include "wave_params.hpp"

namespace ts {

__device__ __forceinline__ bool wslot_before(const WaveSlot& a, const WaveSlot& b) {
  if (a.key != b.key) return a.key > b.key;
  if (a.depth != b.depth) return a.depth < b.depth;
  return a.path < b.path;
}

// Exclusive scan of one int per thread of the workgroup (total: the sum of
// all): a shuffle scan inside each wave, then the wave totals in wave order.
// tmp: at least kWaveThreads / 64 ints of LDS.
__device__ __forceinline__ int wave_block_excl_scan(int v, int* tmp, int& total) {
  constexpr int kW = kWaveThreads / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();  // tmp free (a previous scan's readers are done)
  if (lane == 63) tmp[wv] = x;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kW; ++w) {
    const int tw = tmp[w];
    before += w < wv ? tw : 0;
    total += tw;
  }
  return before + x - v;
}

// Wave 0: every request's root is the one parent; lists empty.  The roots
// and thresholds are read from the host's pinned buffer (no upload copy).
__global__ __launch_bounds__(kWaveThreads) void wave_init_kernel(const WaveParams wp) {
  const int q = blockIdx.x * kWaveThreads + threadIdx.x;
  if (q == 0) {
    for (int i = 0; i < wp.D + 2; ++i) wp.pcount[i] = i == 0 ? (uint64_t)wp.R : 0ull;
  }
  if (q >= wp.R) return;
  const int32_t a = wp.anchor_host[q];
  wp.anchor_w[q] = a;
  wp.log_theta_w[q] = wp.log_theta_host[q];
  wp.lsize[q] = 0;
  wp.evals[q] = 0;
  wp.par[0][q] = ts_parent{a, 0, q, 0.0f, 0ull};
  wp.span[0][q] = WaveSpan{q, 1};
}

// After wave w's expansion: one workgroup per request.  The host guarantees
// N <= kWaveMaxN and (parents of a request in a wave) x K <= kWaveMaxNew.
__global__ __launch_bounds__(kWaveThreads) void wave_control_kernel(const WaveParams wp, int w) {
  __shared__ WaveSlot Ls[kWaveMaxN];
  __shared__ WaveSlot Ns[kWaveMaxNew];
  __shared__ int rank_l[kWaveMaxN];
  __shared__ int rank_n[kWaveMaxNew];
  __shared__ int order[kWaveMaxNew];  // the new children's indices in pop order
  __shared__ int tmp[kWaveThreads];
  __shared__ int base_sh;
  const int q = blockIdx.x, t = threadIdx.x;
  const int N = wp.N, K = wp.K;
  const WaveSpan sp = wp.span[w & 1][q];
  const ts_parent* par = wp.par[w & 1];
  const int s = wp.lsize[q];
  const float lt = wp.log_theta[q];
  WaveSlot* lq = wp.list + (size_t)q * N;
  for (int i = t; i < s; i += kWaveThreads) Ls[i] = lq[i];

  // the request's children of this wave with key >= log(theta), in (row, child) order
  const int mraw = sp.cnt * K;
  const int per = (mraw + kWaveThreads - 1) / kWaveThreads;
  const int k0 = min(t * per, mraw), k1 = min(k0 + per, mraw);
  int c = 0;
  for (int k = k0; k < k1; ++k) c += wp.slot_key[(size_t)sp.off * K + k] >= lt ? 1 : 0;
  int m = 0;
  int pos = wave_block_excl_scan(c, tmp, m);
  for (int k = k0; k < k1; ++k) {
    const size_t o = (size_t)sp.off * K + k;
    const float key = wp.slot_key[o];
    if (!(key >= lt)) continue;
    const ts_parent pa = par[sp.off + k / K];
    const int j = k % K;
    WaveSlot sl;
    sl.key = key;
    sl.depth = pa.depth + 1;
    sl.path = pa.path | ((uint64_t)j << (4 * pa.depth));
    sl.token = wp.child_token[o];
    sl.log_surv = wp.child_log_surv[o];
    sl.log_q0 = wp.child_log_q0[o];
    sl.log_qT = wp.child_log_qT[o];
    Ns[pos++] = sl;
  }
  __syncthreads();

  // The new children in pop order: a bitonic sort of their indices over the
  // next power of two (entries past m sort last).  Slots are distinct (their
  // paths differ), so the order is total and the sort's result unique.
  int M = 1;
  while (M < m) M <<= 1;
  for (int k = t; k < M; k += kWaveThreads) order[k] = k;
  __syncthreads();
  auto before_idx = [&](int a, int b) {  // a ahead of b in pop order, indices past m last
    if (a >= m) return false;
    if (b >= m) return true;
    return wslot_before(Ns[a], Ns[b]);
  };
  for (int k = 2; k <= M; k <<= 1) {
    for (int jj = k >> 1; jj > 0; jj >>= 1) {
      for (int i = t; i < M / 2; i += kWaveThreads) {
        const int lo = 2 * i - (i & (jj - 1)), hi = lo + jj;
        const int a = order[lo], b = order[hi];
        const bool asc = (lo & k) == 0;
        if (asc ? before_idx(b, a) : before_idx(a, b)) {
          order[lo] = b;
          order[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  // ranks in the merged pop order: a new child's place among the new ones
  // plus the list slots ahead of it, and a list slot's place in the list
  // plus the new children ahead of it (binary searches in sorted sequences)
  for (int k = t; k < m; k += kWaveThreads) {
    const int e = order[k];
    const WaveSlot a = Ns[e];
    int lo = 0, hi = s;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (wslot_before(Ls[mid], a)) lo = mid + 1; else hi = mid;
    }
    rank_n[e] = k + lo;
  }
  for (int i = t; i < s; i += kWaveThreads) {
    const WaveSlot a = Ls[i];
    int lo = 0, hi = m;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (wslot_before(Ns[order[mid]], a)) lo = mid + 1; else hi = mid;
    }
    rank_l[i] = i + lo;
  }
  __syncthreads();
  const int total = s + m;
  for (int i = t; i < s; i += kWaveThreads)
    if (rank_l[i] < N) lq[rank_l[i]] = Ls[i];
  for (int k = t; k < m; k += kWaveThreads)
    if (rank_n[k] < N) lq[rank_n[k]] = Ns[k];
  if (t == 0) {
    wp.lsize[q] = min(N, total);
    wp.evals[q] += sp.cnt;
  }

  // next frontier: this wave's children ranked strictly above the N-th known slot
  const int limit = total >= N ? N - 1 : total;
  const int per2 = (m + kWaveThreads - 1) / kWaveThreads;
  const int a0 = min(t * per2, m), a1 = min(a0 + per2, m);
  int cc = 0;
  for (int k = a0; k < a1; ++k) cc += (rank_n[k] < limit && Ns[k].depth < wp.D) ? 1 : 0;
  int nc = 0;
  int cpos = wave_block_excl_scan(cc, tmp, nc);
  if (t == 0) {
    // one atomic reserves this request's rows and counts it as done (the
    // frontier size in the low half, finished workgroups in the high half)
    const uint64_t old = atomicAdd(&wp.pcount[w + 1], (1ull << 32) | (uint64_t)nc);
    const int base = (int)(uint32_t)old;
    base_sh = base;
    wp.span[(w + 1) & 1][q] = WaveSpan{base, nc};
    // the last workgroup to finish knows the final size and hands it to the
    // host with a system-scope store.  Only the count goes to the host (the
    // lists and parents reach the next wave's kernels across the launch
    // boundary).
    if ((int)(old >> 32) == wp.R - 1)
      __hip_atomic_store(const_cast<int32_t*>(wp.host_count + w + 1), base + nc, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
  }
  __syncthreads();
  ts_parent* out = wp.par[(w + 1) & 1] + base_sh;
  for (int k = a0; k < a1; ++k)
    if (rank_n[k] < limit && Ns[k].depth < wp.D) {
      const WaveSlot& sl = Ns[k];
      out[cpos++] = ts_parent{sl.token, sl.depth, q, sl.log_surv, sl.path};
    }
}

// One tree row into one output.
__device__ __forceinline__ void put_tree_row(const WaveTreeOut& o, size_t i, int32_t tok, int32_t parent, int32_t depth,
                                             int32_t rank, uint64_t path, float ls, float lq0, float lqT, float key) {
  o.token[i] = tok;
  o.parent[i] = parent;
  o.depth[i] = depth;
  o.rank[i] = rank;
  o.path[i] = path;
  o.log_surv[i] = ls;
  o.log_q0[i] = lq0;
  o.log_qT[i] = lqT;
  o.key[i] = key;
}

// The trees: node 0 is the root, nodes 1..n the list in pop order; rows past
// n get parent -1, token -1 and NaN values.  Written to o, and to o2 as well
// when o2.n is not null (one pass for the host's copy and a device copy).
__global__ __launch_bounds__(kWaveThreads) void wave_tree_kernel(const WaveParams wp, const WaveTreeOut o,
                                                                 const WaveTreeOut o2) {
  __shared__ int dep[kWaveMaxN + 1];
  __shared__ uint64_t pth[kWaveMaxN + 1];
  const int q = blockIdx.x, t = threadIdx.x;
  const int s = wp.lsize[q], cap = o.cap;
  const WaveSlot* lq = wp.list + (size_t)q * wp.N;
  if (t == 0) {
    dep[0] = 0;
    pth[0] = 0ull;
  }
  for (int i = t; i < s; i += kWaveThreads) {
    dep[i + 1] = lq[i].depth;
    pth[i + 1] = lq[i].path;
  }
  __syncthreads();
  const size_t b = (size_t)q * cap;
  const float nan = __builtin_nanf("");
  for (int c = t; c < cap; c += kWaveThreads) {
    int32_t tok = -1, parent = -1, depth = 0, rank = 0;
    uint64_t path = 0ull;
    float ls = nan, lq0 = nan, lqT = nan, key = nan;
    if (c == 0) {
      tok = wp.anchor[q];
      ls = 0.0f;
      lq0 = 0.0f;
      key = 0.0f;
    } else if (c <= s) {
      const WaveSlot sl = lq[c - 1];
      const int pd = sl.depth - 1;
      if (pd == 0) {
        parent = 0;
      } else {
        const uint64_t pp = sl.path & ((1ull << (4 * pd)) - 1ull);
        for (int j = 1; j < c; ++j)
          if (dep[j] == pd && pth[j] == pp) {
            parent = j;
            break;
          }
      }
      if (parent < 0 && o.err) *o.err = 1;
      tok = sl.token;
      depth = sl.depth;
      rank = (int)((sl.path >> (4 * pd)) & 15ull) + 1;
      path = sl.path;
      ls = sl.log_surv;
      lq0 = sl.log_q0;
      lqT = sl.log_qT;
      key = sl.key;
    }
    put_tree_row(o, b + c, tok, parent, depth, rank, path, ls, lq0, lqT, key);
    if (o2.n) put_tree_row(o2, b + c, tok, parent, depth, rank, path, ls, lq0, lqT, key);
  }
  if (t == 0) {
    o.n[q] = s;
    if (o.evals) o.evals[q] = wp.evals[q];
    if (o2.n) {
      o2.n[q] = s;
      if (o2.evals) o2.evals[q] = wp.evals[q];
    }
  }
}

}  // namespace ts
