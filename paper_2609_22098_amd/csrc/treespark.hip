// C ABI of the TreeSpark draft-tree step: argument checks, launch plans,
// the best-first wave builder and the verification drivers.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "launch.hpp"
#include "verify_fused.hpp"

// The scratch of ts_expand_noalloc, one copy per GPU.  In host code `scratch`
// names a host-side stand-in, not device memory: kernels get the device
// address that hipGetSymbolAddress returns, taken once per device with that
// device current (noalloc_scratch below).
static __device__ __align__(256) char scratch[TS_NOALLOC_SCRATCH_BYTES];

namespace ts {
namespace {

thread_local std::string g_last_error;

int32_t fail(int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

#define TS_HIP(call)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) return fail(TS_EHIP, "%s: %s", #call, hipGetErrorString(e_));  \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Armed once work is queued on a stream: an error return then waits for that
// work, so that no kernel or copy is still writing the caller's workspace or
// the staging buffer when the call returns.  Success paths disarm it.
struct DrainOnError {
  hipStream_t s;
  bool armed = true;
  ~DrainOnError() {
    if (armed) (void)hipStreamSynchronize(s);
  }
};

// Page-locked host staging for the small transfers of the host loops, so that
// they are true asynchronous DMA copies (kernels also read and write parts of
// it directly).  It belongs to the calling host thread, grows on demand and
// lives until ts_release_thread_state() frees it; every user synchronises its
// stream before it rewrites or grows the buffer.  There is deliberately no
// destructor: a thread-exit destructor of the main thread would run inside
// exit(), after the HIP runtime (and any profiler attached to it) may have
// been torn down.
struct ThreadState {
  char* stage = nullptr;
  size_t stage_bytes = 0;
  // T > 0 verification levels run in one launch, run again through the
  // per-stage launches after a wait ran out, and run per stage from the start
  int64_t fused_levels = 0, fused_fallbacks = 0, staged_levels = 0;
  int32_t verify_mode = TS_VERIFY_AUTO;
};
ThreadState& thread_state() {
  thread_local ThreadState st;
  return st;
}

int32_t host_stage(size_t bytes, char** out) {
  ThreadState& st = thread_state();
  if (st.stage_bytes < bytes) {
    if (st.stage) TS_HIP(hipHostFree(st.stage));
    st.stage = nullptr;
    st.stage_bytes = 0;
    void* q = nullptr;
    // coherent: kernels read and write parts of it directly
    TS_HIP(hipHostMalloc(&q, bytes, hipHostMallocCoherent));
    st.stage = static_cast<char*>(q);
    st.stage_bytes = bytes;
  }
  *out = st.stage;
  return TS_OK;
}

// ---------------------------------------------------------------- checks

int32_t check_drafter(const ts_drafter* d) {
  if (!d) return fail(TS_EINVAL, "drafter is NULL");
  if (!d->U || !d->E || !d->W2) return fail(TS_EINVAL, "drafter tensor pointer is NULL");
  if (d->R <= 0 || d->D <= 0 || d->V <= 0 || d->r <= 0)
    return fail(TS_EINVAL, "drafter sizes must be positive (R=%d D=%d V=%d r=%d)", d->R, d->D, d->V, d->r);
  if (d->dtype != TS_F32 && d->dtype != TS_BF16) return fail(TS_EINVAL, "unknown dtype %d", d->dtype);
  if (((reinterpret_cast<uintptr_t>(d->U) | reinterpret_cast<uintptr_t>(d->E) |
        reinterpret_cast<uintptr_t>(d->W2)) & 15) != 0)
    return fail(TS_EINVAL, "U, E and W2 must start at 16-byte aligned addresses");
  if (d->D > TS_MAX_D) return fail(TS_EUNSUPPORTED, "D=%d exceeds %d (4-bit path digits)", d->D, TS_MAX_D);
  if (d->R >= TS_MAX_R) return fail(TS_EUNSUPPORTED, "R=%d exceeds %d", d->R, TS_MAX_R - 1);
  if (d->V > TS_MAX_V) return fail(TS_EUNSUPPORTED, "V=%d exceeds %d", d->V, TS_MAX_V);
  const bool ok = d->dtype == TS_BF16 ? (d->r == 32 || d->r == 64 || d->r == 128 || d->r == 256)
                                      : (d->r == 16 || d->r == 32 || d->r == 64);
  if (!ok) return fail(TS_EUNSUPPORTED, "rank r=%d not supported for dtype %d", d->r, d->dtype);
  return TS_OK;
}

int32_t check_k_T(const ts_drafter* d, int32_t k, float T) {
  if (k < 1 || k > TS_MAX_K) return fail(k < 1 ? TS_EINVAL : TS_EUNSUPPORTED, "k=%d outside [1, %d]", k, TS_MAX_K);
  if (k > d->V) return fail(TS_EINVAL, "k=%d exceeds V=%d", k, d->V);
  if (!(T >= 0.0f) || !std::isfinite(T)) return fail(TS_EINVAL, "T must be finite and >= 0");
  return TS_OK;
}

int32_t check_sampler(int32_t sampler) {
  if (sampler != TS_SAMPLER_GUMBEL && sampler != TS_SAMPLER_SEQUENTIAL)
    return fail(TS_EINVAL, "unknown sampler %d", sampler);
  return TS_OK;
}

PhiloxKeys philox_keys(uint64_t seed) {
  PhiloxKeys k;
  uint32_t a = (uint32_t)seed, b = (uint32_t)(seed >> 32);
  for (int r = 0; r < 10; ++r) {
    k.k0[r] = a;
    k.k1[r] = b;
    a += 0x9E3779B9u;
    b += 0xBB67AE85u;
  }
  return k;
}

// ---------------------------------------------------------------- expansion plan

struct Plan {
  int NB, Vc, S, n_pblocks, wpg, n_pgroups, S8;
  int ks;
  int mode;     // kModeGreedy, kModeGumbel or kModeSeq (the kernels' mode)
  bool sample;  // T > 0: the merge takes lse of z/T and draws
  bool lds;     // LDS-staged bf16 streaming kernel
  int nblk;     // 64-token blocks of the vocabulary
  int blk_ld;   // row stride of the block table (nblk rounded up to 16)
  size_t off_m, off_s0, off_sT, off_z[2], off_g[2], off_blk;
  size_t bytes;
};

// Compute units of the current device (256 when no device answers).
int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Resident blocks per CU of the streaming kernel for this plan (2 if unknown).
int eval_blocks_per_cu(int dtype, int ks, int nb, int mode, bool store_z, bool lds, int block) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int, int, bool, bool, int>, int> cache;
  const auto key = std::make_tuple(dtype, ks, nb, mode, store_z, lds, block);
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  int n = 0;
  if (dtype == TS_BF16) {
    switch (ks) {
      case 1: n = eval_blocks_per_cu_t<uint16_t, 1>(nb, mode, store_z, lds, block); break;
      case 2: n = eval_blocks_per_cu_t<uint16_t, 2>(nb, mode, store_z, lds, block); break;
      case 4: n = eval_blocks_per_cu_t<uint16_t, 4>(nb, mode, store_z, lds, block); break;
      default: n = eval_blocks_per_cu_t<uint16_t, 8>(nb, mode, store_z, lds, block); break;
    }
  } else {
    switch (ks) {
      case 4: n = eval_blocks_per_cu_t<float, 4>(nb, mode, store_z, lds, block); break;
      case 8: n = eval_blocks_per_cu_t<float, 8>(nb, mode, store_z, lds, block); break;
      default: n = eval_blocks_per_cu_t<float, 16>(nb, mode, store_z, lds, block); break;
    }
  }
  if (n <= 0) n = 2;
  std::lock_guard<std::mutex> lock(mu);
  cache[key] = n;
  return n;
}

// Launch plan of one expansion.  store_z: the verification recompute, which
// writes the logits, runs one parent block per wave and makes no draws.
// sizing_only: the workspace size, which must not depend on the device or the
// sampler, so it assumes the largest chunk count and room for both samplers.
static_assert(TS_MAX_V <= kMaxChunks * 4096, "the merge holds kMaxChunks chunks of <= 4096 tokens");

// max_chunks: the most chunks the vocabulary allows (the plan of a launch
// whose parent count is only bounded on the host: parallelism comes from the
// chunks, and workgroups beyond the parents the device holds exit at once).
Plan make_plan(const ts_drafter* d, int P, float T, int sampler, bool store_z = false,
               bool sizing_only = false, bool max_chunks = false) {
  Plan pl{};
  pl.sample = T > 0.0f && !store_z;
  pl.mode = !pl.sample ? kModeGreedy : sampler == TS_SAMPLER_SEQUENTIAL ? kModeSeq : kModeGumbel;
  // the streaming kernel's mode: with the separate z / T sum when T != 1
  const int eval_mode = pl.mode | (pl.sample && T != 1.0f ? kModeNeedT : 0);
  pl.nblk = (d->V + kBlkTokens - 1) / kBlkTokens;
  pl.blk_ld = ((pl.nblk + 15) / 16) * 16;
  pl.ks = d->dtype == TS_BF16 ? d->r / 32 : d->r / 4;
  // two parent blocks per wave pay off only when the parents fill them; a
  // bound on a device-held count (max_chunks) usually overstates them
  pl.NB = (P >= 512 && !max_chunks) ? 2 : 1;
  if (store_z) pl.NB = 1;
  // the LDS kernel reads U and W2 as raw buffers: byte offsets under 2^31
  pl.lds = d->dtype == TS_BF16 && d->V % 8 == 0 && !store_z &&
           ((uint64_t)d->R * d->D + 1) * d->V * 2 + 64 < (1ull << 31) &&
           (uint64_t)d->V * d->r * 2 < (1ull << 31);
  pl.n_pblocks = (P + 16 * pl.NB - 1) / (16 * pl.NB);
  // waves per workgroup (each workgroup loads every W2 tile of its chunk
  // once): eight for the greedy LDS kernel with two blocks per wave at rank
  // <= 64 (that kernel fits four waves per SIMD), else four
  pl.wpg = pl.lds ? 4 : std::min(4, std::max(1, pl.n_pblocks));
  if (pl.lds && pl.NB == 2 && pl.ks <= 2 && pl.mode == kModeGreedy) pl.wpg = 8;
  pl.n_pgroups = (pl.n_pblocks + pl.wpg - 1) / pl.wpg;
  // Chunks: enough workgroups to fill every CU at the kernel's occupancy in
  // whole rounds (all workgroups of a round finish together), chunks of
  // 256..4096 tokens, at most kMaxChunks per parent.
  int vc;
  if (sizing_only || max_chunks) {
    vc = 256;
  } else {
    const int concurrent = device_cus() *
        eval_blocks_per_cu(d->dtype, pl.ks, pl.NB, eval_mode, store_z, pl.lds, 64 * pl.wpg);
    const int s_min = (d->V + 4095) / 4096;
    const int rounds = std::max(1, (pl.n_pgroups * s_min + concurrent - 1) / concurrent);
    // at most rounds * concurrent workgroups: a few more would take a round of their own
    const int s_want = std::max(1, rounds * concurrent / pl.n_pgroups);
    vc = (d->V + s_want - 1) / s_want;
  }
#ifdef TS_DEBUG_RUNS
  if (!sizing_only && getenv("TS_VC")) vc = atoi(getenv("TS_VC"));
#endif
  vc = std::max(vc, (d->V + kMaxChunks - 1) / kMaxChunks);
  // the LDS kernel sums block masses over quads of steps: chunks of whole quads
  const int quantum = pl.lds ? 256 : 64;
  vc = ((vc + quantum - 1) / quantum) * quantum;
  vc = std::min(std::max(vc, 256), 4096);
  pl.Vc = vc;
  pl.S = (d->V + vc - 1) / vc;
  pl.S8 = ((pl.S + 7) / 8) * 8;
#ifdef TS_DEBUG_RUNS
  if (!sizing_only)
    fprintf(stderr, "[plan] P=%d NB=%d lds=%d wpg=%d n_pgroups=%d Vc=%d S=%d grid=%d bpc=%d cus=%d\n", P,
            pl.NB, (int)pl.lds, pl.wpg, pl.n_pgroups, pl.Vc, pl.S, pl.S8 * pl.n_pgroups,
            eval_blocks_per_cu(d->dtype, pl.ks, pl.NB, eval_mode, store_z, pl.lds, 64 * pl.wpg), device_cus());
#endif
  const size_t a = align256((size_t)std::max(P, 1) * pl.S * 4);
  const size_t a4 = align256((size_t)std::max(P, 1) * pl.S * 4 * kTopRuns);
  size_t o = 0;
  pl.off_m = o; o += a;
  pl.off_s0 = o; o += a;
  pl.off_z[0] = o; o += a4;
  pl.off_z[1] = o; o += a;
  if (pl.sample || (sizing_only && T > 0.0f && !store_z)) {
    pl.off_sT = o; o += a;
    if (pl.mode == kModeGumbel || sizing_only) {
      pl.off_g[0] = o; o += a4;
      pl.off_g[1] = o; o += a;
    }
    if (pl.mode == kModeSeq || sizing_only) {
      pl.off_blk = o; o += align256((size_t)std::max(P, 1) * pl.blk_ld * 4);
    }
  }
  pl.bytes = o;
  return pl;
}

RunSummaryPtr summary_ptr(char* ws, const size_t (&off)[2]) {
  RunSummaryPtr r;
  r.m = reinterpret_cast<float*>(ws + off[0]);
  r.rest = reinterpret_cast<float*>(ws + off[1]);
  return r;
}

size_t expand_ws_max(const ts_drafter* d, int Pmax, float T, bool store_z = false) {
  return make_plan(d, std::max(Pmax, 1), T, TS_SAMPLER_GUMBEL, store_z, true).bytes;
}

void launch_eval(const ts_drafter* d, const ExpandParams& p, const Plan& pl, hipStream_t s) {
  const dim3 grid(pl.S8 * pl.n_pgroups), block(64 * pl.wpg);
  const bool z = p.z_out != nullptr;
  const int mode = pl.mode | (p.need_T && pl.mode != kModeGreedy ? kModeNeedT : 0);
  if (d->dtype == TS_BF16) {
    switch (pl.ks) {
      case 1: launch_eval_t<uint16_t, 1>(p, pl.NB, mode, z, pl.lds, grid, block, s); break;
      case 2: launch_eval_t<uint16_t, 2>(p, pl.NB, mode, z, pl.lds, grid, block, s); break;
      case 4: launch_eval_t<uint16_t, 4>(p, pl.NB, mode, z, pl.lds, grid, block, s); break;
      default: launch_eval_t<uint16_t, 8>(p, pl.NB, mode, z, pl.lds, grid, block, s); break;
    }
  } else {
    switch (pl.ks) {
      case 4: launch_eval_t<float, 4>(p, pl.NB, mode, z, false, grid, block, s); break;
      case 8: launch_eval_t<float, 8>(p, pl.NB, mode, z, false, grid, block, s); break;
      default: launch_eval_t<float, 16>(p, pl.NB, mode, z, false, grid, block, s); break;
    }
  }
}

void launch_merge(const ts_drafter* d, const MergeParams& p, const Plan& pl, hipStream_t s) {
  // one parent per wave; sequential draws: one parent per workgroup of two waves
  const bool seq = pl.mode == kModeSeq;
  const dim3 grid(seq ? p.P : (p.P + 3) / 4), block(seq ? 128 : 256);
  if (d->dtype == TS_BF16) {
    switch (pl.ks) {
      case 1: launch_merge_t<uint16_t, 1>(p, pl.mode, grid, block, s); break;
      case 2: launch_merge_t<uint16_t, 2>(p, pl.mode, grid, block, s); break;
      case 4: launch_merge_t<uint16_t, 4>(p, pl.mode, grid, block, s); break;
      default: launch_merge_t<uint16_t, 8>(p, pl.mode, grid, block, s); break;
    }
  } else {
    switch (pl.ks) {
      case 4: launch_merge_t<float, 4>(p, pl.mode, grid, block, s); break;
      case 8: launch_merge_t<float, 8>(p, pl.mode, grid, block, s); break;
      default: launch_merge_t<float, 16>(p, pl.mode, grid, block, s); break;
    }
  }
}

ExpandParams eval_params(const ts_drafter* d, const ts_parent* parents, int P, float T, uint64_t seed,
                         const Plan& pl, char* ws, float* z_out) {
  ExpandParams p{};
  p.U = d->U; p.E = d->E; p.W2 = d->W2;
  p.R = d->R; p.D = d->D; p.V = d->V; p.r = d->r;
  p.parents = parents;
  p.P = P;
  p.Vc = pl.Vc; p.S = pl.S;
  p.n_pblocks = pl.n_pblocks; p.wpg = pl.wpg; p.n_pgroups = pl.n_pgroups;
  p.cT = T > 0.0f ? kLog2e / T : 0.0f;
  p.need_T = (T > 0.0f && T != 1.0f) ? 1 : 0;
  p.hr = 60.0f / std::max(kLog2e, p.cT);
  p.keys = philox_keys(seed);
  p.part_m = reinterpret_cast<float*>(ws + pl.off_m);
  p.part_s0 = reinterpret_cast<float*>(ws + pl.off_s0);
  p.part_sT = pl.sample ? reinterpret_cast<float*>(ws + pl.off_sT) : nullptr;
  p.zs = summary_ptr(ws, pl.off_z);
  if (pl.mode == kModeGumbel) p.gs = summary_ptr(ws, pl.off_g);
  p.nblk = pl.nblk;
  p.blk_ld = pl.blk_ld;
  if (pl.mode == kModeSeq) p.blk = reinterpret_cast<float*>(ws + pl.off_blk);
  p.z_out = z_out;
  return p;
}

// Both passes of one expansion; all arguments already checked.
// P_dev (optional): the device holds the parent count (<= P); P then sizes
// the grids and the plan takes the most chunks.
int32_t run_expand(const ts_drafter* d, const ts_parent* parents, int P, ts_calib calib, int k,
                   float T, uint64_t seed, int sampler, const ts_expand_out* out, char* ws,
                   hipStream_t s, const int* P_dev = nullptr) {
  if (P == 0) return TS_OK;
  const Plan pl = make_plan(d, P, T, sampler, false, false, P_dev != nullptr);
  ExpandParams ep = eval_params(d, parents, P, T, seed, pl, ws, nullptr);
  ep.P_dev = P_dev;
  hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(out->events);
  if (ev) TS_HIP(hipEventRecord(ev[0], s));
  launch_eval(d, ep, pl, s);
  TS_HIP(hipGetLastError());
  if (ev) TS_HIP(hipEventRecord(ev[1], s));
  MergeParams mp{};
  mp.U = d->U; mp.E = d->E; mp.W2 = d->W2;
  mp.R = d->R; mp.D = d->D; mp.V = d->V; mp.r = d->r;
  mp.parents = parents;
  mp.P = P;
  mp.Vc = pl.Vc; mp.S = pl.S;
  mp.K = k;
  mp.T = T; mp.cT = ep.cT; mp.need_T = ep.need_T;
  mp.calib_a = calib.a; mp.calib_b = calib.b;
  mp.keys = ep.keys;
  mp.part_m = ep.part_m; mp.part_s0 = ep.part_s0; mp.part_sT = ep.part_sT;
  mp.zs = ep.zs;
  mp.gs = ep.gs;
  mp.blk = ep.blk;
  mp.nblk = ep.nblk;
  mp.blk_ld = ep.blk_ld;
  mp.out = *out;
  mp.P_dev = P_dev;
  launch_merge(d, mp, pl, s);
  TS_HIP(hipGetLastError());
  if (ev) TS_HIP(hipEventRecord(ev[2], s));
  return TS_OK;
}

// ---------------------------------------------------------------- tree building

struct Slot {
  float key;
  int depth;       // depth of the child this slot creates
  uint64_t path;   // path id of that child
  int token;
  float log_surv, log_q0, log_qT;
  bool evaluated;  // the child has been evaluated (its own slots are known)
};

// (key desc, child depth asc, child path asc): the pop order of Algorithm 1.
inline bool slot_before(const Slot& a, const Slot& b) {
  if (a.key != b.key) return a.key > b.key;
  if (a.depth != b.depth) return a.depth < b.depth;
  return a.path < b.path;
}

// A slot in the global order of a budget shared by all requests:
// (key desc, request asc, child depth asc, child path asc).
struct GlobalRef {
  float key;
  int q;
  int depth;
  uint64_t path;
};
inline bool global_before(const GlobalRef& a, const GlobalRef& b) {
  if (a.key != b.key) return a.key > b.key;
  if (a.q != b.q) return a.q < b.q;
  if (a.depth != b.depth) return a.depth < b.depth;
  return a.path < b.path;
}

// A tree in the ts_tree layout packed into one block (device staging and
// its host copy): n [R], evals [R], err, then token, parent, depth, rank
// [R][cap] int32, path [R][cap] uint64, log_surv, log_q0, log_qT, key
// [R][cap] float.
struct TreeBlock {
  size_t n, evals, err, token, parent, depth, rank, path, log_surv, log_q0, log_qT, key, bytes;
};

TreeBlock tree_block(int R, int cap) {
  TreeBlock t{};
  const size_t rc = (size_t)R * cap;
  size_t o = 0;
  t.n = o; o += align256((size_t)R * 4);
  t.evals = o; o += align256((size_t)R * 4);
  t.err = o; o += 256;
  t.token = o; o += align256(rc * 4);
  t.parent = o; o += align256(rc * 4);
  t.depth = o; o += align256(rc * 4);
  t.rank = o; o += align256(rc * 4);
  t.path = o; o += align256(rc * 8);
  t.log_surv = o; o += align256(rc * 4);
  t.log_q0 = o; o += align256(rc * 4);
  t.log_qT = o; o += align256(rc * 4);
  t.key = o; o += align256(rc * 4);
  t.bytes = o;
  return t;
}

struct BuildLayout {
  size_t off_par, off_out, off_exp;
  // device-resident waves
  size_t off_par2, off_list, off_lsize, off_evals, off_pcount, off_span, off_anchor, off_ltheta;
  size_t bytes;
  int Pmax;
};

BuildLayout build_layout(const ts_drafter* d, int N, int K, float T) {
  BuildLayout b{};
  const int R = d->R;
  b.Pmax = R * std::max(N, 1);
  const size_t pk = align256((size_t)b.Pmax * K * 4);
  size_t o = 0;
  b.off_par = o; o += align256((size_t)b.Pmax * sizeof(ts_parent));
  b.off_out = o; o += 5 * pk;  // child token, log q0, log qT, log S, key: [P][K] each, packed
  b.off_exp = o; o += expand_ws_max(d, b.Pmax, T);
  b.off_par2 = o; o += align256((size_t)b.Pmax * sizeof(ts_parent));
  b.off_list = o; o += align256((size_t)R * std::max(N, 1) * sizeof(WaveSlot));
  b.off_lsize = o; o += align256((size_t)R * 4);
  b.off_evals = o; o += align256((size_t)R * 4);
  b.off_pcount = o; o += align256((size_t)(d->D + 2) * 8);
  b.off_span = o; o += 2 * align256((size_t)R * sizeof(WaveSpan));
  b.off_anchor = o; o += align256((size_t)R * 4);
  b.off_ltheta = o; o += align256((size_t)R * 4);
  b.bytes = o;
  return b;
}

// The waves run on the device when the per-request lists fit the control
// kernel and no budget is shared across requests.
bool device_waves(int N, int K, int budget) {
  return N >= 1 && budget <= 0 && N <= kWaveMaxN && std::max(1, N - 1) * K <= kWaveMaxNew;
}

WaveTreeOut tree_out_of(const ts_tree* t) {
  WaveTreeOut o{};
  o.cap = t->cap;
  o.n = t->n; o.token = t->token; o.parent = t->parent; o.depth = t->depth; o.rank = t->rank;
  o.path = t->path; o.log_surv = t->log_surv; o.log_q0 = t->log_q0; o.log_qT = t->log_qT;
  o.key = t->key; o.evals = t->evals;
  return o;
}

// ts_build_tree with the waves on the device (no budget; N, K within the
// control kernel's limits).  Wave w + 1 is queued before the host learns
// its size (its kernels read the size the control step wrote), so the GPU
// never waits for the host between waves; the host reads each wave's size
// from the pinned word the control step writes and stops queueing at the
// first empty wave.
int32_t build_tree_device(const ts_drafter* d, const int32_t* anchor, const std::vector<float>& log_theta,
                          int N, int K, ts_calib calib, float T, uint64_t seed, int sampler, ts_tree* out,
                          const ts_tree* device_out, char* ws, const BuildLayout& bl, hipStream_t s) {
  const int R = d->R, D = d->D, cap = out->cap;
  const TreeBlock tb = tree_block(R, cap);
  char* hs = nullptr;
  const size_t hs_up = align256((size_t)R * 8), hs_cnt = align256((size_t)(D + 2) * 4);
  int32_t rc = host_stage(hs_up + hs_cnt + tb.bytes, &hs);
  if (rc != TS_OK) return rc;
  // roots and thresholds stay in the pinned buffer: the init kernel reads them
  std::memcpy(hs, anchor, (size_t)R * 4);
  std::memcpy(hs + (size_t)R * 4, log_theta.data(), (size_t)R * 4);
  volatile int32_t* hcnt = reinterpret_cast<volatile int32_t*>(hs + hs_up);
  char* htree = hs + hs_up + hs_cnt;

  WaveParams wp{};
  wp.R = R; wp.N = N; wp.K = K; wp.D = D;
  wp.anchor = reinterpret_cast<const int32_t*>(ws + bl.off_anchor);
  wp.log_theta = reinterpret_cast<const float*>(ws + bl.off_ltheta);
  wp.anchor_host = reinterpret_cast<const int32_t*>(hs);
  wp.log_theta_host = reinterpret_cast<const float*>(hs + (size_t)R * 4);
  wp.anchor_w = reinterpret_cast<int32_t*>(ws + bl.off_anchor);
  wp.log_theta_w = reinterpret_cast<float*>(ws + bl.off_ltheta);
  wp.host_count = hcnt;
  wp.list = reinterpret_cast<WaveSlot*>(ws + bl.off_list);
  wp.lsize = reinterpret_cast<int*>(ws + bl.off_lsize);
  wp.evals = reinterpret_cast<int*>(ws + bl.off_evals);
  wp.pcount = reinterpret_cast<uint64_t*>(ws + bl.off_pcount);
  wp.par[0] = reinterpret_cast<ts_parent*>(ws + bl.off_par);
  wp.par[1] = reinterpret_cast<ts_parent*>(ws + bl.off_par2);
  wp.span[0] = reinterpret_cast<WaveSpan*>(ws + bl.off_span);
  wp.span[1] = reinterpret_cast<WaveSpan*>(ws + bl.off_span + align256((size_t)R * sizeof(WaveSpan)));
  const size_t nk = (size_t)bl.Pmax * K;
  char* dout = ws + bl.off_out;
  ts_expand_out eo{};
  eo.child_token = reinterpret_cast<int32_t*>(dout);
  eo.child_log_q0 = reinterpret_cast<float*>(dout + align256(nk * 4));
  eo.child_log_qT = reinterpret_cast<float*>(dout + 2 * align256(nk * 4));
  eo.child_log_surv = reinterpret_cast<float*>(dout + 3 * align256(nk * 4));
  eo.slot_key = reinterpret_cast<float*>(dout + 4 * align256(nk * 4));
  wp.child_token = eo.child_token;
  wp.child_log_q0 = eo.child_log_q0;
  wp.child_log_qT = eo.child_log_qT;
  wp.child_log_surv = eo.child_log_surv;
  wp.slot_key = eo.slot_key;
  DrainOnError drain{s};
  launch_wave_init(wp, s);
  TS_HIP(hipGetLastError());

  // queue wave w: expansion of par[w & 1] (at most Pub parents; the device
  // holds the count) and the control step, which also writes the next
  // wave's size into hcnt[w + 1] (pinned, -1 until then).  The host polls
  // that word: an event recorded between the waves' kernels would hold the
  // next kernel back by about 6 us on the device.
  for (int i = 0; i < D + 2; ++i) hcnt[i] = -1;
  auto queue_wave = [&](int w, int Pub) -> int32_t {
    int32_t r = run_expand(d, wp.par[w & 1], Pub, calib, K, T, seed, sampler, &eo, ws + bl.off_exp, s,
                           reinterpret_cast<const int*>(wp.pcount + w));
    if (r != TS_OK) return r;
    launch_wave_control(wp, w, s);
    TS_HIP(hipGetLastError());
    return TS_OK;
  };
  // the size of wave i from its word.  After 20 ms the wait also asks the
  // stream (a stream query enqueues a marker, which would hold the next
  // kernel back like an event): one that has drained or failed without
  // writing the word ends it
  auto wave_size = [&](int i, int* out_n) -> int32_t {
    const auto t0 = std::chrono::steady_clock::now();
    for (unsigned n = 1;; ++n) {
      const int v = hcnt[i];
      if (v >= 0) {
        *out_n = v;
        return TS_OK;
      }
      if ((n & 4095) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(20)) {
        const hipError_t q = hipStreamQuery(s);
        if (q != hipSuccess && q != hipErrorNotReady) return fail(TS_EHIP, "HIP error %d while waiting for wave %d", (int)q, i);
        if (q == hipSuccess && hcnt[i] < 0) return fail(TS_EINTERNAL, "wave %d ended without its size", i);
      }
    }
  };
  const int per_req = std::max(0, N - 1);  // children a request can send to the next wave
  int Pw = R;                              // size of wave w, known
  if ((rc = queue_wave(0, R)) != TS_OK) return rc;
  for (int w = 0;; ++w) {
    const long long ub = std::min<long long>((long long)Pw * K, (long long)R * per_req);
    if (w + 1 < D && ub > 0)
      if ((rc = queue_wave(w + 1, (int)ub)) != TS_OK) return rc;
    int Pn = 0;
    if ((rc = wave_size(w + 1, &Pn)) != TS_OK) return rc;
    if (Pn <= 0 || w + 1 >= D || ub == 0) break;
    if (Pn > ub) return fail(TS_EINTERNAL, "wave %d has %d parents, more than the bound %lld", w + 1, Pn, ub);
    Pw = Pn;
  }

  // the trees: written straight into the pinned block, and into the caller's
  // device arrays
  char* dt = htree;
  *reinterpret_cast<volatile int32_t*>(htree + tb.err) = 0;
  ts_tree st{};
  st.R = R; st.cap = cap;
  st.n = reinterpret_cast<int32_t*>(dt + tb.n);
  st.evals = reinterpret_cast<int32_t*>(dt + tb.evals);
  st.token = reinterpret_cast<int32_t*>(dt + tb.token);
  st.parent = reinterpret_cast<int32_t*>(dt + tb.parent);
  st.depth = reinterpret_cast<int32_t*>(dt + tb.depth);
  st.rank = reinterpret_cast<int32_t*>(dt + tb.rank);
  st.path = reinterpret_cast<uint64_t*>(dt + tb.path);
  st.log_surv = reinterpret_cast<float*>(dt + tb.log_surv);
  st.log_q0 = reinterpret_cast<float*>(dt + tb.log_q0);
  st.log_qT = reinterpret_cast<float*>(dt + tb.log_qT);
  st.key = reinterpret_cast<float*>(dt + tb.key);
  WaveTreeOut ho = tree_out_of(&st);
  ho.err = reinterpret_cast<int32_t*>(htree + tb.err);
  // one launch writes the host's copy and, when given, the device copy
  launch_wave_tree(wp, ho, device_out ? tree_out_of(device_out) : WaveTreeOut{}, s);
  TS_HIP(hipGetLastError());
  TS_HIP(hipStreamSynchronize(s));
  if (*reinterpret_cast<const volatile int32_t*>(htree + tb.err) != 0)
    return fail(TS_EINTERNAL, "a tree slot has no materialised parent");
  const size_t rcn = (size_t)R * cap;
  std::memcpy(out->n, htree + tb.n, (size_t)R * 4);
  if (out->evals) std::memcpy(out->evals, htree + tb.evals, (size_t)R * 4);
  std::memcpy(out->token, htree + tb.token, rcn * 4);
  std::memcpy(out->parent, htree + tb.parent, rcn * 4);
  std::memcpy(out->depth, htree + tb.depth, rcn * 4);
  std::memcpy(out->rank, htree + tb.rank, rcn * 4);
  std::memcpy(out->path, htree + tb.path, rcn * 8);
  std::memcpy(out->log_surv, htree + tb.log_surv, rcn * 4);
  std::memcpy(out->log_q0, htree + tb.log_q0, rcn * 4);
  std::memcpy(out->log_qT, htree + tb.log_qT, rcn * 4);
  std::memcpy(out->key, htree + tb.key, rcn * 4);
  drain.armed = false;
  return TS_OK;
}

// The children of every tree node, in creation order, as flat per-request
// lists: node p of request q has count(q, p) children starting at
// first(q, p).  The arrays are kept per thread and reused, so indexing a
// tree allocates nothing once they have grown to its size.
struct KidIndex {
  std::vector<int> off;   // [R][cap + 1]: start of node p's children in list
  std::vector<int> list;  // [R][cap]: child ids, grouped by parent
  int cap = 0;
  const int* first(int q, int p) const { return list.data() + (size_t)q * cap + off[(size_t)q * (cap + 1) + p]; }
  int count(int q, int p) const {
    const size_t o = (size_t)q * (cap + 1) + p;
    return off[o + 1] - off[o];
  }
};

// Builds the index of a tree whose parents were checked (0 <= parent[i] < i).
const KidIndex& kid_index(const ts_tree* t) {
  thread_local KidIndex k;
  const int R = t->R, cap = t->cap;
  k.cap = cap;
  k.off.assign((size_t)R * (cap + 1), 0);
  k.list.resize((size_t)R * cap);
  for (int q = 0; q < R; ++q) {
    const int n = t->n[q];
    int* off = k.off.data() + (size_t)q * (cap + 1);
    const int32_t* par = t->parent + (size_t)q * cap;
    for (int i = 1; i <= n; ++i) ++off[par[i] + 1];
    for (int p = 0; p < cap; ++p) off[p + 1] += off[p];
    // fill in increasing id order, which is creation order; off[p] ends at
    // the start of node p + 1 and is moved back afterwards
    int* list = k.list.data() + (size_t)q * cap;
    for (int i = 1; i <= n; ++i) list[off[par[i]]++] = i;
    for (int p = cap; p > 0; --p) off[p] = off[p - 1];
    off[0] = 0;
  }
  return k;
}

struct VerifyLayout {
  size_t off_rows, off_arg, off_gap, off_items, off_z, off_exp;
  size_t off_pa, off_zp, off_bp, off_cst, off_rec, off_sync, bytes;
  int max_chunks;
};

// Vocabulary chunks per item for the T > 0 passes: about 2048 workgroups in
// all, chunks a multiple of kVChunkQuantum tokens.
void verify_chunks(int V, int nitems, int* nchunks, int* chunk) {
  const int max_chunks = (V + kVChunkQuantum - 1) / kVChunkQuantum;
  int nc = std::min(max_chunks, std::max(1, (2048 + nitems - 1) / std::max(nitems, 1)));
  int len = (V + nc - 1) / nc;
  len = ((len + kVChunkQuantum - 1) / kVChunkQuantum) * kVChunkQuantum;
  *chunk = len;
  *nchunks = (V + len - 1) / len;
}

// Launch shape of a level in one launch (register-resident chunks), or ok =
// false when the level's chunks would not all be resident at once.  Chunks
// are at least kVChunkQuantum tokens long (the partial arrays hold that many
// per item) and at most what a workgroup holds.
struct FusedPlan {
  bool ok;
  int cpi, chunk;
};
// Polls of one wait before it gives up (a poll takes about a microsecond).
constexpr int kFusedSpinLimit = 1 << 16;
FusedPlan fused_plan(int V, int nitems, bool bf16) {
  FusedPlan fp{false, 0, 0};
  const int bpc = verify_fused_blocks_per_cu(bf16);
  if (nitems < 1 || bpc < 1) return fp;
  const long long capacity = (long long)bpc * device_cus();
  const int per_wg = verify_fused_quads(bf16) * kVChunkQuantum;
  const int cpi_min = (V + per_wg - 1) / per_wg;
  if (cpi_min > kFusedMaxCpi || (long long)nitems * cpi_min > std::min<long long>(capacity, kFusedMaxGrid)) return fp;
  const int max_chunks = (V + kVChunkQuantum - 1) / kVChunkQuantum;
  int cpi = (int)std::min<long long>(std::min<long long>(capacity, kFusedMaxGrid) / nitems,
                                     std::min(max_chunks, kFusedMaxChunks));
  cpi = std::max(cpi, cpi_min);
  int chunk = (V + cpi - 1) / cpi;
  chunk = (chunk + 3) / 4 * 4;
  fp.ok = true;
  fp.chunk = chunk;
  fp.cpi = (V + chunk - 1) / chunk;
  return fp;
}

// Slot words of the one-launch levels: kSlotWords per workgroup, for the
// most workgroups a launch over R items can have.
size_t fused_slot_words(int R) {
  return (size_t)kSlotWords * (size_t)std::min<long long>((long long)R * kFusedMaxCpi, kFusedMaxGrid);
}

VerifyLayout verify_layout(const ts_drafter* d, int cap, float T) {
  VerifyLayout v{};
  size_t o = 0;
  if (T == 0.0f) {
    const size_t rows = (size_t)d->R * cap;
    v.off_rows = o; o += align256(rows * 4);
    v.off_arg = o; o += align256(rows * 4);
    v.off_gap = o; o += align256(rows * 4);
  } else {
    v.off_items = o; o += align256((size_t)d->R * sizeof(VerifyItem));
    v.off_z = o; o += align256((size_t)d->R * d->V * 4);
    v.off_exp = o; o += expand_ws_max(d, d->R, T, true);
    v.max_chunks = (d->V + kVChunkQuantum - 1) / kVChunkQuantum;
    const size_t ic = (size_t)d->R * v.max_chunks;
    v.off_pa = o; o += align256(ic * sizeof(VPartA));
    v.off_zp = o; o += align256(ic * TS_MAX_K * sizeof(double));
    v.off_bp = o; o += align256(ic * sizeof(VBonusPart));
    v.off_cst = o; o += align256((size_t)d->R * sizeof(VConst));
    v.off_rec = o; o += align256((size_t)d->R * TS_MAX_K * sizeof(VRec));
    v.off_sync = o; o += align256(fused_slot_words(d->R) * 8 + 4);
  }
  v.bytes = o;
  return v;
}

// Host checks shared by ts_expand and ts_expand_noalloc.
int32_t check_expand_args(const ts_drafter* d, const ts_parent* parents, int P, ts_calib calib, int k, float T,
                          int sampler, const ts_expand_out* out) {
  int32_t rc = check_drafter(d);
  if (rc != TS_OK) return rc;
  if ((rc = check_k_T(d, k, T)) != TS_OK) return rc;
  if ((rc = check_sampler(sampler)) != TS_OK) return rc;
  if (P < 0) return fail(TS_EINVAL, "P=%d is negative", P);
  if (P == 0) return TS_OK;
  if (!parents) return fail(TS_EINVAL, "parents is NULL");
  if (!out || !out->child_token || !out->child_log_q0 || !out->child_log_surv || !out->slot_key)
    return fail(TS_EINVAL, "a required output pointer is NULL");
  if (!std::isfinite(calib.a) || !std::isfinite(calib.b)) return fail(TS_EINVAL, "calibration must be finite");
  return TS_OK;
}

int32_t noalloc_scratch(char** out) {
  static std::mutex mu;
  static void* addr[64] = {nullptr};
  int dev = 0;
  TS_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(TS_EUNSUPPORTED, "device %d beyond the 64 the library tracks", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    TS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(TS_EHIP, "hipGetSymbolAddress returned no address for the scratch array");
    addr[dev] = p;
  }
  *out = static_cast<char*>(addr[dev]);
  return TS_OK;
}

}  // namespace
}  // namespace ts

using namespace ts;

extern "C" {

const char* ts_last_error(void) { return g_last_error.c_str(); }

const char* ts_version(void) { return "treespark-mi355x 0.2 (gfx950)"; }

int32_t ts_verify_set_mode(int32_t mode) {
  g_last_error.clear();
  if (mode != TS_VERIFY_AUTO && mode != TS_VERIFY_STAGED) return fail(TS_EINVAL, "unknown verify mode %d", mode);
  thread_state().verify_mode = mode;
  return TS_OK;
}

int32_t ts_verify_level_counts(int64_t* fused, int64_t* fallbacks, int64_t* staged) {
  g_last_error.clear();
  if (!fused || !fallbacks || !staged) return fail(TS_EINVAL, "an output is NULL");
  const ThreadState& st = thread_state();
  *fused = st.fused_levels;
  *fallbacks = st.fused_fallbacks;
  *staged = st.staged_levels;
  return TS_OK;
}

int32_t ts_release_thread_state(void) {
  g_last_error.clear();
  ThreadState& st = thread_state();
  if (!st.stage) return TS_OK;
  // every stream that used them has been synchronised by its call, but a
  // caller's later work may still reference the staging buffer's contents:
  // wait for the device before freeing anything
  TS_HIP(hipDeviceSynchronize());
  if (st.stage) TS_HIP(hipHostFree(st.stage));
  st.stage = nullptr;
  st.stage_bytes = 0;
  return TS_OK;
}

size_t ts_expand_workspace_size(const ts_drafter* d, int32_t P, int32_t k, float T) {
  (void)k;
  if (check_drafter(d) != TS_OK || P <= 0) return 0;
  return make_plan(d, P, T, TS_SAMPLER_GUMBEL, false, true).bytes;
}

int32_t ts_expand(const ts_drafter* d, const ts_parent* parents, int32_t P, ts_calib calib,
                  int32_t k, float T, uint64_t seed, int32_t sampler, const ts_expand_out* out,
                  void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int32_t rc = check_expand_args(d, parents, P, calib, k, T, sampler, out);
  if (rc != TS_OK || P == 0) return rc;
  const size_t need = make_plan(d, P, T, TS_SAMPLER_GUMBEL, false, true).bytes;
  if (!workspace || workspace_bytes < need)
    return fail(TS_ENOSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
  return run_expand(d, parents, P, calib, k, T, seed, sampler, out, static_cast<char*>(workspace),
                    static_cast<hipStream_t>(stream));
}

int32_t ts_expand_noalloc(const ts_drafter* d, const ts_parent* parents, int32_t P, ts_calib calib,
                          int32_t k, float T, uint64_t seed, int32_t sampler, const ts_expand_out* out,
                          void* stream) {
  g_last_error.clear();
  int32_t rc = check_expand_args(d, parents, P, calib, k, T, sampler, out);
  if (rc != TS_OK || P == 0) return rc;
  const size_t need = make_plan(d, P, T, sampler).bytes;
  if (need > (size_t)TS_NOALLOC_SCRATCH_BYTES)
    return fail(TS_EUNSUPPORTED, "this launch needs %zu bytes of scratch, more than the %u of ts_expand_noalloc",
                need, TS_NOALLOC_SCRATCH_BYTES);
  char* scratch = nullptr;
  if ((rc = noalloc_scratch(&scratch)) != TS_OK) return rc;
  return run_expand(d, parents, P, calib, k, T, seed, sampler, out, scratch, static_cast<hipStream_t>(stream));
}

size_t ts_build_tree_workspace_size(const ts_drafter* d, int32_t N, int32_t K, float T) {
  if (check_drafter(d) != TS_OK || N < 0 || K < 1 || K > TS_MAX_K) return 0;
  return build_layout(d, N, K, T).bytes;
}

int32_t ts_build_tree(const ts_drafter* d, const int32_t* anchor, const float* theta, int32_t N,
                      int32_t budget, int32_t K, ts_calib calib, float T, uint64_t seed,
                      int32_t sampler, ts_tree* out, const ts_tree* device_out, void* workspace,
                      size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int32_t rc = check_drafter(d);
  if (rc != TS_OK) return rc;
  if ((rc = check_k_T(d, K, T)) != TS_OK) return rc;
  if ((rc = check_sampler(sampler)) != TS_OK) return rc;
  if (N < 0) return fail(TS_EINVAL, "N=%d is negative", N);
  if (!anchor || !theta || !out) return fail(TS_EINVAL, "anchor, theta or out is NULL");
  if (!out->n || !out->token || !out->parent || !out->depth || !out->rank || !out->path ||
      !out->log_surv || !out->log_q0 || !out->log_qT || !out->key)
    return fail(TS_EINVAL, "a tree array is NULL");
  if (out->R != d->R || out->cap < N + 1) return fail(TS_EINVAL, "tree has R=%d cap=%d, need R=%d cap>=%d", out->R, out->cap, d->R, N + 1);
  if (device_out && (device_out->R != out->R || device_out->cap != out->cap || !device_out->n ||
                     !device_out->token || !device_out->parent || !device_out->depth || !device_out->rank ||
                     !device_out->path || !device_out->log_surv || !device_out->log_q0 ||
                     !device_out->log_qT || !device_out->key))
    return fail(TS_EINVAL, "device_out must have the R and cap of out and no NULL array");
  if (!std::isfinite(calib.a) || !std::isfinite(calib.b)) return fail(TS_EINVAL, "calibration must be finite");
  const int R = d->R;
  for (int q = 0; q < R; ++q) {
    if (anchor[q] < 0 || anchor[q] >= d->V) return fail(TS_EINVAL, "anchor[%d]=%d outside [0, V)", q, anchor[q]);
    if (!(theta[q] >= 0.0f) || !std::isfinite(theta[q])) return fail(TS_EINVAL, "theta[%d] must be finite and >= 0", q);
  }
  const BuildLayout bl = build_layout(d, N, K, T);
  if (!workspace || workspace_bytes < bl.bytes)
    return fail(TS_ENOSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, bl.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  ts_parent* dpar = reinterpret_cast<ts_parent*>(ws + bl.off_par);
  ts_expand_out eo{};
  char* hs = nullptr;
  const size_t hs_par = align256((size_t)bl.Pmax * sizeof(ts_parent));
  if ((rc = host_stage(hs_par + (size_t)5 * bl.Pmax * K * 4, &hs)) != TS_OK) return rc;

  std::vector<float> log_theta(R);
  for (int q = 0; q < R; ++q) log_theta[q] = theta[q] > 0.0f ? logf(theta[q]) : -INFINITY;
  if (device_waves(N, K, budget))
    return build_tree_device(d, anchor, log_theta, N, K, calib, T, seed, sampler, out, device_out, ws, bl, s);
  DrainOnError drain{s};
  std::vector<std::vector<Slot>> known(R);
  std::vector<ts_parent> frontier;
  std::vector<int32_t> evals(R, 0);
  if (N > 0)
    for (int q = 0; q < R; ++q) frontier.push_back(ts_parent{anchor[q], 0, q, 0.0f, 0});
  while (!frontier.empty()) {
    const int P = (int)frontier.size();
    const size_t nk = (size_t)P * K;
    // this wave's five outputs, packed, so that one copy brings them back
    char* dout = ws + bl.off_out;
    eo.child_token = reinterpret_cast<int32_t*>(dout);
    eo.child_log_q0 = reinterpret_cast<float*>(dout + nk * 4);
    eo.child_log_qT = reinterpret_cast<float*>(dout + nk * 8);
    eo.child_log_surv = reinterpret_cast<float*>(dout + nk * 12);
    eo.slot_key = reinterpret_cast<float*>(dout + nk * 16);
    std::memcpy(hs, frontier.data(), P * sizeof(ts_parent));
    TS_HIP(hipMemcpyAsync(dpar, hs, P * sizeof(ts_parent), hipMemcpyHostToDevice, s));
    rc = run_expand(d, dpar, P, calib, K, T, seed, sampler, &eo, ws + bl.off_exp, s);
    if (rc != TS_OK) return rc;
    char* hout = hs + hs_par;
    TS_HIP(hipMemcpyAsync(hout, dout, nk * 20, hipMemcpyDeviceToHost, s));
    const int32_t* h_tok = reinterpret_cast<const int32_t*>(hout);
    const float* h_q0 = reinterpret_cast<const float*>(hout + nk * 4);
    const float* h_qT = reinterpret_cast<const float*>(hout + nk * 8);
    const float* h_ls = reinterpret_cast<const float*>(hout + nk * 12);
    const float* h_key = reinterpret_cast<const float*>(hout + nk * 16);
    TS_HIP(hipStreamSynchronize(s));
    for (int i = 0; i < P; ++i) {
      const ts_parent& par = frontier[i];
      ++evals[par.request];
      for (int j = 0; j < K; ++j) {
        const size_t o = (size_t)i * K + j;
        Slot sl;
        sl.key = h_key[o];
        sl.depth = par.depth + 1;
        sl.path = par.path | ((uint64_t)j << (4 * par.depth));
        sl.token = h_tok[o];
        sl.log_surv = h_ls[o];
        sl.log_q0 = h_q0[o];
        sl.log_qT = h_qT[o];
        sl.evaluated = false;
        known[par.request].push_back(sl);
      }
    }
    // Next wave: children of the slots that can still be among the tree's
    // nodes: key >= log(theta_q), strictly above the request's N-th such slot
    // and, under a global budget B, strictly above the B-th best of all
    // requests' top-N slots in the global order (key desc, request asc,
    // depth asc, path asc).  Any node of the final trees descends from such
    // a child, because a slot's key never exceeds the key of the slot whose
    // pop created it.
    frontier.clear();
    std::vector<Slot> nth(R);
    std::vector<char> have_n(R, 0);
    std::vector<GlobalRef> pool;
    for (int q = 0; q < R; ++q) {
      std::vector<Slot> el;
      for (const Slot& sl : known[q])
        if (sl.key >= log_theta[q]) el.push_back(sl);
      if (N > 0 && (int)el.size() >= N) {
        std::nth_element(el.begin(), el.begin() + (N - 1), el.end(), slot_before);
        nth[q] = el[N - 1];
        have_n[q] = 1;
      }
      if (budget > 0) {
        const int take = std::min<int>(N, (int)el.size());
        if (take < (int)el.size()) el.resize(take);  // nth_element left the top N first
        for (const Slot& sl : el) pool.push_back(GlobalRef{sl.key, q, sl.depth, sl.path});
      }
    }
    bool have_g = false;
    GlobalRef gth{};
    if (budget > 0 && (int)pool.size() >= budget) {
      std::nth_element(pool.begin(), pool.begin() + (budget - 1), pool.end(), global_before);
      gth = pool[budget - 1];
      have_g = true;
    }
    for (int q = 0; q < R; ++q) {
      const size_t first = frontier.size();
      for (Slot& sl : known[q]) {
        if (sl.evaluated || sl.depth >= d->D || sl.key < log_theta[q]) continue;
        if (have_n[q] && !slot_before(sl, nth[q])) continue;
        if (have_g && !global_before(GlobalRef{sl.key, q, sl.depth, sl.path}, gth)) continue;
        sl.evaluated = true;
        frontier.push_back(ts_parent{sl.token, sl.depth, q, sl.log_surv, sl.path});
      }
      std::sort(frontier.begin() + first, frontier.end(),
                [](const ts_parent& a, const ts_parent& b) { return a.depth < b.depth; });
    }
  }
  // The trees: each request's slots in pop order, at most N, stopping below
  // log(theta_q); under a global budget, the best B of those in the global order.
  std::vector<int> take(R, 0);
  {
    std::vector<GlobalRef> pool;
    for (int q = 0; q < R; ++q) {
      std::vector<Slot>& ks = known[q];
      std::sort(ks.begin(), ks.end(), slot_before);
      int t = 0;
      while (t < (int)ks.size() && t < N && ks[t].key >= log_theta[q]) ++t;
      take[q] = t;
      if (budget > 0)
        for (int i = 0; i < t; ++i) pool.push_back(GlobalRef{ks[i].key, q, ks[i].depth, ks[i].path});
    }
    if (budget > 0 && (int)pool.size() > budget) {
      std::nth_element(pool.begin(), pool.begin() + budget, pool.end(), global_before);
      std::fill(take.begin(), take.end(), 0);
      for (int i = 0; i < budget; ++i) ++take[pool[i].q];  // a prefix of each request's order
    }
  }
  const int cap = out->cap;
  for (int q = 0; q < R; ++q) {
    std::vector<Slot>& ks = known[q];
    const size_t b = (size_t)q * cap;
    out->token[b] = anchor[q];
    out->parent[b] = -1;
    out->depth[b] = 0;
    out->rank[b] = 0;
    out->path[b] = 0;
    out->log_surv[b] = 0.0f;
    out->log_q0[b] = 0.0f;
    out->log_qT[b] = NAN;
    out->key[b] = 0.0f;
    std::unordered_map<uint64_t, int> node_of[TS_MAX_D + 1];
    node_of[0][0] = 0;
    int n = 0;
    for (const Slot& sl : ks) {
      if (n >= take[q]) break;
      const int pd = sl.depth - 1;
      const uint64_t ppath = sl.path & ((pd == 0) ? 0ull : ((1ull << (4 * pd)) - 1ull));
      const auto it = node_of[pd].find(ppath);
      if (it == node_of[pd].end()) return fail(TS_EINTERNAL, "request %d: slot without a materialised parent", q);
      const int c = ++n;
      out->token[b + c] = sl.token;
      out->parent[b + c] = it->second;
      out->depth[b + c] = sl.depth;
      out->rank[b + c] = (int)((sl.path >> (4 * pd)) & 15ull) + 1;
      out->path[b + c] = sl.path;
      out->log_surv[b + c] = sl.log_surv;
      out->log_q0[b + c] = sl.log_q0;
      out->log_qT[b + c] = sl.log_qT;
      out->key[b + c] = sl.key;
      node_of[sl.depth][sl.path] = c;
    }
    out->n[q] = n;
    if (out->evals) out->evals[q] = evals[q];
    for (int c = n + 1; c < cap; ++c) {  // rows past the tree, as the device waves leave them
      out->token[b + c] = -1;
      out->parent[b + c] = -1;
      out->depth[b + c] = 0;
      out->rank[b + c] = 0;
      out->path[b + c] = 0;
      out->log_surv[b + c] = NAN;
      out->log_q0[b + c] = NAN;
      out->log_qT[b + c] = NAN;
      out->key[b + c] = NAN;
    }
  }
  if (device_out) {
    const size_t rcn = (size_t)R * cap;
    const hipMemcpyKind h2d = hipMemcpyHostToDevice;
    TS_HIP(hipMemcpyAsync(device_out->n, out->n, (size_t)R * 4, h2d, s));
    if (device_out->evals && out->evals) TS_HIP(hipMemcpyAsync(device_out->evals, out->evals, (size_t)R * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->token, out->token, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->parent, out->parent, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->depth, out->depth, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->rank, out->rank, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->path, out->path, rcn * 8, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->log_surv, out->log_surv, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->log_q0, out->log_q0, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->log_qT, out->log_qT, rcn * 4, h2d, s));
    TS_HIP(hipMemcpyAsync(device_out->key, out->key, rcn * 4, h2d, s));
    TS_HIP(hipStreamSynchronize(s));
  }
  drain.armed = false;
  return TS_OK;
}

size_t ts_verify_workspace_size(const ts_drafter* d, int32_t cap, float T) {
  if (check_drafter(d) != TS_OK || cap < 1 || !(T >= 0.0f)) return 0;
  return verify_layout(d, cap, T).bytes;
}

int32_t ts_verify(const ts_drafter* d, const ts_tree* tree, const void* target, int32_t target_dtype,
                  float T, uint64_t seed, int32_t* path_nodes, int32_t* path_len, int32_t* bonus,
                  void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int32_t rc = check_drafter(d);
  if (rc != TS_OK) return rc;
  if (!tree || !target || !path_nodes || !path_len || !bonus)
    return fail(TS_EINVAL, "tree, target or an output is NULL");
  if (!tree->n || !tree->token || !tree->parent || !tree->depth || !tree->path)
    return fail(TS_EINVAL, "a tree array is NULL");
  if (tree->R != d->R || tree->cap < 1) return fail(TS_EINVAL, "tree R=%d cap=%d does not match R=%d", tree->R, tree->cap, d->R);
  if (target_dtype != TS_F32 && target_dtype != TS_BF16) return fail(TS_EINVAL, "unknown target dtype %d", target_dtype);
  if (!(T >= 0.0f) || !std::isfinite(T)) return fail(TS_EINVAL, "T must be finite and >= 0");
  const int R = d->R, cap = tree->cap, V = d->V;
  for (int q = 0; q < R; ++q) {
    const int n = tree->n[q];
    if (n < 0 || n >= cap) return fail(TS_EINVAL, "tree n[%d]=%d outside [0, cap)", q, n);
    for (int i = 1; i <= n; ++i) {
      const size_t o = (size_t)q * cap + i;
      const int pa = tree->parent[o];
      if (pa < 0 || pa >= i || tree->token[o] < 0 || tree->token[o] >= V ||
          tree->depth[o] != tree->depth[(size_t)q * cap + pa] + 1 || tree->depth[o] > d->D)
        return fail(TS_EINVAL, "tree of request %d is malformed at node %d", q, i);
    }
    if (tree->token[(size_t)q * cap] < 0 || tree->token[(size_t)q * cap] >= V)
      return fail(TS_EINVAL, "root token of request %d outside [0, V)", q);
  }
  const VerifyLayout vl = verify_layout(d, cap, T);
  if (!workspace || workspace_bytes < vl.bytes)
    return fail(TS_ENOSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, vl.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);

  DrainOnError drain{s};
  for (int q = 0; q < R; ++q) path_len[q] = 0;

  if (T == 0.0f) {
    // children of every node in creation order
    const KidIndex& kids = kid_index(tree);
    std::vector<int> rows;
    for (int q = 0; q < R; ++q)
      for (int i = 0; i <= tree->n[q]; ++i) rows.push_back(q * cap + i);
    const int nrows = (int)rows.size();
    int* drows = reinterpret_cast<int*>(ws + vl.off_rows);
    int* darg = reinterpret_cast<int*>(ws + vl.off_arg);
    float* dgap = reinterpret_cast<float*>(ws + vl.off_gap);
    char* hs = nullptr;
    if ((rc = host_stage((size_t)nrows * 8, &hs)) != TS_OK) return rc;
    std::memcpy(hs, rows.data(), (size_t)nrows * 4);
    TS_HIP(hipMemcpyAsync(drows, hs, nrows * 4, hipMemcpyHostToDevice, s));
    launch_verify_argmax(target, target_dtype == TS_BF16, V, drows, nrows, darg, dgap, s);
    TS_HIP(hipGetLastError());
    const int* arg = reinterpret_cast<const int*>(hs + (size_t)nrows * 4);
    TS_HIP(hipMemcpyAsync(hs + (size_t)nrows * 4, darg, nrows * 4, hipMemcpyDeviceToHost, s));
    TS_HIP(hipStreamSynchronize(s));
    int base = 0;
    for (int q = 0; q < R; ++q) {
      int cur = 0, len = 0;
      for (;;) {
        const int gtok = arg[base + cur];
        int next = -1;
        const int* ch = kids.first(q, cur);
        for (int j = 0, m = kids.count(q, cur); j < m; ++j)
          if (tree->token[(size_t)q * cap + ch[j]] == gtok) { next = ch[j]; break; }
        if (next < 0 || len >= TS_MAX_D) { bonus[q] = gtok; break; }
        path_nodes[(size_t)q * TS_MAX_D + len++] = next;
        cur = next;
      }
      path_len[q] = len;
      base += tree->n[q] + 1;
    }
    drain.armed = false;
    return TS_OK;
  }

  // T > 0: one level of the walk per iteration, batched over the requests still walking.
  VerifyItem* ditems = reinterpret_cast<VerifyItem*>(ws + vl.off_items);
  float* zbuf = reinterpret_cast<float*>(ws + vl.off_z);
  const PhiloxKeys keys = philox_keys(seed);
  std::vector<int> cur(R, 0), active(R);
  for (int q = 0; q < R; ++q) active[q] = q;
  std::vector<VerifyItem> items;
  std::vector<ts_parent> zpar;
  char* hs = nullptr;
  const size_t hs_items = align256((size_t)R * sizeof(VerifyItem));
  const size_t hs_par = align256((size_t)R * sizeof(ts_parent));
  const size_t hs_res = align256((size_t)R * sizeof(VerifyResult));
  const size_t hs_next = align256((size_t)R * sizeof(VerifyNext));
  if ((rc = host_stage(hs_items + hs_par + hs_res + hs_next + 256, &hs)) != TS_OK) return rc;
  // The first level's logit recompute is queued first: its rows are the roots
  // of the trees that have children (n > 0), in request order, which the
  // level loop below assigns the same way; the child index and the level's
  // items are built while it runs.
  int first_rows = 0;
  for (int q = 0; q < R; ++q) {
    if (tree->n[q] <= 0) continue;
    const size_t o = (size_t)q * cap;
    reinterpret_cast<ts_parent*>(hs + hs_items)[first_rows++] =
        ts_parent{tree->token[o], tree->depth[o], q, 0.0f, tree->path[o]};
  }
  auto launch_recompute = [&](int P) -> int32_t {
    const Plan pl = make_plan(d, P, T, TS_SAMPLER_GUMBEL, true);
    const ExpandParams ep =
        eval_params(d, reinterpret_cast<const ts_parent*>(hs + hs_items), P, T, seed, pl, ws + vl.off_exp, zbuf);
    launch_eval(d, ep, pl, s);
    TS_HIP(hipGetLastError());
    return TS_OK;
  };
  if (first_rows > 0 && (rc = launch_recompute(first_rows)) != TS_OK) return rc;
  // children of every node in creation order (= draw order)
  const KidIndex& kids = kid_index(tree);
  bool first_level = true;
  const VerifyResult* res = reinterpret_cast<const VerifyResult*>(hs + hs_items + hs_par);
  VerifyNext* hnext = reinterpret_cast<VerifyNext*>(hs + hs_items + hs_par + hs_res);
  volatile int32_t* herr = reinterpret_cast<volatile int32_t*>(hs + hs_items + hs_par + hs_res + hs_next);
  // the one-launch levels' slots and flag start the call at zero; each
  // launch tags its slot words with an epoch of its own
  uint64_t* dslots = reinterpret_cast<uint64_t*>(ws + vl.off_sync);
  const size_t nslots = fused_slot_words(R);
  int* derr = reinterpret_cast<int*>(dslots + nslots);
  const int nclear = (int)(nslots * 2 + 1);
  const bool bf16 = target_dtype == TS_BF16;
  uint32_t epoch = 0;
  launch_verify_clear(reinterpret_cast<int*>(dslots), nclear, s);
  TS_HIP(hipGetLastError());
  while (!active.empty()) {
    items.clear();
    zpar.clear();
    for (int q : active) {
      const size_t o = (size_t)q * cap + cur[q];
      VerifyItem it{};
      it.request = q;
      it.node = cur[q];
      it.depth = tree->depth[o];
      it.path = tree->path[o];
      const int* ch = kids.first(q, cur[q]);
      it.m = std::min(kids.count(q, cur[q]), TS_MAX_K);
      for (int j = 0; j < it.m; ++j) it.child_tok[j] = tree->token[(size_t)q * cap + ch[j]];
      it.zrow = -1;
      if (it.m > 0) {
        it.zrow = (int)zpar.size();
        zpar.push_back(ts_parent{tree->token[o], tree->depth[o], q, 0.0f, tree->path[o]});
      }
      items.push_back(it);
    }
    const int ni = (int)items.size();
    if (first_level) {
      if ((int)zpar.size() != first_rows)
        return fail(TS_EINTERNAL, "first verification level has %d recompute rows, %d queued", (int)zpar.size(),
                    first_rows);
    } else if (!zpar.empty()) {
      // the recompute reads its parents from the pinned buffer
      std::memcpy(hs + hs_items, zpar.data(), zpar.size() * sizeof(ts_parent));
      if ((rc = launch_recompute((int)zpar.size())) != TS_OK) return rc;
    }
    first_level = false;
    // pass A reads the items from the pinned buffer and stages them in ditems
    std::memcpy(hs, items.data(), ni * sizeof(VerifyItem));
    VerifyPass vp{};
    vp.target = target;
    vp.cap = cap;
    vp.V = V;
    vp.items = ditems;
    vp.items_host = reinterpret_cast<const VerifyItem*>(hs);
    vp.items_w = ditems;
    vp.nitems = ni;
    vp.zbuf = zbuf;
    vp.c = kLog2e / T;
    vp.keys = keys;
    verify_chunks(V, ni, &vp.nchunks, &vp.chunk);
    vp.pa = reinterpret_cast<VPartA*>(ws + vl.off_pa);
    vp.zp = reinterpret_cast<double*>(ws + vl.off_zp);
    vp.bp = reinterpret_cast<VBonusPart*>(ws + vl.off_bp);
    vp.consts = reinterpret_cast<VConst*>(ws + vl.off_cst);
    vp.recs = reinterpret_cast<VRec*>(ws + vl.off_rec);
    vp.results = const_cast<VerifyResult*>(res);  // pinned: the resolve kernel writes it
    int mmax = 0;
    for (const VerifyItem& it : items) mmax = std::max(mmax, it.m);
    const FusedPlan fp = thread_state().verify_mode == TS_VERIFY_STAGED ? FusedPlan{false, 0, 0}
                                                                          : fused_plan(V, ni, bf16);
    if (fp.ok) {
      ++thread_state().fused_levels;
      // one launch for the level; a wait that ran out (some workgroup was
      // not resident) sends the level through the per-stage launches
      VerifyPass fvp = vp;
      fvp.nchunks = fp.cpi;
      fvp.chunk = fp.chunk;
      VFused f{};
      f.cpi = fp.cpi;
      f.chunk = fp.chunk;
      f.slots = dslots;
      f.epoch = ++epoch;
      f.err = derr;
      f.herr = const_cast<int32_t*>(herr);
      f.spin_limit = kFusedSpinLimit;
      f.next_host = hnext;
      // each item's children: node, path, and whether the walk ends there
      for (int i = 0; i < ni; ++i) {
        const VerifyItem& it = items[i];
        VerifyNext nx{};
        const int* ch = kids.first(it.request, it.node);
        for (int j = 0; j < it.m; ++j) {
          const size_t o = (size_t)it.request * cap + ch[j];
          nx.child_node[j] = ch[j];
          nx.child_path[j] = tree->path[o];
          if (kids.count(it.request, ch[j]) == 0) nx.leaf_mask |= 1u << j;
        }
        hnext[i] = nx;
      }
      *herr = 0;
      launch_verify_fused(fvp, f, bf16, s);
      TS_HIP(hipGetLastError());
      TS_HIP(hipStreamSynchronize(s));
      if (*herr != 0) {
        ++thread_state().fused_fallbacks;
        launch_verify_clear(derr, 1, s);
        launch_verify_level(vp, bf16, mmax, s);
        TS_HIP(hipGetLastError());
        TS_HIP(hipStreamSynchronize(s));
      }
    } else {
      ++thread_state().staged_levels;
      launch_verify_level(vp, bf16, mmax, s);
      TS_HIP(hipGetLastError());
      TS_HIP(hipStreamSynchronize(s));
    }
    std::vector<int> next;
    for (int i = 0; i < ni; ++i) {
      const int q = items[i].request;
      if (res[i].accepted > 0 && path_len[q] < TS_MAX_D) {
        const int c = kids.first(q, cur[q])[res[i].accepted - 1];
        path_nodes[(size_t)q * TS_MAX_D + path_len[q]++] = c;
        cur[q] = c;
        if (res[i].leaf_bonus)
          bonus[q] = res[i].bonus;  // the accepted child has no children: its bonus is drawn
        else
          next.push_back(q);
      } else {
        bonus[q] = res[i].bonus;
      }
    }
    active.swap(next);
  }
  drain.armed = false;
  return TS_OK;
}

int32_t ts_ladder_lookup(const ts_ladder_rung* rungs, int32_t n, int32_t bs, float T, int32_t K,
                         int32_t N, int32_t block_len, ts_round_policy* out) {
  g_last_error.clear();
  if (!rungs || !out) return fail(TS_EINVAL, "rungs or out is NULL");
  if (n < 1) return fail(TS_EINVAL, "the ladder has no rungs");
  if (bs < 1) return fail(TS_EINVAL, "batch size %d < 1", bs);
  if (!(T >= 0.0f) || !std::isfinite(T)) return fail(TS_EINVAL, "T must be finite and >= 0");
  if (K < 1 || K > TS_MAX_K) return fail(TS_EINVAL, "K=%d outside [1, %d]", K, TS_MAX_K);
  if (N < 0) return fail(TS_EINVAL, "N=%d is negative", N);
  if (block_len < 1 || block_len > TS_MAX_D) return fail(TS_EINVAL, "block length %d outside [1, %d]", block_len, TS_MAX_D);
  // nearest tabulated temperature, ties to the lower one
  float best_T = rungs[0].T;
  for (int i = 1; i < n; ++i) {
    const float d = std::fabs(rungs[i].T - T), db = std::fabs(best_T - T);
    if (d < db || (d == db && rungs[i].T < best_T)) best_T = rungs[i].T;
  }
  int pick = -1, widest = -1;
  for (int i = 0; i < n; ++i) {
    if (rungs[i].T != best_T) continue;
    if (widest < 0 || rungs[i].bs_max > rungs[widest].bs_max) widest = i;
    if (rungs[i].bs_max >= bs && (pick < 0 || rungs[i].bs_max < rungs[pick].bs_max)) pick = i;
  }
  if (pick < 0) pick = widest;
  if (rungs[pick].theta < 0.0f) {
    *out = ts_round_policy{0.0f, 1, block_len, 1};
  } else {
    *out = ts_round_policy{rungs[pick].theta, K, N, 0};
  }
  return TS_OK;
}

int32_t ts_ladder_default(ts_ladder_rung* rungs, int32_t cap) {
  static const ts_ladder_rung kLadder[] = {
      {4, 0.0f, 0.02f}, {8, 0.0f, 0.05f}, {INT32_MAX, 0.0f, 0.15f},
      {8, 0.5f, 0.05f}, {INT32_MAX, 0.5f, -1.0f},
      {8, 1.0f, 0.05f}, {INT32_MAX, 1.0f, -1.0f}};
  const int32_t count = (int32_t)(sizeof(kLadder) / sizeof(kLadder[0]));
  for (int32_t i = 0; rungs && i < cap && i < count; ++i) rungs[i] = kLadder[i];
  return count;
}

// ---------------------------------------------------------------- calibration

namespace {
struct CalibLayout {
  size_t parent, token, log_q0, n, rows, off, upload, greedy, gap, bytes;
};
CalibLayout calib_layout(int R, int cap) {
  CalibLayout c{};
  const size_t rc = (size_t)R * cap;
  size_t o = 0;
  c.parent = o; o += align256(rc * 4);
  c.token = o; o += align256(rc * 4);
  c.log_q0 = o; o += align256(rc * 4);
  c.n = o; o += align256((size_t)R * 4);
  c.rows = o; o += align256(rc * 4);
  c.off = o; o += align256((size_t)R * 4);
  c.upload = o;  // everything above is one host-to-device copy
  c.greedy = o; o += align256(rc * 4);
  c.gap = o; o += align256(rc * 4);
  c.bytes = o;
  return c;
}
}  // namespace

size_t ts_calib_labels_workspace_size(int32_t R, int32_t cap) {
  if (R < 1 || cap < 1) return 0;
  return calib_layout(R, cap).bytes;
}

int32_t ts_calib_labels(const ts_tree* tree, const void* target, int32_t target_dtype, int32_t V, float* x,
                        int32_t* y, int32_t* sel, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!tree || !target || !x || !y || !sel) return fail(TS_EINVAL, "tree, target or an output is NULL");
  if (!tree->n || !tree->token || !tree->parent || !tree->log_q0) return fail(TS_EINVAL, "a tree array is NULL");
  if (tree->R < 1 || tree->cap < 1) return fail(TS_EINVAL, "tree R=%d cap=%d", tree->R, tree->cap);
  if (V < 1) return fail(TS_EINVAL, "V=%d", V);
  if (target_dtype != TS_F32 && target_dtype != TS_BF16) return fail(TS_EINVAL, "unknown target dtype %d", target_dtype);
  const int R = tree->R, cap = tree->cap;
  for (int q = 0; q < R; ++q) {
    const int nq = tree->n[q];
    if (nq < 0 || nq >= cap) return fail(TS_EINVAL, "tree n[%d]=%d outside [0, cap)", q, nq);
    for (int i = 1; i <= nq; ++i) {
      const size_t o = (size_t)q * cap + i;
      if (tree->parent[o] < 0 || tree->parent[o] >= i || tree->token[o] < 0 || tree->token[o] >= V)
        return fail(TS_EINVAL, "tree of request %d is malformed at node %d", q, i);
    }
  }
  const CalibLayout cl = calib_layout(R, cap);
  if (!workspace || workspace_bytes < cl.bytes)
    return fail(TS_ENOSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, cl.bytes);
  char* hs = nullptr;
  int32_t rc = host_stage(cl.upload, &hs);
  if (rc != TS_OK) return rc;
  const size_t rcn = (size_t)R * cap;
  std::memcpy(hs + cl.parent, tree->parent, rcn * 4);
  std::memcpy(hs + cl.token, tree->token, rcn * 4);
  std::memcpy(hs + cl.log_q0, tree->log_q0, rcn * 4);
  std::memcpy(hs + cl.n, tree->n, (size_t)R * 4);
  int32_t* rows = reinterpret_cast<int32_t*>(hs + cl.rows);
  int32_t* off = reinterpret_cast<int32_t*>(hs + cl.off);
  int nrows = 0;
  for (int q = 0; q < R; ++q) {
    off[q] = nrows;
    for (int i = 0; i <= tree->n[q]; ++i) rows[nrows++] = q * cap + i;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  DrainOnError drain{s};
  TS_HIP(hipMemcpyAsync(ws, hs, cl.upload, hipMemcpyHostToDevice, s));
  int32_t* greedy = reinterpret_cast<int32_t*>(ws + cl.greedy);
  launch_verify_argmax(target, target_dtype == TS_BF16, V, reinterpret_cast<const int*>(ws + cl.rows), nrows,
                       greedy, reinterpret_cast<float*>(ws + cl.gap), s);
  TS_HIP(hipGetLastError());
  launch_calib_labels(reinterpret_cast<const int32_t*>(ws + cl.parent), reinterpret_cast<const int32_t*>(ws + cl.token),
                      reinterpret_cast<const float*>(ws + cl.log_q0), reinterpret_cast<const int32_t*>(ws + cl.n), R,
                      cap, greedy, reinterpret_cast<const int32_t*>(ws + cl.off), x, y, sel, s);
  TS_HIP(hipGetLastError());
  TS_HIP(hipStreamSynchronize(s));
  drain.armed = false;
  return TS_OK;
}

int32_t ts_calib_fit(const float* x, const int32_t* y, const int32_t* sel, int32_t n, int32_t max_iter,
                     double tol, float* out, void* stream) {
  g_last_error.clear();
  if (!x || !y || !sel || !out) return fail(TS_EINVAL, "an array is NULL");
  if (n < 0 || max_iter < 1 || !(tol > 0.0)) return fail(TS_EINVAL, "n=%d max_iter=%d tol=%g", n, max_iter, tol);
  launch_calib_fit(x, y, sel, n, max_iter, tol, out, static_cast<hipStream_t>(stream));
  TS_HIP(hipGetLastError());
  return TS_OK;
}

int32_t ts_tree_mask_words(int32_t cap) { return cap < 1 ? 0 : (cap + 31) / 32; }

int32_t ts_tree_mask(const int32_t* parent, const int32_t* n, int32_t R, int32_t cap,
                     const int32_t* pos_offset, uint32_t* mask, int32_t* pos, void* stream) {
  g_last_error.clear();
  if (R < 0) return fail(TS_EINVAL, "R=%d is negative", R);
  if (cap < 1 || cap > TS_MAX_CAP) return fail(TS_EINVAL, "cap=%d outside [1, %d]", cap, TS_MAX_CAP);
  if (R == 0) return TS_OK;
  if (!parent || !n || !mask || !pos) return fail(TS_EINVAL, "parent, n, mask or pos is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  launch_tree_mask(parent, n, R, cap, pos_offset, mask, pos, s);
  TS_HIP(hipGetLastError());
  return TS_OK;
}

}  // extern "C"
