// Definitions of the expansion launchers; included only by the per-rank
// translation units (expand_<dtype>_ks<KS>.hip), which instantiate them.
#pragma once

#include "launch.hpp"

namespace ts {

// The kernel of a launch for one (dtype, rank, parent blocks per wave):
// the verification recompute stores z and needs no draws (mode 0).
template <typename TE, int KS, int NB, bool LDS, int WPG = 4>
struct EvalKernels {
  template <int MODE>
  static auto pick() {
    if constexpr (LDS)
      return expand_eval_lds_kernel<KS, NB, MODE, WPG>;
    else
      return expand_eval_kernel<TE, KS, NB, MODE, false>;
  }
  // mode: kModeGreedy, kModeGumbel or kModeSeq, with kModeNeedT for T != 1
  // (the LDS kernel has a variant for it; the other takes it from the params)
  static auto get(int mode) {
    decltype(pick<0>()) k = pick<0>();
    const bool nt = LDS && (mode & kModeNeedT);
    const int base = mode & 3;
    if (base == kModeGumbel) k = nt ? pick<(LDS ? kModeGumbel | kModeNeedT : kModeGumbel)>() : pick<kModeGumbel>();
    if (base == kModeSeq) k = nt ? pick<(LDS ? kModeSeq | kModeNeedT : kModeSeq)>() : pick<kModeSeq>();
    return k;
  }
};

// The LDS kernel with two parent blocks per wave runs in workgroups of 8
// waves for greedy launches at rank <= 64 (half the W2 tile loads per parent;
// four waves per SIMD need <= 128 VGPRs, which only the greedy epilogue fits),
// else of 4; the plan's choice arrives as the block size.  The other kernels
// use 4.
template <typename TE, int KS>
static void (*eval_kernel_for(int nb, int mode, bool store_z, bool lds, int block))(ExpandParams) {
  if (store_z) return expand_eval_kernel<TE, KS, 1, kModeGreedy, true>;
  if constexpr (sizeof(TE) == 2) {
    if (lds) {
      if (nb == 1) return EvalKernels<TE, KS, 1, true>::get(mode);
      if constexpr (KS <= 2) {  // larger ranks: the W2 tiles leave LDS for four waves only
        if (block == 8 * 64 && (mode & 3) == kModeGreedy) return expand_eval_lds_kernel<KS, 2, kModeGreedy, 8>;
      }
      return EvalKernels<TE, KS, 2, true>::get(mode);
    }
  }
  return nb == 1 ? EvalKernels<TE, KS, 1, false>::get(mode) : EvalKernels<TE, KS, 2, false>::get(mode);
}

template <typename TE, int KS>
void launch_eval_t(const ExpandParams& p, int nb, int mode, bool store_z, bool lds, dim3 grid,
                   dim3 block, hipStream_t s) {
  void (*kernel)(ExpandParams) = eval_kernel_for<TE, KS>(nb, mode, store_z, lds, (int)block.x);
  hipLaunchKernelGGL(kernel, grid, block, 0, s, p);
}

template <typename TE, int KS>
int eval_blocks_per_cu_t(int nb, int mode, bool store_z, bool lds, int block) {
  int n = 0;
  void (*kernel)(ExpandParams) = eval_kernel_for<TE, KS>(nb, mode, store_z, lds, block);
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, block, 0);
  return e == hipSuccess ? n : 0;
}

template <typename TE, int KS>
void launch_merge_t(const MergeParams& p, int mode, dim3 grid, dim3 block, hipStream_t s) {
  if (mode == kModeGumbel)
    hipLaunchKernelGGL((expand_merge_kernel<TE, KS, kModeGumbel>), grid, block, 0, s, p);
  else if (mode == kModeSeq)
    hipLaunchKernelGGL((expand_merge_kernel<TE, KS, kModeSeq>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((expand_merge_kernel<TE, KS, kModeGreedy>), grid, block, 0, s, p);
}

}  // namespace ts
