// Definitions of the expansion launchers; included only by the per-rank
// translation units (expand_<dtype>_ks<KS>.hip), which instantiate them.
#pragma once

#include "launch.hpp"

namespace ts {

template <typename TE, int KS, int NB>
void launch_eval_nb(const ExpandParams& p, bool sample, bool store_z, dim3 grid, dim3 block,
                    hipStream_t s) {
  if constexpr (NB == 1) {
    if (store_z) {
      if (sample)
        hipLaunchKernelGGL((expand_eval_kernel<TE, KS, 1, true, true>), grid, block, 0, s, p);
      else
        hipLaunchKernelGGL((expand_eval_kernel<TE, KS, 1, false, true>), grid, block, 0, s, p);
      return;
    }
  }
  if (sample)
    hipLaunchKernelGGL((expand_eval_kernel<TE, KS, NB, true, false>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((expand_eval_kernel<TE, KS, NB, false, false>), grid, block, 0, s, p);
}

template <int KS, int NB>
void launch_eval_lds_nb(const ExpandParams& p, bool sample, dim3 grid, dim3 block, hipStream_t s) {
  if (sample)
    hipLaunchKernelGGL((expand_eval_lds_kernel<KS, NB, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((expand_eval_lds_kernel<KS, NB, false>), grid, block, 0, s, p);
}

template <typename TE, int KS>
void launch_eval_t(const ExpandParams& p, int nb, bool sample, bool store_z, bool lds, dim3 grid,
                   dim3 block, hipStream_t s) {
  if constexpr (sizeof(TE) == 2) {
    if (lds && !store_z) {
      if (nb == 1)
        launch_eval_lds_nb<KS, 1>(p, sample, grid, block, s);
      else if (nb == 2)
        launch_eval_lds_nb<KS, 2>(p, sample, grid, block, s);
      else
        launch_eval_lds_nb<KS, 4>(p, sample, grid, block, s);
      return;
    }
  }
  if (nb == 1 || store_z)
    launch_eval_nb<TE, KS, 1>(p, sample, store_z, grid, block, s);
  else if (nb == 2)
    launch_eval_nb<TE, KS, 2>(p, sample, false, grid, block, s);
  else
    launch_eval_nb<TE, KS, 4>(p, sample, false, grid, block, s);
}

template <typename TE, int KS>
int eval_blocks_per_cu_t(int nb, bool sample, bool store_z, bool lds, int block) {
  int n = 0;
  hipError_t e = hipSuccess;
#define TS_OCC(kern) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, block, 0)
  if constexpr (sizeof(TE) == 2) {
    if (lds && !store_z) {
      if (nb == 1) { if (sample) TS_OCC((expand_eval_lds_kernel<KS, 1, true>)); else TS_OCC((expand_eval_lds_kernel<KS, 1, false>)); }
      else if (nb == 2) { if (sample) TS_OCC((expand_eval_lds_kernel<KS, 2, true>)); else TS_OCC((expand_eval_lds_kernel<KS, 2, false>)); }
      else { if (sample) TS_OCC((expand_eval_lds_kernel<KS, 4, true>)); else TS_OCC((expand_eval_lds_kernel<KS, 4, false>)); }
      return e == hipSuccess ? n : 0;
    }
  }
  if (nb == 1 || store_z) {
    if (store_z) { if (sample) TS_OCC((expand_eval_kernel<TE, KS, 1, true, true>)); else TS_OCC((expand_eval_kernel<TE, KS, 1, false, true>)); }
    else { if (sample) TS_OCC((expand_eval_kernel<TE, KS, 1, true, false>)); else TS_OCC((expand_eval_kernel<TE, KS, 1, false, false>)); }
  } else if (nb == 2) {
    if (sample) TS_OCC((expand_eval_kernel<TE, KS, 2, true, false>)); else TS_OCC((expand_eval_kernel<TE, KS, 2, false, false>));
  } else {
    if (sample) TS_OCC((expand_eval_kernel<TE, KS, 4, true, false>)); else TS_OCC((expand_eval_kernel<TE, KS, 4, false, false>));
  }
#undef TS_OCC
  return e == hipSuccess ? n : 0;
}

template <typename TE, int KS>
void launch_merge_t(const MergeParams& p, bool sample, dim3 grid, dim3 block, hipStream_t s) {
  if (sample)
    hipLaunchKernelGGL((expand_merge_kernel<TE, KS, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((expand_merge_kernel<TE, KS, false>), grid, block, 0, s, p);
}

}  // namespace ts
