// Instantiations of the verification kernels.
#include "launch.hpp"

namespace ts {

void launch_verify_argmax(const void* target, bool bf16, int V, const int* rows, int nrows,
                          int* argmax_out, float* gap_out, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL((verify_argmax_kernel<uint16_t>), dim3(nrows), dim3(kVerifyThreads), 0, s,
                       static_cast<const uint16_t*>(target), V, rows, nrows, argmax_out, gap_out);
  else
    hipLaunchKernelGGL((verify_argmax_kernel<float>), dim3(nrows), dim3(kVerifyThreads), 0, s,
                       static_cast<const float*>(target), V, rows, nrows, argmax_out, gap_out);
}

void launch_verify_stage(const void* target, bool bf16, int cap, int V, const VerifyItem* items,
                         int nitems, const float* zbuf, float T, PhiloxKeys keys,
                         VerifyResult* results, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL((verify_stage_kernel<uint16_t>), dim3(nitems), dim3(kVerifyThreads), 0, s,
                       static_cast<const uint16_t*>(target), cap, V, items, nitems, zbuf, T, keys,
                       results);
  else
    hipLaunchKernelGGL((verify_stage_kernel<float>), dim3(nitems), dim3(kVerifyThreads), 0, s,
                       static_cast<const float*>(target), cap, V, items, nitems, zbuf, T, keys,
                       results);
}

}  // namespace ts
