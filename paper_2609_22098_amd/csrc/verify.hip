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

template <typename TT>
static void verify_level_t(const VerifyPass& vp, int mmax, hipStream_t s) {
  const dim3 grid(vp.nitems * vp.nchunks), block(kVerifyThreads);
  const int J = mmax > 1 ? mmax : 1;
  hipLaunchKernelGGL((verify_pass_a_kernel<TT>), grid, block, 0, s, vp);
  for (int j = 1; j <= J; ++j) hipLaunchKernelGGL((verify_stage_kernel<TT>), grid, block, 0, s, vp, j);
  hipLaunchKernelGGL((verify_resolve_kernel<TT>), dim3(vp.nitems), dim3(64), 0, s, vp, J);
}

void launch_verify_level(const VerifyPass& vp, bool bf16, int mmax, hipStream_t s) {
  if (bf16)
    verify_level_t<uint16_t>(vp, mmax, s);
  else
    verify_level_t<float>(vp, mmax, s);
}

}  // namespace ts
