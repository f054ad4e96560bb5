// Instantiations of the verification kernels.
#include "launch.hpp"
#include "verify_fused.hpp"

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

int verify_fused_quads(bool bf16) { return bf16 ? kFusedQuadsBf16 : kFusedQuadsF32; }

int verify_fused_blocks_per_cu(bool bf16) {
  static int cached[2] = {-1, -1};
  int& n = cached[bf16 ? 1 : 0];
  if (n < 0) {
    int b = 0;
    const hipError_t e =
        bf16 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                   &b, verify_fused_kernel<uint16_t, kFusedQuadsBf16>, kVerifyThreads, 0)
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                   &b, verify_fused_kernel<float, kFusedQuadsF32>, kVerifyThreads, 0);
    n = (e == hipSuccess && b > 0) ? b : 0;
  }
  return n;
}

void launch_verify_fused(const VerifyPass& vp, const VFused& f, bool bf16, hipStream_t s) {
  const dim3 grid(vp.nitems * f.cpi), block(kVerifyThreads);
  if (bf16)
    hipLaunchKernelGGL((verify_fused_kernel<uint16_t, kFusedQuadsBf16>), grid, block, 0, s, vp, f);
  else
    hipLaunchKernelGGL((verify_fused_kernel<float, kFusedQuadsF32>), grid, block, 0, s, vp, f);
}

// Clears n words (the counters and the flag before a ts_verify call's first
// fused launch).
__global__ void verify_clear_kernel(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

void launch_verify_clear(int* p, int n, hipStream_t s) {
  if (n > 0) hipLaunchKernelGGL(verify_clear_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, n);
}

}  // namespace ts
