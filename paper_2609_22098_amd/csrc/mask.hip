// Launcher of the tree attention mask kernel.
#include "launch.hpp"
#include "mask_kernels.hpp"

namespace ts {

void launch_tree_mask(const int32_t* parent, const int32_t* n, int R, int cap, const int32_t* pos_offset,
                      uint32_t* mask, int32_t* pos, hipStream_t s) {
  const int W = (cap + 31) / 32;
  hipLaunchKernelGGL(tree_mask_kernel, dim3(R), dim3(kMaskThreads), (size_t)cap * sizeof(int32_t), s, parent,
                     n, R, cap, W, pos_offset, mask, pos);
}

}  // namespace ts
