// Expansion kernels for f32 drafter tensors with KS = 8.
#include "expand_inst.hpp"

namespace ts {
template void launch_eval_t<float, 8>(const ExpandParams&, int, int, bool, bool, dim3, dim3, hipStream_t);
template void launch_merge_t<float, 8>(const MergeParams&, int, dim3, dim3, hipStream_t);
template int eval_blocks_per_cu_t<float, 8>(int, int, bool, bool, int);
}  // namespace ts
