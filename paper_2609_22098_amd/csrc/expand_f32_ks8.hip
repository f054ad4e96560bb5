// Expansion kernels for f32 drafter tensors with KS = 8.
#include "expand_inst.hpp"

namespace ts {
template void launch_eval_t<float, 8>(const ExpandParams&, int, bool, bool, bool, dim3, dim3, hipStream_t);
template void launch_merge_t<float, 8>(const MergeParams&, bool, dim3, dim3, hipStream_t);
template int eval_blocks_per_cu_t<float, 8>(int, bool, bool, bool, int);
}  // namespace ts
