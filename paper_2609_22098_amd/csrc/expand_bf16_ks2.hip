// Expansion kernels for bf16 drafter tensors with KS = 2.
#include "expand_inst.hpp"

namespace ts {
template void launch_eval_t<uint16_t, 2>(const ExpandParams&, int, int, bool, bool, dim3, dim3, hipStream_t);
template void launch_merge_t<uint16_t, 2>(const MergeParams&, int, dim3, dim3, hipStream_t);
template int eval_blocks_per_cu_t<uint16_t, 2>(int, int, bool, bool, int);
}  // namespace ts
