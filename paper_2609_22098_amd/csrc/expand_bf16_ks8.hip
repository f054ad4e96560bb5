// Merge kernels for bf16 drafter tensors with KS = 8 (the streaming passes
// are in expand_eval_bf16_ks8.hip).
#include "expand_inst.hpp"

namespace ts {
template void launch_merge_t<uint16_t, 8>(const MergeParams&, int, dim3, dim3, hipStream_t);
}  // namespace ts
