// Streaming-pass kernels for bf16 drafter tensors with KS = 8.  Compiled
// with the max-ILP instruction scheduler (the build's per-unit flags): on the
// 2048-parent serving frontier the pass took 121.3 us against 122.6 with
// sequential draws and 275.0 against 290.4 with Gumbel draws, while the
// merge kernels, in their own unit, are faster with the default scheduler.
#include "expand_inst.hpp"

namespace ts {
template void launch_eval_t<uint16_t, 8>(const ExpandParams&, int, int, bool, bool, dim3, dim3, hipStream_t);
template int eval_blocks_per_cu_t<uint16_t, 8>(int, int, bool, bool, int);
}  // namespace ts
