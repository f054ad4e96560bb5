// Tree attention mask and position ids (ts_tree_mask).
//
// Row i of a request's flattened tree sees the nodes on its root path,
// itself included (§3.2 item 3; the per-row ancestor bitmask of §5).  One
// workgroup per request copies the request's parent array into LDS; each
// (row, word) item then walks the row's parent chain (at most depth + 1
// steps) and keeps the ancestors that fall into its 32-bit word.  Items
// are consecutive words, so the mask rows are written contiguously.
#pragma once

#include "device_common.hpp"

namespace ts {

constexpr int kMaskThreads = 256;

__global__ __launch_bounds__(kMaskThreads) void tree_mask_kernel(const int32_t* parent, const int32_t* n,
                                                                  int R, int cap, int W,
                                                                  const int32_t* pos_offset,
                                                                  uint32_t* mask, int32_t* pos) {
  extern __shared__ int32_t par[];  // cap entries
  const int q = blockIdx.x;
  if (q >= R) return;
  int nq = n[q];
  nq = nq < 0 ? -1 : min(nq, cap - 1);
  const int32_t* pq = parent + (size_t)q * cap;
  for (int i = threadIdx.x; i < cap; i += kMaskThreads) par[i] = i <= nq ? pq[i] : -1;
  __syncthreads();
  const int off = pos_offset ? pos_offset[q] : 0;
  const int items = cap * W;
  uint32_t* mq = mask + (size_t)q * cap * W;
  int32_t* posq = pos + (size_t)q * cap;
  for (int t = threadIdx.x; t < items; t += kMaskThreads) {
    const int i = t / W, w = t - (t / W) * W;
    uint32_t bits = 0u;
    int depth = 0;
    if (i <= nq) {
      int a = i;
      for (;;) {
        if ((a >> 5) == w) bits |= 1u << (a & 31);
        if (a == 0) break;
        const int pa = par[a];
        if (pa < 0 || pa >= a) break;  // a broken chain stops here
        a = pa;
        ++depth;
      }
    }
    mq[t] = bits;
    if (w == 0) posq[i] = i <= nq ? off + depth : -1;
  }
}

}  // namespace ts
