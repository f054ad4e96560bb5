// Kernel launchers shared by the host API.  Each (dtype, rank) pair is
// instantiated in its own translation unit so the kernels compile in parallel.
#pragma once

#include "merge_kernels.hpp"
#include "verify_kernels.hpp"
#include "wave_params.hpp"

namespace ts {

// Streaming pass of the expansion.  KS = r / 32 (bf16) or r / 4 (f32); nb =
// parent blocks of 16 per wave (1, 2 or 4); mode is kModeGreedy, kModeGumbel
// or kModeSeq; store_z (the verification recompute) runs with nb == 1 and no
// draws.  lds selects the LDS-staged bf16 kernel (V % 8 == 0, four waves).
template <typename TE, int KS>
void launch_eval_t(const ExpandParams& p, int nb, int mode, bool store_z, bool lds, dim3 grid,
                   dim3 block, hipStream_t s);
// Resident blocks per CU of the streaming kernel a launch would use (0 if unknown).
template <typename TE, int KS>
int eval_blocks_per_cu_t(int nb, int mode, bool store_z, bool lds, int block);
// Per-parent merge: exact top-k, the draws, child scoring.
template <typename TE, int KS>
void launch_merge_t(const MergeParams& p, int mode, dim3 grid, dim3 block, hipStream_t s);

// Verification.
void launch_verify_argmax(const void* target, bool bf16, int V, const int* rows, int nrows,
                          int* argmax_out, float* gap_out, hipStream_t s);
// Tree attention mask and position ids, one workgroup per request.
void launch_tree_mask(const int32_t* parent, const int32_t* n, int R, int cap, const int32_t* pos_offset,
                      uint32_t* mask, int32_t* pos, hipStream_t s);
// Device-resident tree waves: set-up, the control step after wave w's
// expansion (one workgroup per request), the trees.
void launch_wave_init(const WaveParams& wp, hipStream_t s);
void launch_wave_control(const WaveParams& wp, int w, hipStream_t s);
void launch_wave_tree(const WaveParams& wp, const WaveTreeOut& o, const WaveTreeOut& o2, hipStream_t s);
// Calibration: greedy labels of host-built trees, and the two-scalar fit.
void launch_calib_labels(const int32_t* parent, const int32_t* token, const float* log_q0, const int32_t* n,
                         int R, int cap, const int32_t* greedy, const int32_t* off, float* x, int32_t* y,
                         int32_t* sel, hipStream_t s);
void launch_calib_fit(const float* x, const int32_t* y, const int32_t* sel, int n, int max_iter, double tol,
                      float* out, hipStream_t s);
// One level of the T > 0 walk: pass A, stages 1..max(mmax, 1), bonus, resolve.
void launch_verify_level(const VerifyPass& vp, bool bf16, int mmax, hipStream_t s);
// The same level in one launch with register-resident chunks: quads per
// thread, resident workgroups per CU (0 if unknown), the launch, and the
// clearing of its counters.
struct VFused;
int verify_fused_quads(bool bf16);
int verify_fused_blocks_per_cu(bool bf16);
void launch_verify_fused(const VerifyPass& vp, const VFused& f, bool bf16, hipStream_t s);
void launch_verify_clear(int* p, int n, hipStream_t s);

}  // namespace ts
