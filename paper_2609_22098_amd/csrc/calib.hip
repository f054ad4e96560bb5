// Launchers of the calibration kernels.
#include "calib_kernels.hpp"
#include "launch.hpp"

namespace ts {

void launch_calib_labels(const int32_t* parent, const int32_t* token, const float* log_q0, const int32_t* n,
                         int R, int cap, const int32_t* greedy, const int32_t* off, float* x, int32_t* y,
                         int32_t* sel, hipStream_t s) {
  hipLaunchKernelGGL(calib_labels_kernel, dim3(R), dim3(kCalibThreads), 0, s, parent, token, log_q0, n, cap,
                     greedy, off, x, y, sel);
}

void launch_calib_fit(const float* x, const int32_t* y, const int32_t* sel, int n, int max_iter, double tol,
                      float* out, hipStream_t s) {
  hipLaunchKernelGGL(calib_fit_kernel, dim3(1), dim3(kFitThreads), 0, s, x, y, sel, n, max_iter, tol, out);
}

}  // namespace ts
