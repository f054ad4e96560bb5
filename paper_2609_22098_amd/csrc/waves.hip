// Launchers of the device-resident tree waves.
#include <algorithm>

#include "launch.hpp"
#include "wave_kernels.hpp"

namespace ts {

void launch_wave_init(const WaveParams& wp, hipStream_t s) {
  const int blocks = std::max(1, (wp.R + kWaveThreads - 1) / kWaveThreads);
  hipLaunchKernelGGL(wave_init_kernel, dim3(blocks), dim3(kWaveThreads), 0, s, wp);
}

void launch_wave_control(const WaveParams& wp, int w, hipStream_t s) {
  hipLaunchKernelGGL(wave_control_kernel, dim3(wp.R), dim3(kWaveThreads), 0, s, wp, w);
}

void launch_wave_tree(const WaveParams& wp, const WaveTreeOut& o, const WaveTreeOut& o2, hipStream_t s) {
  hipLaunchKernelGGL(wave_tree_kernel, dim3(wp.R), dim3(kWaveThreads), 0, s, wp, o, o2);
}

}  // namespace ts
