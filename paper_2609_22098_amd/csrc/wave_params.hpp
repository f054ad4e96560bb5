// Parameter blocks of the device-resident tree waves (kernels in wave_kernels.hpp).
#pragma once

#include "device_common.hpp"

namespace ts {

constexpr int kWaveThreads = 256;
constexpr int kWaveMaxN = TS_DEVICE_WAVES_MAX_N;  // list capacity per request (N)
constexpr int kWaveMaxNew = TS_DEVICE_WAVES_MAX_CHILDREN;  // children of a request in one wave

struct WaveSlot {  // 32 bytes
  float key;       // slot key: the pop priority
  int depth;       // depth of the child the slot creates
  uint64_t path;   // the child's structural path id
  int token;
  float log_surv, log_q0, log_qT;
};

struct WaveSpan {  // a request's rows in a wave's frontier
  int off, cnt;
};

struct WaveParams {
  int R, N, K, D;
  const int32_t* anchor;   // [R] root tokens
  const float* log_theta;  // [R] log(theta_q), -inf for theta = 0
  // the two arrays above as the host wrote them (pinned host memory, read by
  // the init step, which writes them to anchor_w and log_theta_w: the same
  // buffers as anchor and log_theta)
  const int32_t* anchor_host;
  const float* log_theta_host;
  int32_t* anchor_w;
  float* log_theta_w;
  volatile int32_t* host_count;  // [D + 2] pinned host memory: the size of wave w, written
                                 // by the last control workgroup of wave w - 1
  WaveSlot* list;          // [R][N] best known slots with key >= log(theta), pop order
  int* lsize;              // [R] entries of list in use
  int* evals;              // [R] parents evaluated so far
  // [D + 2] wave w: frontier size in the low 32 bits (the expansion reads
  // that half as an int), control workgroups of wave w - 1 finished in the high
  uint64_t* pcount;
  ts_parent* par[2];       // frontier of wave w in par[w & 1]
  WaveSpan* span[2];       // [R] rows of each request in par[w & 1]
  // outputs of the current wave's expansion, [P][K] row-major
  const int32_t* child_token;
  const float* child_log_q0;
  const float* child_log_qT;
  const float* child_log_surv;
  const float* slot_key;
};

// A tree in the ts_tree layout, device arrays.
struct WaveTreeOut {
  int cap;
  int32_t* n;
  int32_t* token;
  int32_t* parent;
  int32_t* depth;
  int32_t* rank;
  uint64_t* path;
  float* log_surv;
  float* log_q0;
  float* log_qT;
  float* key;
  int32_t* evals;  // may be null
  int32_t* err;    // may be null: set to 1 when a slot's parent is not listed
};

}  // namespace ts
