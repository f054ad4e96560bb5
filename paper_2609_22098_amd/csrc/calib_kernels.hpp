// Calibration of the edge-acceptance estimate (§3.4 Eq. 3).
//
// Labels: in a greedy round the verifier shows, for every materialised node,
// whether its token is the target's greedy choice at its parent (the row of
// a node attends only to its root path).  An edge is labelled 1 when it is;
// the two scalars are fitted on the edges whose ancestors were all accepted,
// the population that path-survival products condition on.
//
// Fit: the maximum-likelihood (a, b) of y ~ Bernoulli(sigmoid(a x + b)) with
// x = logit q0, by Newton's method with step halving.  One workgroup; every
// sum is accumulated in fp64 in a fixed order (per thread, then a fixed
// tree), so the fit is deterministic.
#pragma once

#include "device_common.hpp"

namespace ts {

constexpr int kCalibThreads = 256;
constexpr int kFitThreads = 1024;

// One workgroup per request.  parent, token, log_q0: [R][cap] (host tree
// copied up); greedy[off[q] + i]: the target argmax of row i of request q,
// for i <= n[q].  Outputs [R][cap]: x = logit q0, y in {0, 1}, sel in {0, 1};
// row 0 and rows past n: x NaN, y -1, sel 0.
__global__ __launch_bounds__(kCalibThreads) void calib_labels_kernel(
    const int32_t* parent, const int32_t* token, const float* log_q0, const int32_t* n, int cap,
    const int32_t* greedy, const int32_t* off, float* x, int32_t* y, int32_t* sel) {
  const int q = blockIdx.x;
  const int nq = min(max(n[q], 0), cap - 1);
  const size_t b = (size_t)q * cap;
  const int32_t* gq = greedy + off[q];
  for (int i = threadIdx.x; i < cap; i += kCalibThreads) {
    float xi = __builtin_nanf("");
    int32_t yi = -1, si = 0;
    if (i >= 1 && i <= nq) {
      const int p = parent[b + i];
      if (p >= 0 && p < i) {
        yi = token[b + i] == gq[p] ? 1 : 0;
        // ancestors-accepted: every edge on the root path of the parent
        int ok = 1, j = p, steps = 0;
        while (j > 0 && steps < cap) {
          const int pj = parent[b + j];
          if (pj < 0 || pj >= j) { ok = 0; break; }
          if (token[b + j] != gq[pj]) { ok = 0; break; }
          j = pj;
          ++steps;
        }
        si = ok;
      }
      const float lq = log_q0[b + i];
      if (lq < 0.0f) {
        const float l1m = (lq > -kLn2) ? logf(-expm1f(lq)) : log1pf(-expf(lq));
        xi = lq - l1m;
      } else {
        xi = __builtin_huge_valf();  // q0 == 1
      }
    }
    x[b + i] = xi;
    y[b + i] = yi;
    sel[b + i] = si;
  }
}

__device__ __forceinline__ double fit_block_sum(double v, double* red) {
  const int t = threadIdx.x;
  red[t] = v;
  __syncthreads();
  for (int s = kFitThreads / 2; s > 0; s >>= 1) {
    if (t < s) red[t] += red[t + s];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__device__ __forceinline__ double softplus_d(double z) {
  return z > 0.0 ? z + log1p(exp(-z)) : log1p(exp(z));
}

// A sample takes part iff sel = 1, y is 0 or 1 and x is finite.
__device__ __forceinline__ bool fit_sample(const float* x, const int32_t* y, const int32_t* sel, int i) {
  return sel[i] == 1 && (y[i] == 0 || y[i] == 1) && __builtin_isfinite(x[i]);
}

// out: {a, b, mean negative log-likelihood, Newton steps}; NaN when no sample
// takes part or the Hessian is singular.
__global__ __launch_bounds__(kFitThreads) void calib_fit_kernel(const float* x, const int32_t* y,
                                                                const int32_t* sel, int n, int max_iter,
                                                                double tol, float* out) {
  __shared__ double red[kFitThreads];
  const int t = threadIdx.x;
  auto nll_at = [&](double a, double b) {
    double acc = 0.0;
    for (int i = t; i < n; i += kFitThreads)
      if (fit_sample(x, y, sel, i)) {
        const double z = a * (double)x[i] + b;
        acc += softplus_d(z) - (double)y[i] * z;
      }
    return fit_block_sum(acc, red);
  };
  double cnt = 0.0;
  for (int i = t; i < n; i += kFitThreads) cnt += fit_sample(x, y, sel, i) ? 1.0 : 0.0;
  cnt = fit_block_sum(cnt, red);
  const double nan = __builtin_nan("");
  double a = 0.0, b = 0.0;
  double f = nll_at(a, b);
  int steps = 0;
  bool ok = cnt > 0.0;
  for (int it = 1; ok && it <= max_iter; ++it) {
    steps = it;
    double g0 = 0.0, g1 = 0.0, h00 = 0.0, h01 = 0.0, h11 = 0.0;
    for (int i = t; i < n; i += kFitThreads)
      if (fit_sample(x, y, sel, i)) {
        const double xi = x[i];
        const double p = 1.0 / (1.0 + exp(-(a * xi + b)));
        const double r = p - (double)y[i], w = p * (1.0 - p);
        g0 += r * xi;
        g1 += r;
        h00 += w * xi * xi;
        h01 += w * xi;
        h11 += w;
      }
    g0 = fit_block_sum(g0, red);
    g1 = fit_block_sum(g1, red);
    h00 = fit_block_sum(h00, red);
    h01 = fit_block_sum(h01, red);
    h11 = fit_block_sum(h11, red);
    const double det = h00 * h11 - h01 * h01;
    if (!(det != 0.0) || !__builtin_isfinite(det)) {
      ok = false;
      break;
    }
    const double da = (h11 * g0 - h01 * g1) / det, db = (h00 * g1 - h01 * g0) / det;
    double step = 1.0, fa = a, fb = b, fc = f;
    for (;;) {
      fa = a - step * da;
      fb = b - step * db;
      fc = nll_at(fa, fb);
      if (fc <= f || step < 0x1p-30) break;
      step *= 0.5;
    }
    a = fa;
    b = fb;
    f = fc;
    if (fmax(fabs(step * da), fabs(step * db)) < tol) break;
  }
  if (t == 0) {
    out[0] = ok ? (float)a : (float)nan;
    out[1] = ok ? (float)b : (float)nan;
    out[2] = ok ? (float)(f / cnt) : (float)nan;
    out[3] = (float)steps;
  }
}

}  // namespace ts
