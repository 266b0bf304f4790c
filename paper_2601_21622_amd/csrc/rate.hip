// Acceptance rate of every draft position (Sec. 3, eq. beta_cond): for
// request b and draft position i, beta = the sum over the vocabulary of
// min(p_i(v), q_i(v)), where p_i is the target distribution at position i
// (row b * (gamma + 1) + i: exp(logit - lse), or the probabilities given) and
// q_i the draft distribution x_{i+1} was drawn from.  It is one minus the
// total-variation distance of the two, and the probability that the ratio
// test accepts a draft drawn from q_i; averaged over positions it is the
// beta of the expected accept length (eq. El_closed).
//
// Two launches.  The slice kernel runs S workgroups of 256 threads per row;
// workgroup (r, s) sums min(p, q) over vocabulary slice s of row r in float64
// (each thread in index order, then across the waves in a fixed order) into
// part[r][s].  The final kernel adds each row's S partials in order, so the
// result depends only on the shapes.  HBM-bound: 8 bytes (p and q) per entry,
// read once, each thread keeping 8 loads of each row in flight.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kRateThreads = 256;
constexpr int kRateUnroll = 8;                         // entries per thread per pass
constexpr int kRateSpan = kRateThreads * kRateUnroll;  // entries per workgroup pass
constexpr int kRateTargetGroups = 2048;                // slice workgroups aimed for per launch

struct RatePlan {
  int rows, S, per;  // rows = B * gamma; S slices of `per` entries (the last may be shorter)
};

RatePlan rate_plan(int B, int gamma, int V) {
  RatePlan p;
  p.rows = B * gamma;
  const int max_s = (V + kRateSpan - 1) / kRateSpan;
  const int want = (kRateTargetGroups + p.rows - 1) / p.rows;
  const int s = std::max(1, std::min(want, max_s));
  p.per = (V + s - 1) / s;
  p.per = (p.per + kWave - 1) / kWave * kWave;
  p.S = (V + p.per - 1) / p.per;
  return p;
}

// Workgroup blockIdx.x = r * S + s.
template <bool LOGITS>
__global__ __launch_bounds__(kRateThreads)
void rate_slice_kernel(int gamma, int V, int S, int per, const float* __restrict__ x, const float* __restrict__ lse,
                       const float* __restrict__ q, double* __restrict__ part) {
  __shared__ double red[kRateThreads / kWave];
  const int r = blockIdx.x / S;
  const int s = blockIdx.x - r * S;
  const int b = r / gamma;
  const int64_t xr = (int64_t)b * (gamma + 1) + (r - b * gamma);
  const float* xrow = x + xr * V;
  const float* qrow = q + (int64_t)r * V;
  const float l = LOGITS ? lse[xr] : 0.f;
  const int v0 = s * per;
  const int v1 = min(V, v0 + per);
  double acc = 0.0;
  for (int base = v0; base < v1; base += kRateSpan) {
    float xs[kRateUnroll], qs[kRateUnroll];
#pragma unroll
    for (int e = 0; e < kRateUnroll; ++e) {
      const int v = min(base + e * kRateThreads + (int)threadIdx.x, v1 - 1);
      xs[e] = __builtin_nontemporal_load(xrow + v);
      qs[e] = __builtin_nontemporal_load(qrow + v);
    }
#pragma unroll
    for (int e = 0; e < kRateUnroll; ++e) {
      const float pv = LOGITS ? exp_diff(xs[e], l) : xs[e];
      const bool in = base + e * kRateThreads + (int)threadIdx.x < v1;
      acc += in ? (double)fminf(pv, qs[e]) : 0.0;
    }
  }
  acc = wave_sum_f64(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kRateThreads / kWave; ++w) t += red[w];
    part[(int64_t)r * S + s] = t;
  }
}

__global__ __launch_bounds__(kRateThreads)
void rate_final_kernel(int rows, int S, const double* __restrict__ part, double* __restrict__ beta) {
  const int r = blockIdx.x * kRateThreads + threadIdx.x;
  if (r >= rows) return;
  double t = 0.0;
  for (int s = 0; s < S; ++s) t += part[(int64_t)r * S + s];
  beta[r] = t;
}

}  // namespace

size_t rate_workspace_bytes(int B, int gamma, int V) {
  const RatePlan p = rate_plan(B, gamma, V);
  return sizeof(double) * static_cast<size_t>(p.rows) * p.S;
}

hipError_t launch_rate(int gamma, int V, int B, const float* x, const float* row_lse, const float* q_draft, void* ws,
                       double* beta, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (B <= 0 || gamma <= 0) return hipSuccess;
  const RatePlan p = rate_plan(B, gamma, V);
  double* part = static_cast<double*>(ws);
  const int64_t groups = (int64_t)p.rows * p.S;
  if (groups > 0x7fffffff) return hipErrorInvalidValue;
  if (row_lse != nullptr)
    hipExtLaunchKernelGGL(rate_slice_kernel<true>, dim3((unsigned)groups), dim3(kRateThreads), 0, stream, ev_start,
                          nullptr, 0, gamma, V, p.S, p.per, x, row_lse, q_draft, part);
  else
    hipExtLaunchKernelGGL(rate_slice_kernel<false>, dim3((unsigned)groups), dim3(kRateThreads), 0, stream, ev_start,
                          nullptr, 0, gamma, V, p.S, p.per, x, row_lse, q_draft, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(rate_final_kernel, dim3((p.rows + kRateThreads - 1) / kRateThreads), dim3(kRateThreads), 0,
                        stream, nullptr, ev_stop, 0, p.rows, p.S, part, beta);
  return hipGetLastError();
}

}  // namespace sdv
