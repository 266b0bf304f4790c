// Draft-side tree expansion (Algorithm 2, ExpandLayer), batched over the
// pooled requests of a draft server: every frontier node of every request
// gets as children the top-k tokens of the draft's next-token distribution at
// that node, with their draft probabilities q (which the correction step of
// verification needs).
//
// One workgroup of 1024 threads per frontier row (request b, node f).
// Rank keys are the float32 order key of the logit, then the inverted token
// id, so that equal logits rank by increasing id and every key is unique.
//  1. Each wave scans its share of the row, 64 entries per step, keeping the
//     k best keys seen so far sorted across its lanes (lane i: the i-th best).
//     A ballot against the list's k-th key finds the few entries that enter
//     it; each is placed by counting the better keys and shifting the rest
//     down one lane.  The wave also keeps the row maximum.
//  2. The waves' lists meet in LDS and wave 0 selects the k best of them the
//     same way; the row maximum M is combined across waves.
//  3. A second pass over the row (now in L2) sums exp(logit - M) in float64,
//     giving lse; q(child) = exp(logit - lse) with the difference kept exact.
// Children of node f are numbered first_child + f*k + j in rank order.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kExpThreads = 1024;
constexpr int kExpWaves = kExpThreads / kWave;
constexpr int kExpUnroll = 32;  // 64-entry steps whose loads a wave issues together (a 32000-entry row: one round)

__device__ __forceinline__ uint64_t rank_key(float x, int v) {
  return ((uint64_t)order_key(x) << 32) | (uint64_t)(0xffffffffu - (uint32_t)v);
}

// Offer this lane's key to the wave's sorted list (lane i < k holds the i-th
// best key so far, 0 below; thr is the k-th best, 0 while the list is short).
// Keys are unique and never 0 for a real entry.  Every cross-lane move is a
// lane read (uniform source lane) or a one-lane DPP shift, so an insertion
// costs no LDS round trip.
__device__ __forceinline__ void offer(uint64_t key, int k, uint64_t& lst, uint64_t& thr) {
  const int lane = threadIdx.x & 63;
  unsigned long long cand = __ballot(key > thr);
  while (cand) {
    const int c = __ffsll(cand) - 1;
    cand &= cand - 1;
    const uint64_t kc = lane_u64(key, c);
    if (kc <= thr) continue;
    const int pos = __popcll(__ballot(lane < k && lst > kc));
    const uint64_t up = dpp_u64<kDppWaveShr1>(lst);
    lst = lane == pos ? kc : (lane > pos && lane < k ? up : lst);
    thr = lane_u64(lst, k - 1);
  }
}

__global__ __launch_bounds__(kExpThreads)
void expand_kernel(ExpandArgs e, const float* __restrict__ logits, int32_t* __restrict__ tokens,
                   int32_t* __restrict__ parent, float* __restrict__ q_child) {
  __shared__ uint64_t s_lst[kExpWaves][kExpandMaxK];
  __shared__ float s_m[kExpWaves];
  __shared__ double s_s[kExpWaves];
  const int row = blockIdx.x;  // b * F + f
  const int b = row / e.F;
  const int f = row - b * e.F;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const float* x = logits + (int64_t)row * e.V;

  // 1. Wave lists and row maximum.
  uint64_t lst = 0, thr = 0;
  float m = -INFINITY;
  for (int base = wave * kWave; base < e.V; base += kExpThreads * kExpUnroll) {
    float xs[kExpUnroll];
#pragma unroll
    for (int u = 0; u < kExpUnroll; ++u) xs[u] = x[min(base + u * kExpThreads + lane, e.V - 1)];
#pragma unroll
    for (int u = 0; u < kExpUnroll; ++u) {
      const int v = base + u * kExpThreads + lane;
      const bool in = v < e.V;
      m = in ? fmaxf(m, xs[u]) : m;
      offer(in ? rank_key(xs[u], v) : 0, e.k, lst, thr);
    }
  }
  if (lane < kExpandMaxK) s_lst[wave][lane] = lane < e.k ? lst : 0;
  const float mw = wave_max(m);
  if (lane == 0) s_m[wave] = mw;
  __syncthreads();
  float M = s_m[0];
#pragma unroll
  for (int w = 1; w < kExpWaves; ++w) M = fmaxf(M, s_m[w]);

  // 3. Sum of exp(logit - M), float64, fixed order.
  double acc = 0.0;
  for (int base = wave * kWave; base < e.V; base += kExpThreads * kExpUnroll) {
    float xs[kExpUnroll];
#pragma unroll
    for (int u = 0; u < kExpUnroll; ++u) xs[u] = x[min(base + u * kExpThreads + lane, e.V - 1)];
#pragma unroll
    for (int u = 0; u < kExpUnroll; ++u) {
      const bool in = base + u * kExpThreads + lane < e.V;
      acc += in && xs[u] != -INFINITY ? (double)expf(xs[u] - M) : 0.0;
    }
  }
  const double sw = wave_sum_f64(acc);
  if (lane == 0) s_s[wave] = sw;
  __syncthreads();
  if (wave != 0) return;
  double S = 0.0;
#pragma unroll
  for (int w = 0; w < kExpWaves; ++w) S += s_s[w];
  const float lse = (float)((double)M + log(S));

  // 2. Wave 0 selects the k best of the waves' lists.
  uint64_t best = 0, bthr = 0;
  constexpr int kCand = kExpWaves * kExpandMaxK;
#pragma unroll
  for (int i = 0; i < kCand / kWave; ++i) {
    const int c = i * kWave + lane;
    offer(s_lst[c / kExpandMaxK][c % kExpandMaxK], e.k, best, bthr);
  }
  if (lane < e.k) {
    const int v = (int)(0xffffffffu - (uint32_t)(best & 0xffffffffu));
    const int64_t o = (int64_t)b * e.N + e.first_child + f * e.k + lane;
    tokens[o] = v;
    parent[o] = e.frontier0 < 0 ? -1 : e.frontier0 + f;
    q_child[o] = exp_diff(x[v], lse);
  }
}

}  // namespace

hipError_t launch_expand(const ExpandArgs& e, const float* logits, int32_t* tokens, int32_t* parent, float* q_child,
                         hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int64_t rows = (int64_t)e.B * e.F;
  if (rows <= 0) return hipSuccess;
  if (rows > 0x7fffffff || e.k < 1 || e.k > kExpandMaxK || e.k > e.V) return hipErrorInvalidValue;
  hipExtLaunchKernelGGL(expand_kernel, dim3((unsigned)rows), dim3(kExpThreads), 0, stream, ev_start, ev_stop, 0, e,
                        logits, tokens, parent, q_child);
  return hipGetLastError();
}

}  // namespace sdv
