// Acceptance test, first rejection, residual resampling and output assembly.
//
// One workgroup per request:
//  1. wave 0 evaluates the gamma ratio tests in float64 (lane i tests x_{i+1}:
//     u < p_i(x_i) / q_i(x_i)) and finds the first failure with a ballot;
//  2. the four waves sum the unnormalised continuation distribution
//     r = max(0, p_{l+1} - q_{l+1}) (or p_{gamma+1} after a full accept) over
//     512-entry segments of the vocabulary, in float64;
//  3. wave 0 prefix-sums the segment totals (Z is the last one), finds the
//     segment holding u * Z and scans it in token order for the first entry
//     whose cumulative sum exceeds u * Z.
// p(v) = exp(logit - lse) is evaluated with the difference kept exact (TwoSum)
// so its error stays a few float32 ulp, far below the 1e-6 decision band.
#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kAccThreads = 256;
constexpr int kAccWaves = 4;
constexpr int kSeg = 512;
constexpr int kMaxSeg = 4096;  // vocabularies up to 2,097,152 entries

// exp(a - b), with a - b carried exactly as s + err.
__device__ __forceinline__ float exp_diff(float a, float b) {
  const float s = a - b;
  const float bb = s - a;
  const float err = (a - (s - bb)) + (-b - bb);
  const float e = expf(s);
  return fmaf(e, err, e);
}

struct RowView {
  const float* x;    // logits or probabilities of the row p_{l+1}
  const float* q;    // q_{l+1}, or nullptr for the bonus row
  float lse;
  bool from_logits;
  bool residual;

  __device__ __forceinline__ float r(int v) const {
    const float p = from_logits ? exp_diff(x[v], lse) : x[v];
    if (!residual) return p;
    const float d = p - q[v];
    return d > 0.f ? d : 0.f;
  }
};

__global__ __launch_bounds__(kAccThreads)
void accept_kernel(int gamma, int V, const AcceptBatch bt, const float* __restrict__ x,
                   const float* __restrict__ row_lse, const float* __restrict__ q_draft,
                   const int32_t* __restrict__ draft_tok, const float* __restrict__ u,
                   int32_t* __restrict__ accept_len, int32_t* __restrict__ out_tok,
                   int32_t* __restrict__ new_kv_len) {
  __shared__ double seg[kMaxSeg];
  __shared__ int s_l;
  __shared__ int s_t;
  __shared__ double s_z;

  const int b = blockIdx.x;
  const int req = bt.req0 + b;
  const int G = gamma + 1;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const float* xr = x + (int64_t)req * G * V;
  const bool from_logits = row_lse != nullptr;

  // 1. Ratio tests and the first rejection.
  if (wave == 0) {
    bool fail = false;
    if (lane < gamma) {
      const int tok = draft_tok[(int64_t)req * gamma + lane];
      double ratio = 0.0;
      if (tok >= 0 && tok < V) {
        const double px = from_logits
                              ? exp((double)xr[(int64_t)lane * V + tok] - (double)row_lse[(int64_t)req * G + lane])
                              : (double)xr[(int64_t)lane * V + tok];
        const double qx = (double)q_draft[((int64_t)req * gamma + lane) * V + tok];
        ratio = (px <= 0.0) ? 0.0 : (qx <= 0.0 ? (double)INFINITY : px / qx);
      }
      fail = !((double)u[(int64_t)req * G + lane] < ratio);
    }
    const unsigned long long fails = __ballot(fail);
    if (lane == 0) s_l = fails ? (__ffsll(fails) - 1) : gamma;
  }
  __syncthreads();
  const int l = s_l;

  RowView rv;
  rv.x = xr + (int64_t)l * V;
  rv.q = (l < gamma) ? q_draft + ((int64_t)req * gamma + l) * V : nullptr;
  rv.lse = from_logits ? row_lse[(int64_t)req * G + l] : 0.f;
  rv.from_logits = from_logits;
  rv.residual = l < gamma;
  const int nseg = (V + kSeg - 1) / kSeg;
  const double uf = (double)u[(int64_t)req * G + gamma];

  double z = 0.0;
  for (int attempt = 0; attempt < 2; ++attempt) {
    // 2. Segment sums.
    for (int sg = wave; sg < nseg; sg += kAccWaves) {
      double acc = 0.0;
#pragma unroll 4
      for (int e = 0; e < kSeg / kWave; ++e) {
        const int v = sg * kSeg + e * kWave + lane;
        if (v < V) acc += (double)rv.r(v);
      }
      acc = wave_sum_f64(acc);
      if (lane == 0) seg[sg] = acc;
    }
    __syncthreads();
    // 3a. Inclusive prefix of the segment sums.
    if (wave == 0) {
      double carry = 0.0;
      for (int base = 0; base < nseg; base += kWave) {
        const int i = base + lane;
        const double v = i < nseg ? seg[i] : 0.0;
        const double c = wave_inclusive_scan_f64(v) + carry;
        if (i < nseg) seg[i] = c;
        carry = __shfl(c, 63);
      }
      if (lane == 0) s_z = carry;
    }
    __syncthreads();
    z = s_z;
    if (z > 0.0 || !rv.residual) break;
    // Residual vanished (possible only through rounding): sample from p_{l+1}.
    rv.residual = false;
    __syncthreads();
  }

  // 3b. Locate u * Z and scan its segment in token order.
  if (wave == 0) {
    const double thr = uf * z;
    int found = -1;
    for (int base = 0; base < nseg && found < 0; base += kWave) {
      const int i = base + lane;
      const unsigned long long hit = __ballot(i < nseg && seg[i] > thr);
      if (hit) found = base + __ffsll(hit) - 1;
    }
    int t = -1;
    if (found >= 0) {
      double c = found > 0 ? seg[found - 1] : 0.0;
      int last_pos = -1;
      for (int e = 0; e < kSeg / kWave && t < 0; ++e) {
        const int v = found * kSeg + e * kWave + lane;
        const double r = v < V ? (double)rv.r(v) : 0.0;
        const double cum = wave_inclusive_scan_f64(r) + c;
        const unsigned long long hit = __ballot(v < V && r > 0.0 && cum > thr);
        if (hit) t = found * kSeg + e * kWave + __ffsll(hit) - 1;
        const unsigned long long pos = __ballot(v < V && r > 0.0);
        if (pos) last_pos = found * kSeg + e * kWave + 63 - __clzll(pos);
        c = __shfl(cum, 63);
      }
      if (t < 0) t = last_pos;  // rounding put u * Z past this segment's scan
    }
    if (t < 0) {
      // No prefix sum exceeds u * Z: the largest token with mass.
      for (int sg = nseg - 1; sg >= 0 && t < 0; --sg) {
        for (int e = kSeg / kWave - 1; e >= 0 && t < 0; --e) {
          const int v = sg * kSeg + e * kWave + lane;
          const unsigned long long pos = __ballot(v < V && rv.r(v) > 0.f);
          if (pos) t = sg * kSeg + e * kWave + 63 - __clzll(pos);
        }
      }
      if (t < 0) t = 0;  // no mass at all (non-finite input)
    }
    if (lane == 0) s_t = t;
  }
  __syncthreads();

  // Output assembly.
  if (threadIdx.x < G) {
    const int i = threadIdx.x;
    int32_t v = -1;
    if (i < l) v = draft_tok[(int64_t)req * gamma + i];
    else if (i == l) v = s_t;
    out_tok[(int64_t)req * G + i] = v;
  }
  if (threadIdx.x == 0) {
    accept_len[req] = l;
    if (new_kv_len != nullptr && bt.has_kv_len) new_kv_len[req] = bt.kv_len[b] - gamma + l;
  }
}

}  // namespace

hipError_t launch_accept(int gamma, int V, const AcceptBatch& bt, const float* x, const float* row_lse,
                         const float* q_draft, const int32_t* draft_tok, const float* u,
                         int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len, hipStream_t stream) {
  if (bt.nreq <= 0) return hipSuccess;
  hipLaunchKernelGGL(accept_kernel, dim3(bt.nreq), dim3(kAccThreads), 0, stream, gamma, V, bt, x, row_lse,
                     q_draft, draft_tok, u, accept_len, out_tok, new_kv_len);
  return hipGetLastError();
}

}  // namespace sdv
