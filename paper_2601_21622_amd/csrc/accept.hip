// Acceptance test, first rejection, residual resampling and output assembly.
//
// Three short kernels, so that no single workgroup walks a whole vocabulary
// row and each has one or two dependent memory round trips:
//  accept_prepare: one workgroup per request.  Optionally folds the
//     vocabulary kernel's per-tile statistics into the row log-sum-exp of the
//     request's rows (one wave per row); then lanes 0..gamma-1 run the ratio
//     tests in float64 (lane i: u < p_i(x_i) / q_i(x_i)) and a ballot gives
//     the accept length l.
//  accept_segments: one wave per (512-entry vocabulary segment, request) sums,
//     in float64, the unnormalised continuation distribution over its segment:
//     r = max(0, p_{l+1} - q_{l+1}) after a rejection, p_{gamma+1} after a
//     full accept.
//  accept_finalize: one wave per request prefix-sums the segment totals (Z is
//     the last), finds the segment holding u * Z and scans it in token order
//     for the first entry whose running sum exceeds u * Z; then writes the
//     accept length, the emitted tokens and the new cache length.
// p(v) = exp(logit - lse) keeps the difference exact (TwoSum) so its error is
// a few float32 ulp, far below the 1e-6 decision band.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kSeg = 512;
constexpr int kPerLane = kSeg / kWave;
constexpr int kMaxSeg = 4096;  // vocabularies up to 2,097,152 entries

// exp(a - b), with a - b carried exactly as s + err.
__device__ __forceinline__ float exp_diff(float a, float b) {
  const float s = a - b;
  const float bb = s - a;
  const float err = (a - (s - bb)) + (-b - bb);
  const float e = expf(s);
  return fmaf(e, err, e);
}

struct AcceptArgs {
  int gamma, V, nseg;
  const float* x;        // [M][V] logits (lse != nullptr) or probabilities
  const float* lse;      // [M] or nullptr
  const float* q;        // [B][gamma][V]
  const int32_t* draft;  // [B][gamma]
  const float* u;        // [B][G]
  double* segsum;        // [B][nseg]
  int2* desc;            // [B] (accept length l, bits of the log-sum-exp of row l) from prepare
};

__device__ __forceinline__ float r_of(const AcceptArgs& a, const float* xrow, const float* qrow, float lse,
                                      bool residual, int v) {
  const float p = a.lse != nullptr ? exp_diff(xrow[v], lse) : xrow[v];
  if (!residual) return p;
  const float d = p - qrow[v];
  return d > 0.f ? d : 0.f;
}

// One workgroup per request.  The ratio-test operands (draft token, its logit
// or probability, its draft probability, the draw) are gathered first, so
// their latency overlaps the log-sum-exp fold; with `partials` the fold of the
// request's rows (one wave per row) writes row_lse; then wave 0 runs the tests
// in float64 and stores (l, lse of row l) for the next two kernels.
__global__ __launch_bounds__(512)
void accept_prepare_kernel(const AcceptArgs a, int req0, const float2* __restrict__ partials, int ntiles) {
  __shared__ float s_lse[kWave];
  const int req = req0 + blockIdx.x;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int G = a.gamma + 1;

  float xv = 0.f, qv = 0.f, uv = 0.f;
  bool valid = false;
  if (wave == 0 && lane < a.gamma) {
    const int tok = a.draft[(int64_t)req * a.gamma + lane];
    valid = tok >= 0 && tok < a.V;
    if (valid) {
      xv = a.x[((int64_t)req * G + lane) * a.V + tok];
      qv = a.q[((int64_t)req * a.gamma + lane) * a.V + tok];
    }
    uv = a.u[(int64_t)req * G + lane];
  }
  if (partials != nullptr) {
    for (int j = wave; j < G; j += 8) {
      const float v = row_lse_from_partials(partials + ((int64_t)req * G + j) * ntiles, ntiles);
      if (lane == 0) {
        s_lse[j] = v;
        const_cast<float*>(a.lse)[(int64_t)req * G + j] = v;
      }
    }
  } else if (a.lse != nullptr && threadIdx.x < G) {
    s_lse[threadIdx.x] = a.lse[(int64_t)req * G + threadIdx.x];
  }
  __syncthreads();
  if (wave == 0) {
    bool fail = false;
    if (lane < a.gamma) {
      double ratio = 0.0;
      if (valid) {
        const double px = a.lse != nullptr ? exp((double)xv - (double)s_lse[lane]) : (double)xv;
        const double qx = (double)qv;
        ratio = (px <= 0.0) ? 0.0 : (qx <= 0.0 ? (double)INFINITY : px / qx);
      }
      fail = !((double)uv < ratio);
    }
    const unsigned long long fails = __ballot(fail);
    const int l = fails ? (__ffsll(fails) - 1) : a.gamma;
    if (lane == 0) a.desc[req] = make_int2(l, __float_as_int(a.lse != nullptr ? s_lse[l] : 0.f));
  }
}

__global__ __launch_bounds__(kWave)
void accept_segments_kernel(const AcceptArgs a, int req0) {
  const int sg = blockIdx.x;
  const int req = req0 + blockIdx.y;
  const int lane = threadIdx.x;
  const int G = a.gamma + 1;
  const int2 d = a.desc[req];
  const int l = d.x;
  const float lse = __int_as_float(d.y);
  const bool residual = l < a.gamma;
  const int64_t row = (int64_t)req * G + l;
  const float* xrow = a.x + row * a.V;
  const float* qrow = residual ? a.q + ((int64_t)req * a.gamma + l) * a.V : nullptr;
  float r[kPerLane];
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    const int v = sg * kSeg + e * kWave + lane;
    r[e] = v < a.V ? r_of(a, xrow, qrow, lse, residual, v) : 0.f;
  }
  double acc = 0.0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) acc += (double)r[e];
  acc = wave_sum_f64(acc);
  if (lane == 0) a.segsum[(int64_t)req * a.nseg + sg] = acc;
}

// Sum of r over one segment, recomputed (used only on the rare fallback path).
__device__ double segment_sum(const AcceptArgs& a, const float* xrow, const float* qrow, float lse, bool residual,
                              int sg) {
  const int lane = threadIdx.x & 63;
  double acc = 0.0;
  for (int e = 0; e < kPerLane; ++e) {
    const int v = sg * kSeg + e * kWave + lane;
    if (v < a.V) acc += (double)r_of(a, xrow, qrow, lse, residual, v);
  }
  return wave_sum_f64(acc);
}

__global__ __launch_bounds__(kWave)
void accept_finalize_kernel(const AcceptArgs a, const AcceptBatch bt, int32_t* __restrict__ accept_len,
                            int32_t* __restrict__ out_tok, int32_t* __restrict__ new_kv_len) {
  const int b = blockIdx.x;
  const int req = bt.req0 + b;
  const int lane = threadIdx.x;
  const int G = a.gamma + 1;
  __shared__ double seg[kMaxSeg];
  for (int i = lane; i < a.nseg; i += kWave) seg[i] = a.segsum[(int64_t)req * a.nseg + i];
  const int2 d = a.desc[req];
  const int l = d.x;
  const float lse = __int_as_float(d.y);
  bool residual = l < a.gamma;
  const int64_t row = (int64_t)req * G + l;
  const float* xrow = a.x + row * a.V;
  const float* qrow = residual ? a.q + ((int64_t)req * a.gamma + l) * a.V : nullptr;
  lds_wait();

  // Inclusive prefix of the segment totals, in place (LDS, one wave).
  auto prefix = [&]() -> double {
    lds_wait();
    double carry = 0.0;
    for (int base = 0; base < a.nseg; base += kWave) {
      const int i = base + lane;
      const double v = i < a.nseg ? seg[i] : 0.0;
      const double c = wave_inclusive_scan_f64(v) + carry;
      if (i < a.nseg) seg[i] = c;
      carry = __shfl(c, 63);
    }
    lds_wait();
    return carry;
  };
  double z = prefix();
  if (!(z > 0.0) && residual) {
    // The residual vanished (possible only through rounding): sample from p_{l+1}.
    residual = false;
    for (int sg = 0; sg < a.nseg; ++sg) {
      const double s = segment_sum(a, xrow, qrow, lse, false, sg);
      if (lane == 0) seg[sg] = s;
    }
    z = prefix();
  }

  const double thr = (double)a.u[(int64_t)req * G + a.gamma] * z;
  int found = -1;
  for (int base = 0; base < a.nseg && found < 0; base += kWave) {
    const int i = base + lane;
    const unsigned long long hit = __ballot(i < a.nseg && seg[i] > thr);
    if (hit) found = base + __ffsll(hit) - 1;
  }
  int t = -1;
  if (found >= 0) {
    float rv[kPerLane];
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) {
      const int v = found * kSeg + e * kWave + lane;
      rv[e] = v < a.V ? r_of(a, xrow, qrow, lse, residual, v) : 0.f;
    }
    double c = found > 0 ? seg[found - 1] : 0.0;
    int last_pos = -1;
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) {
      const int v = found * kSeg + e * kWave + lane;
      const double r = (double)rv[e];
      const double cum = wave_inclusive_scan_f64(r) + c;
      const unsigned long long hit = __ballot(v < a.V && r > 0.0 && cum > thr);
      if (hit && t < 0) t = found * kSeg + e * kWave + __ffsll(hit) - 1;
      const unsigned long long pos = __ballot(v < a.V && r > 0.0);
      if (pos) last_pos = found * kSeg + e * kWave + 63 - __clzll(pos);
      c = __shfl(cum, 63);
    }
    if (t < 0) t = last_pos;  // rounding put u * Z past this segment's own scan
  }
  if (t < 0) {
    // No prefix sum exceeds u * Z: the largest token with mass.
    for (int sg = a.nseg - 1; sg >= 0 && t < 0; --sg) {
      for (int e = kPerLane - 1; e >= 0 && t < 0; --e) {
        const int v = sg * kSeg + e * kWave + lane;
        const unsigned long long pos = __ballot(v < a.V && r_of(a, xrow, qrow, lse, residual, v) > 0.f);
        if (pos) t = sg * kSeg + e * kWave + 63 - __clzll(pos);
      }
    }
    if (t < 0) t = 0;  // no mass at all (non-finite input)
  }

  if (lane < G) {
    int32_t v = -1;
    if (lane < l) v = a.draft[(int64_t)req * a.gamma + lane];
    else if (lane == l) v = t;
    out_tok[(int64_t)req * G + lane] = v;
  }
  if (lane == 0) {
    accept_len[req] = l;
    if (new_kv_len != nullptr && bt.has_kv_len) new_kv_len[req] = bt.kv_len[b] - a.gamma + l;
  }
}

}  // namespace

size_t accept_workspace_bytes(int B, int V) {
  const int nseg = (V + kSeg - 1) / kSeg;
  return sizeof(double) * static_cast<size_t>(B) * nseg + sizeof(int2) * static_cast<size_t>(B) + 512;
}

hipError_t launch_accept(int gamma, int V, int B, const AcceptBatch& bt, const float* x, const float* row_lse,
                         const float2* partials, int ntiles, const float* q_draft, const int32_t* draft_tok,
                         const float* u, void* ws, int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                         hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (bt.nreq <= 0) return hipSuccess;
  AcceptArgs a;
  a.gamma = gamma;
  a.V = V;
  a.nseg = (V + kSeg - 1) / kSeg;
  a.x = x;
  a.lse = row_lse;
  a.q = q_draft;
  a.draft = draft_tok;
  a.u = u;
  a.segsum = static_cast<double*>(ws);
  a.desc = reinterpret_cast<int2*>(static_cast<char*>(ws) + sizeof(double) * static_cast<size_t>(B) * a.nseg);
  hipLaunchKernelGGL(accept_prepare_kernel, dim3(bt.nreq), dim3(512), 0, stream, a, bt.req0, partials, ntiles);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(accept_segments_kernel, dim3(a.nseg, bt.nreq), dim3(kWave), 0, stream, ev_start, ev_stop,
                        0, a, bt.req0);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_finalize_kernel, dim3(bt.nreq), dim3(kWave), 0, stream, a, bt, accept_len, out_tok,
                     new_kv_len);
  return hipGetLastError();
}

}  // namespace sdv
