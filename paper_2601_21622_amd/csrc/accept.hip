// Acceptance test, first rejection, residual resampling and output assembly.
//
// Two launches, or one in a step.  The sums kernel runs S workgroups of 8
// waves per request;
// each workgroup
//  1. gathers the ratio-test operands (draft token, its logit or probability,
//     its draft probability, the draw) and, with the vocabulary kernel's
//     per-tile statistics, folds the log-sum-exp of each of the request's rows
//     (one wave per row; the first workgroup writes them out);
//  2. runs the ratio tests in float64 on wave 0 (lane i: u < p_i(x_i) / q_i(x_i))
//     and a ballot gives the accept length l (the first workgroup writes it);
//  3. sums, per 512-entry vocabulary segment of its slice and in float64, the
//     unnormalised continuation distribution: r = max(0, p_{l+1} - q_{l+1})
//     after a rejection, p_{gamma+1} after a full accept; each wave issues the
//     loads of several segments before reducing them.
// Steps 1 and 2 are repeated by every workgroup of a request: they read a few
// kilobytes, far less than the slice.  The pick kernel (one wave per request)
// prefix-sums the segment totals (Z is the last), finds the segment holding
// u * Z, scans it in token order for the first entry whose running sum
// exceeds u * Z, and writes the emitted tokens and the new cache length.
// In a whole verification step both run as one launch (accept_fused_kernel):
// the last workgroup of each request to finish its sums, counted by an
// arrival counter that the step's vocabulary launch clears, runs the pick.
// p(v) = exp(logit - lse) is evaluated in float64 from the float32 inputs.
#include <hip/hip_ext.h>
#include <string.h>

#include "combine.h"
#include "common.h"
#include "launch.h"

namespace sdv {

namespace {


struct AcceptArgs {
  int gamma, V, nseg, segs_per_group;
  const float* x;        // [M][V] logits (lse != nullptr or warp != nullptr) or probabilities
  const float* lse;      // [M] or nullptr
  const WarpRow* warp;   // [M] or nullptr: warped target (sampled verification)
  const float* q;        // [B][gamma][V]
  const int32_t* draft;  // [B][gamma]
  const float* u;        // [B][G]
  double* segsum;        // [B][nseg] segment totals
  const struct TreeFinal* tree;  // tree verification: per request, where the walk ended, or nullptr
};

// Where a request's tree walk ended: the position whose row the final token
// is drawn from, and the candidates rejected there (excluded from that draw).
struct TreeFinal {
  int32_t pos;
  int32_t nrej;
  int32_t pad[2];
  int32_t rej_tok[kWave];
};

// How a row's p is evaluated: from probabilities, from logits and the row
// log-sum-exp, or from logits and the row's warp (sampled verification).
enum { kProbs = 0, kLogits = 1, kWarped = 2 };

struct RowP {
  float lse, inv_t;
  uint32_t theta;
  int argmax;
};

// p(v) in float64 from the row's float32 entry: the difference (or product
// and difference) of float32 operands is exact in float64, so p is within an
// ulp of float64 of exp(logit - lse) -- the value a float64 evaluation of the
// same inputs gives -- and the inverse CDF built from it agrees with one to
// about 1e-13 of Z.  A masked logit (-inf) gives 0.
template <int PM>
__device__ __forceinline__ double p_of(const RowP& rp, float x, int v) {
  if (PM == kProbs) return (double)x;
  if (PM == kLogits) return exp((double)x - (double)rp.lse);
  const double w = order_key(x) >= rp.theta ? exp((double)x * (double)rp.inv_t - (double)rp.lse) : 0.0;
  return v == rp.argmax ? 1.0 : w;
}

__device__ __forceinline__ RowP row_p(const AcceptArgs& a, int64_t row, float lse) {
  RowP rp{lse, 1.f, 0u, -1};
  if (a.warp != nullptr) {
    const WarpRow w = a.warp[row];
    rp.lse = w.lse;
    rp.inv_t = w.inv_t;
    rp.theta = w.theta;
    rp.argmax = w.argmax;
  }
  return rp;
}

constexpr int kSumWaves = 8;            // waves per workgroup of the sums kernel
constexpr int kSeg = 512;               // vocabulary entries per segment
constexpr int kPerLane = kSeg / kWave;  // lane holds entries sg*512 + e*64 + lane
constexpr int kMaxSeg = 4096;           // vocabularies up to 2,097,152 entries
constexpr int kSegBatch = 4;            // segments whose loads a wave issues together
constexpr int kTargetGroups = 512;      // sums-kernel workgroups aimed for per launch
// The fused kernel keeps two workgroups per CU (at most 128 registers), like
// the sums kernel, so its carried merge runs beside the sums; that register
// cap takes a segment batch of 3.
constexpr int kFusedWgsPerCu = 2;
constexpr int kFusedSegBatch = 3;

// r over one segment, per lane (entries sg*512 + e*64 + lane): the raw loads
// (indexes past the vocabulary clamped), then r from them.
template <bool RES>
__device__ __forceinline__ void segment_issue(const float* xrow, const float* qrow, int V, int sg,
                                              float (&xs)[kPerLane], float (&qs)[kPerLane]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    const int v = min(sg * kSeg + e * kWave + lane, V - 1);
    xs[e] = __builtin_nontemporal_load(xrow + v);
    if (RES) qs[e] = __builtin_nontemporal_load(qrow + v);
  }
}

template <int PM, bool RES>
__device__ __forceinline__ void segment_finish(const RowP& rp, int V, int sg, const float (&xs)[kPerLane],
                                               const float (&qs)[kPerLane], double (&r)[kPerLane]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    const int v = sg * kSeg + e * kWave + lane;
    double pv = p_of<PM>(rp, xs[e], v);
    if (RES) {
      const double d = pv - (double)qs[e];
      pv = d > 0.0 ? d : 0.0;
    }
    r[e] = v < V ? pv : 0.0;
  }
}

template <int PM, bool RES>
__device__ __forceinline__ void segment_r(const float* xrow, const float* qrow, const RowP& rp, int V, int sg,
                                          double (&r)[kPerLane]) {
  float xs[kPerLane], qs[kPerLane];
  segment_issue<RES>(xrow, qrow, V, sg, xs, qs);
  segment_finish<PM, RES>(rp, V, sg, xs, qs, r);
}

__device__ __forceinline__ int p_mode(const AcceptArgs& a) {
  return a.warp != nullptr ? kWarped : (a.lse != nullptr ? kLogits : kProbs);
}

__device__ __forceinline__ double p_of_mode(const AcceptArgs& a, const RowP& rp, float x, int v) {
  switch (p_mode(a)) {
    case kWarped: return p_of<kWarped>(rp, x, v);
    case kLogits: return p_of<kLogits>(rp, x, v);
    default: return p_of<kProbs>(rp, x, v);
  }
}

__device__ __forceinline__ void segment_load(const AcceptArgs& a, const float* xrow, const float* qrow, const RowP& rp,
                                             bool residual, int sg, double (&r)[kPerLane]) {
  switch (p_mode(a)) {
    case kWarped:
      if (residual) segment_r<kWarped, true>(xrow, qrow, rp, a.V, sg, r);
      else segment_r<kWarped, false>(xrow, qrow, rp, a.V, sg, r);
      break;
    case kLogits:
      if (residual) segment_r<kLogits, true>(xrow, qrow, rp, a.V, sg, r);
      else segment_r<kLogits, false>(xrow, qrow, rp, a.V, sg, r);
      break;
    default:
      if (residual) segment_r<kProbs, true>(xrow, qrow, rp, a.V, sg, r);
      else segment_r<kProbs, false>(xrow, qrow, rp, a.V, sg, r);
  }
}

// Float64 sum of one segment: per lane in order of e, then across the lanes.
__device__ __forceinline__ double segment_total(const double (&r)[kPerLane]) {
  double acc = 0.0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) acc += r[e];
  return wave_sum_f64(acc);
}

// Totals of segments [sg0, sg1) into out[]: wave w takes sg0 + w, sg0 + w +
// nwaves, ..., issuing the loads of up to SB segments (kSegBatch, or fewer
// where registers are short) before reducing any.  Batch entries past sg1 are skipped (wave-uniform), so a wave with a
// single segment issues and reduces only that one.
// Global totals are stored as device-scope atomic stores (written through to
// the device-coherent level), which the fused launch's last workgroup reads
// with device-scope atomic loads; `out` in LDS takes plain stores.
template <int PM, bool RES, int SB>
__device__ __forceinline__ void segment_totals_t(const float* xrow, const float* qrow, const RowP& rp, int V, int sg0,
                                                 int sg1, int nwaves, double* out, bool global_out) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  for (int s0 = sg0 + wave; s0 < sg1; s0 += nwaves * SB) {
    float xs[SB][kPerLane], qs[SB][kPerLane];
#pragma unroll
    for (int k = 0; k < SB; ++k)
      if (s0 + k * nwaves < sg1) segment_issue<RES>(xrow, qrow, V, s0 + k * nwaves, xs[k], qs[k]);
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int sg = s0 + k * nwaves;
      if (sg >= sg1) break;
      double r[kPerLane];
      segment_finish<PM, RES>(rp, V, sg, xs[k], qs[k], r);
      const double t = segment_total(r);
      if (lane == 0) {
        if (global_out) __hip_atomic_store(out + sg, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else out[sg] = t;
      }
    }
  }
}

template <int SB = kSegBatch>
__device__ __forceinline__ void segment_totals(const AcceptArgs& a, const float* xrow, const float* qrow,
                                               const RowP& rp, bool residual, int sg0, int sg1, int nwaves,
                                               double* out, bool global_out = true) {
  switch (p_mode(a)) {
    case kWarped:
      if (residual) segment_totals_t<kWarped, true, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
      else segment_totals_t<kWarped, false, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
      break;
    case kLogits:
      if (residual) segment_totals_t<kLogits, true, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
      else segment_totals_t<kLogits, false, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
      break;
    default:
      if (residual) segment_totals_t<kProbs, true, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
      else segment_totals_t<kProbs, false, SB>(xrow, qrow, rp, a.V, sg0, sg1, nwaves, out, global_out);
  }
}

// LDS of one request's workgroup in the sums stage.
struct SumsLds {
  float lse[kWave];
  WarpRow warp[kWave];
  int l;
};

// Steps 1-3 for workgroup s of request req (chain or warped mode), SB
// segments' loads in flight per wave: the row
// log-sum-exps and warps land in sl, the accept length in sl.l (and in
// accept_len from workgroup 0), this workgroup's segment totals in a.segsum.
template <int SB>
__device__ __forceinline__ void sums_request(const AcceptArgs& a, const float2* __restrict__ partials, int ntiles,
                                             int32_t* __restrict__ accept_len, int s, int req, SumsLds& sl) {
  float* s_lse = sl.lse;
  WarpRow* s_warp = sl.warp;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int G = a.gamma + 1;

  // 1. Test operands (gathered by the last wave, whose second load waits on
  // the draft tokens), and the row log-sum-exp folds (row j on wave j mod
  // kSumWaves, so the last wave folds none while gamma + 1 < kSumWaves and
  // the other waves' partial loads issue at once).
  constexpr int kTestWave = kSumWaves - 1;
  float xv = 0.f, qv = 0.f, uv = 0.f;
  bool valid = false;
  if (wave == kTestWave && lane < a.gamma) {
    const int tok = a.draft[(int64_t)req * a.gamma + lane];
    valid = tok >= 0 && tok < a.V;
    if (valid) {
      xv = a.x[((int64_t)req * G + lane) * a.V + tok];
      qv = a.q[((int64_t)req * a.gamma + lane) * a.V + tok];
    }
    uv = a.u[(int64_t)req * G + lane];
  }
  if (partials != nullptr) {
    for (int j = wave; j < G; j += kSumWaves) {
      const float v = row_lse_from_partials(partials + ((int64_t)req * G + j) * ntiles, ntiles);
      if (lane == 0) {
        s_lse[j] = v;
        if (s == 0) const_cast<float*>(a.lse)[(int64_t)req * G + j] = v;
      }
    }
  } else if (a.lse != nullptr && threadIdx.x < G) {
    s_lse[threadIdx.x] = a.lse[(int64_t)req * G + threadIdx.x];
  }
  // Warped target: every row's cut, ahead of the accept length that picks one.
  if (a.warp != nullptr && threadIdx.x >= kWave && threadIdx.x < kWave + G)
    s_warp[threadIdx.x - kWave] = a.warp[(int64_t)req * G + threadIdx.x - kWave];
  __syncthreads();

  // 2. Ratio tests in float64; l = number of leading accepts.
  if (wave == kTestWave) {
    bool fail = false;
    if (lane < a.gamma) {
      double ratio = 0.0;
      if (valid) {
        double px;
        if (a.warp != nullptr) {
          // Warped target: the row's cut and normaliser (greedy: one-hot).
          const WarpRow w = s_warp[lane];
          const int tok = a.draft[(int64_t)req * a.gamma + lane];
          px = tok == w.argmax ? 1.0
                               : (order_key(xv) >= w.theta ? exp((double)xv * (double)w.inv_t - (double)w.lse) : 0.0);
        } else {
          px = a.lse != nullptr ? exp((double)xv - (double)s_lse[lane]) : (double)xv;
        }
        const double qx = (double)qv;
        ratio = (px <= 0.0) ? 0.0 : (qx <= 0.0 ? (double)INFINITY : px / qx);
      }
      fail = !((double)uv < ratio);
    }
    const unsigned long long fails = __ballot(fail);
    const int l = fails ? (__ffsll(fails) - 1) : a.gamma;
    if (lane == 0) {
      sl.l = l;
      if (s == 0) accept_len[req] = l;
    }
  }
  __syncthreads();
  const int l = sl.l;
  RowP rp{a.lse != nullptr ? s_lse[l] : 0.f, 1.f, 0u, -1};
  if (a.warp != nullptr) {
    const WarpRow w = s_warp[l];
    rp = RowP{w.lse, w.inv_t, w.theta, w.argmax};
  }
  const bool residual = l < a.gamma;
  const float* xrow = a.x + ((int64_t)req * G + l) * a.V;
  const float* qrow = residual ? a.q + ((int64_t)req * a.gamma + l) * a.V : nullptr;

  // 3. This workgroup's segment totals.
  const int sg0 = s * a.segs_per_group;
  const int sg1 = min(a.nseg, sg0 + a.segs_per_group);
  segment_totals<SB>(a, xrow, qrow, rp, residual, sg0, sg1, kSumWaves, a.segsum + (int64_t)req * a.nseg);
}

// Grid (S, requests); workgroup s covers segments [s * segs_per_group, ...).
__global__ __launch_bounds__(kSumWaves * kWave)
void accept_sums_kernel(const AcceptArgs a, const AcceptBatch bt, const float2* __restrict__ partials, int ntiles,
                        int32_t* __restrict__ accept_len) {
  __shared__ SumsLds sl;
  const int s = blockIdx.x;
  const int req = bt.req0 + blockIdx.y;
  if (a.tree != nullptr) {
    // Tree verification: the walk chose the row; sum its p (the rejected
    // candidates are taken out by the pick kernel).
    const int pos = a.tree[req].pos;
    const int64_t row = (int64_t)req * (a.gamma + 1) + pos;
    const RowP rp = row_p(a, row, a.lse != nullptr ? a.lse[row] : 0.f);
    const int sg0 = s * a.segs_per_group;
    const int sg1 = min(a.nseg, sg0 + a.segs_per_group);
    segment_totals(a, a.x + row * a.V, nullptr, rp, false, sg0, sg1, kSumWaves, a.segsum + (int64_t)req * a.nseg);
    return;
  }
  sums_request<kSegBatch>(a, partials, ntiles, accept_len, s, req, sl);
}

// Segment totals tot[0, nseg) into LDS seg[] by one wave, 8 loads per lane
// in flight (device-scope atomic loads: the totals of other workgroups of
// the same launch).
__device__ __forceinline__ void pick_load_totals(const double* __restrict__ tot, int nseg, double* seg) {
  const int lane = threadIdx.x & 63;
  for (int base = 0; base < nseg; base += 8 * kWave) {
    double v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      v[k] = __hip_atomic_load(tot + min(base + k * kWave + lane, nseg - 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (base + k * kWave + lane < nseg) seg[base + k * kWave + lane] = v[k];
  }
}

// The rest of the draw of request req = bt.req0 + b on one wave, once the
// segment totals are in seg[] (LDS) and the accept length l, the row's p
// (rp, of position pos) and the draw uu are known: the candidates rejected at
// a tree's final position are taken out, the totals are prefix-summed, the
// segment holding u * Z is scanned in token order, and the outputs are
// written.  my_draft: lane i < gamma holds draft token i (chain).  s_rej: a
// kWave-entry LDS array.
__device__ __forceinline__ void pick_finish(const AcceptArgs& a, const AcceptBatch& bt, int b, int l, int pos,
                                            int nrej, int rej, const RowP& rp, float uu, int my_draft,
                                            double* seg, int* s_rej, int32_t* __restrict__ out_tok,
                                            int32_t* __restrict__ new_kv_len) {
  const int req = bt.req0 + b;
  const int lane = threadIdx.x & 63;
  const int G = a.gamma + 1;
  const int nseg = a.nseg;
  const bool tree = a.tree != nullptr;
  const int64_t row = (int64_t)req * G + pos;
  bool residual = !tree && l < a.gamma;
  const float* xrow = a.x + row * a.V;
  const float* qrow = residual ? a.q + ((int64_t)req * a.gamma + l) * a.V : nullptr;
  // The p of each rejected candidate, evaluated as the segment sums did, is
  // taken out of its segment (in candidate order, so deterministically).
  const double rej_p = (tree && rej >= 0) ? p_of_mode(a, rp, xrow[rej], rej) : 0.0;
  s_rej[lane] = rej;
  lds_wait();
  for (int k = 0; k < nrej; ++k) {
    const int tk = __shfl(rej, k);
    const double pk = __shfl(rej_p, k);
    if (lane == 0 && tk >= 0) seg[tk / kSeg] -= pk;
    lds_wait();
  }
  int nexcl = nrej;
  auto excluded = [&](int v) {
    bool e = false;
    for (int k = 0; k < nexcl; ++k) e |= s_rej[k] == v;
    return e;
  };

  // Inclusive prefix of the segment totals, in place.
  auto prefix = [&]() -> double {
    lds_wait();
    double carry = 0.0;
    for (int base = 0; base < nseg; base += kWave) {
      const int i = base + lane;
      const double v = i < nseg ? seg[i] : 0.0;
      const double c = wave_inclusive_scan_f64(v) + carry;
      if (i < nseg) seg[i] = c;
      carry = lane_f64(c, 63);  // a scalar: branches on the total stay uniform
    }
    lds_wait();
    return carry;
  };
  double z = prefix();
  if (!(z > 0.0) && (residual || nexcl > 0)) {
    // The residual vanished (possible only through rounding): sample from p_{l+1}
    // (tree: from the final row's p, no candidate excluded).
    residual = false;
    nexcl = 0;
    segment_totals(a, xrow, qrow, rp, false, 0, nseg, 1, seg, false);
    z = prefix();
  }

  const double thr = (double)uu * z;
  int found = -1;
  for (int base = 0; base < nseg && found < 0; base += kWave) {
    const int i = base + lane;
    const unsigned long long hit = __ballot(i < nseg && seg[i] > thr);
    if (hit) found = base + __ffsll(hit) - 1;
  }
  int t = -1;
  if (found >= 0) {
    double rv[kPerLane];
    segment_load(a, xrow, qrow, rp, residual, found, rv);
    double c = found > 0 ? seg[found - 1] : 0.0;
    int last_pos = -1;
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) {
      const int v = found * kSeg + e * kWave + lane;
      const double r = excluded(v) ? 0.0 : rv[e];
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
    for (int sg = nseg - 1; sg >= 0 && t < 0; --sg) {
      double rv[kPerLane];
      segment_load(a, xrow, qrow, rp, residual, sg, rv);
      for (int e = kPerLane - 1; e >= 0 && t < 0; --e) {
        const unsigned long long pos = __ballot(rv[e] > 0.0 && !excluded(sg * kSeg + e * kWave + lane));
        if (pos) t = sg * kSeg + e * kWave + 63 - __clzll(pos);
      }
    }
    if (t < 0) t = 0;  // no mass at all (non-finite input)
  }

  if (tree) {
    // The walk wrote the accepted nodes' tokens and the cache length.
    if (lane < G && lane >= l) out_tok[(int64_t)req * G + lane] = lane == l ? t : -1;
    return;
  }
  if (lane < G) {
    int32_t v = -1;
    if (lane < l) v = my_draft;
    else if (lane == l) v = t;
    out_tok[(int64_t)req * G + lane] = v;
  }
  if (lane == 0 && new_kv_len != nullptr && bt.has_kv_len) new_kv_len[req] = bt.kv_len[b] - a.gamma + l;
}

// One wave per request: prefix of the segment totals, the segment holding
// u * Z, and the scan of that segment in token order.  Blocks past the
// requests carry an attention merge (cj.nblocks blocks), which then runs in
// the idle CUs of this latency-bound launch; a request's block uses its
// first wave only.
__global__ __launch_bounds__(kCombineThreads)
void accept_pick_kernel(const AcceptArgs a, const AcceptBatch bt, const int32_t* __restrict__ accept_len,
                        int32_t* __restrict__ out_tok, int32_t* __restrict__ new_kv_len, const CombineJob cj) {
  __shared__ double seg[kMaxSeg];
  if ((int)blockIdx.x >= bt.nreq) {
    combine_job_block(cj, blockIdx.x - bt.nreq, threadIdx.x);
    return;
  }
  if (threadIdx.x >= kWave) return;
  const int b = blockIdx.x;
  const int req = bt.req0 + b;
  const int lane = threadIdx.x;
  const int G = a.gamma + 1;
  const int nseg = a.nseg;
  const double* tot = a.segsum + (int64_t)req * nseg;

  // Segment totals into LDS, 8 loads per lane in flight; l and u alongside,
  // and everything else that does not depend on them: the drafts to emit and
  // each row's normaliser (lane j: row j), so that only the segment loads
  // wait for the draw's position.
  const int l = accept_len[req];
  const float uu = a.u[(int64_t)req * G + a.gamma];
  const bool tree = a.tree != nullptr;
  const int my_draft = (!tree && lane < a.gamma) ? a.draft[(int64_t)req * a.gamma + lane] : -1;
  float my_lse = 0.f;
  WarpRow my_warp{1.f, 0u, 0.f, -1};
  if (lane < G) {
    if (a.warp != nullptr) my_warp = a.warp[(int64_t)req * G + lane];
    else if (a.lse != nullptr) my_lse = a.lse[(int64_t)req * G + lane];
  }
  pick_load_totals(tot, nseg, seg);
  // Chain: row l, residual after a rejection.  Tree: the walk's final row,
  // plain p without the candidates rejected there.
  const int pos = tree ? a.tree[req].pos : l;
  const int nrej = tree ? a.tree[req].nrej : 0;
  const int rej = tree && lane < nrej ? a.tree[req].rej_tok[lane] : -1;
  RowP rp{__shfl(my_lse, pos), 1.f, 0u, -1};
  if (a.warp != nullptr) {
    rp.lse = __shfl(my_warp.lse, pos);
    rp.inv_t = __shfl(my_warp.inv_t, pos);
    rp.theta = (uint32_t)__shfl((int)my_warp.theta, pos);
    rp.argmax = __shfl(my_warp.argmax, pos);
  }
  __shared__ int s_rej[kWave];
  pick_finish(a, bt, b, l, pos, nrej, rej, rp, uu, my_draft, seg, s_rej, out_tok, new_kv_len);
}

// Chain, warped and tree modes in one launch (the verification steps): the
// sums stage of accept_sums_kernel, after which the last workgroup of each
// request to finish its segment totals (counted by a per-request arrival
// counter, which the vocabulary launch that precedes this one in the step
// clears) draws the request's token on its first wave, as accept_pick_kernel
// does.
// Workgroups past the requests carry an attention merge, two merge blocks
// each.
__global__ __launch_bounds__(kSumWaves * kWave, kFusedWgsPerCu * kSumWaves / 4)  // waves per SIMD
void accept_fused_kernel(const AcceptArgs a, const AcceptBatch bt, const float2* __restrict__ partials, int ntiles,
                         int32_t* __restrict__ accept_len, int32_t* __restrict__ out_tok,
                         int32_t* __restrict__ new_kv_len, int* __restrict__ arrivals, const CombineJob cj) {
  __shared__ SumsLds sl;
  __shared__ double seg[kMaxSeg];
  __shared__ int s_rej[kWave];
  __shared__ int s_last;
  static_assert(kSumWaves * kWave == 2 * kCombineThreads, "two merge blocks per workgroup");
  if ((int)blockIdx.y >= bt.nreq) {
    const int k = (((int)blockIdx.y - bt.nreq) * (int)gridDim.x + (int)blockIdx.x) * 2 +
                  ((int)threadIdx.x >= kCombineThreads ? 1 : 0);
    if (k < cj.nblocks) combine_job_block(cj, k, threadIdx.x & (kCombineThreads - 1));
    return;
  }
  const int b = blockIdx.y;
  const int req = bt.req0 + b;
  const int G = a.gamma + 1;
  RowP rp_tree{0.f, 1.f, 0u, -1};
  int pos_tree = 0;
  if (a.tree != nullptr) {
    // Tree verification: the walk (previous launch) chose the row; sum its p.
    pos_tree = a.tree[req].pos;
    const int64_t row = (int64_t)req * G + pos_tree;
    rp_tree = row_p(a, row, a.lse != nullptr ? a.lse[row] : 0.f);
    const int sg0 = blockIdx.x * a.segs_per_group;
    const int sg1 = min(a.nseg, sg0 + a.segs_per_group);
    segment_totals<kFusedSegBatch>(a, a.x + row * a.V, nullptr, rp_tree, false, sg0, sg1, kSumWaves,
                                   a.segsum + (int64_t)req * a.nseg);
  } else {
    sums_request<kFusedSegBatch>(a, partials, ntiles, accept_len, blockIdx.x, req, sl);
  }
  // Count this workgroup in once its totals are published; the last of the
  // request's gridDim.x workgroups goes on.  The totals are device-scope
  // atomic stores; every wave waits until its stores have completed, and
  // the barrier orders those waits before the arrival.  The last workgroup
  // issues its device-scope atomic loads of the totals only after its own
  // arrival returned, i.e. after every other arrival and so after every
  // store it waits on had completed: no cache write-back or invalidation is
  // needed on either side.
  wait_vmcnt<0>();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(arrivals + req, 1) == (int)gridDim.x - 1 ? 1 : 0;
  __syncthreads();
  if (s_last == 0 || threadIdx.x >= kWave) return;
  const int lane = threadIdx.x;
  const float uu = a.u[(int64_t)req * G + a.gamma];
  if (a.tree != nullptr) {
    // The walk wrote the accept length and the candidates rejected at pos.
    const int l = accept_len[req];
    const int nrej = a.tree[req].nrej;
    const int rej = lane < nrej ? a.tree[req].rej_tok[lane] : -1;
    pick_load_totals(a.segsum + (int64_t)req * a.nseg, a.nseg, seg);
    pick_finish(a, bt, b, l, pos_tree, nrej, rej, rp_tree, uu, -1, seg, s_rej, out_tok, new_kv_len);
    return;
  }
  const int l = sl.l;
  const int my_draft = lane < a.gamma ? a.draft[(int64_t)req * a.gamma + lane] : -1;
  pick_load_totals(a.segsum + (int64_t)req * a.nseg, a.nseg, seg);
  RowP rp{a.lse != nullptr ? sl.lse[l] : 0.f, 1.f, 0u, -1};
  if (a.warp != nullptr) {
    const WarpRow w = sl.warp[l];
    rp = RowP{w.lse, w.inv_t, w.theta, w.argmax};
  }
  pick_finish(a, bt, b, l, l, 0, -1, rp, uu, my_draft, seg, s_rej, out_tok, new_kv_len);
}

// Tree verification, one wave per request (N = gamma nodes, N + 1 <= 64
// positions; lane i stands for node i).  Candidates are point-mass proposals
// of the ratio test: at the current position its children (nodes whose parent
// sits there) are tested in node order, child c passing iff
//   u[c] < p(token_c) / (1 - mass of the candidates already rejected here),
// a token already rejected among its siblings having mass 0; the first child
// that passes is accepted and the walk moves to it.  The walk ends at a
// position none of whose children passes (or that has none); the final token
// is drawn there from p without the rejected candidates by the sums and pick
// kernels.  All test operands are gathered at once (lane i: node i's token
// under its parent's row); the walk itself runs on registers and ballots.
// With `partials` (a whole tree step), the block's kSumWaves waves first fold
// the request's row log-sum-exps from the vocabulary kernel's per-tile
// statistics and write them to a.lse; wave 0 then walks.
__global__ __launch_bounds__(kSumWaves * kWave)
void tree_walk_kernel(const AcceptArgs a, const AcceptBatch bt, const int32_t* __restrict__ tokens,
                      const int32_t* __restrict__ parent, TreeFinal* __restrict__ fin,
                      int32_t* __restrict__ accept_len, int32_t* __restrict__ out_tok,
                      int32_t* __restrict__ out_node, int32_t* __restrict__ new_kv_len,
                      const float2* __restrict__ partials, int ntiles) {
  __shared__ float s_lse[kWave];
  const int b = blockIdx.x;
  const int req = bt.req0 + b;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int N = a.gamma;
  const int G = N + 1;

  // Wave 0 gathers the test operands while the waves fold the row
  // log-sum-exps (row j on wave j mod kSumWaves).
  int tok = -1, par = -1;
  float xv = 0.f;
  float uc = 1.f;
  if (wave == 0 && lane < N) {
    tok = tokens[(int64_t)req * N + lane];
    const int pp = parent[(int64_t)req * N + lane];
    par = (pp >= -1 && pp < lane) ? pp : -1;
    uc = a.u[(int64_t)req * G + lane];
    if (tok >= 0 && tok < a.V) xv = a.x[((int64_t)req * G + par + 1) * a.V + tok];
    else tok = -1;
  }
  if (partials != nullptr) {
    for (int j = wave; j < G; j += kSumWaves) {
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
  if (wave != 0) return;
  double pc = 0.0;
  if (tok >= 0) pc = a.lse != nullptr ? exp((double)xv - (double)s_lse[par + 1]) : (double)xv;

  int pos = 0, l = 0, nrej = 0, rej_tok = -1;
  int path = -1;  // lane j: the j-th accepted node
  while (true) {
    unsigned long long kids = __ballot(lane < N && par + 1 == pos);
    double rejected_mass = 0.0;
    nrej = 0;
    rej_tok = -1;
    int accepted = -1;
    while (kids) {
      const int c = __ffsll(kids) - 1;
      kids &= kids - 1;
      const int t = __shfl(tok, c);
      const double pt = __shfl(pc, c);
      const float ut = __shfl(uc, c);
      const bool dup = t < 0 || __ballot(lane < nrej && rej_tok == t) != 0;
      const double rest = 1.0 - rejected_mass;
      const double thr = (dup || !(rest > 0.0)) ? 0.0 : pt / rest;
      if ((double)ut < thr) {
        accepted = c;
        break;
      }
      if (!dup) {
        rejected_mass += pt;
        if (lane == nrej) rej_tok = t;
        ++nrej;
      }
    }
    if (accepted < 0) break;
    if (lane == l) path = accepted;
    ++l;
    pos = accepted + 1;
  }

  if (lane < G) {
    out_node[(int64_t)req * G + lane] = lane < l ? path : -1;
    if (lane < l) out_tok[(int64_t)req * G + lane] = tokens[(int64_t)req * N + path];
  }
  if (lane == 0) {
    accept_len[req] = l;
    fin[req].pos = pos;
    fin[req].nrej = nrej;
    if (new_kv_len != nullptr && bt.has_kv_len) new_kv_len[req] = bt.kv_len[b] - N + l;
  }
  fin[req].rej_tok[lane] = lane < nrej ? rej_tok : -1;
}

}  // namespace

// Workspace: segment totals [B][nseg] (float64), then one arrival counter
// per request (the fused launch).
static size_t segsum_bytes(int B, int V) {
  const int nseg = (V + kSeg - 1) / kSeg;
  return (sizeof(double) * static_cast<size_t>(B) * nseg + 255) / 256 * 256;
}

size_t accept_workspace_bytes(int B, int V) { return segsum_bytes(B, V) + sizeof(int) * static_cast<size_t>(B); }

int* accept_arrivals(void* ws, int B, int V) {
  return reinterpret_cast<int*>(static_cast<char*>(ws) + segsum_bytes(B, V));
}

hipError_t launch_accept(int gamma, int V, int B, const AcceptBatch& bt, const float* x, const float* row_lse,
                         const float2* partials, int ntiles, const float* q_draft, const int32_t* draft_tok,
                         const float* u, void* ws, int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                         hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop, const WarpRow* warp,
                         const CombineJob* combine, bool fused) {
  if (bt.nreq <= 0) return hipSuccess;
  AcceptArgs a;
  a.gamma = gamma;
  a.V = V;
  a.nseg = (V + kSeg - 1) / kSeg;
  if (a.nseg > kMaxSeg || gamma + 1 > kWave) return hipErrorInvalidValue;
  // Segments per workgroup: a multiple of the wave count, enough workgroups
  // to cover the chip about twice.
  const int64_t want = ((int64_t)a.nseg * bt.nreq + kTargetGroups - 1) / kTargetGroups;
  a.segs_per_group = (int)std::min<int64_t>(a.nseg, std::max<int64_t>(kSumWaves, (want + kSumWaves - 1) / kSumWaves * kSumWaves));
  a.x = x;
  a.lse = warp != nullptr ? nullptr : row_lse;
  a.warp = warp;
  a.tree = nullptr;
  a.q = q_draft;
  a.draft = draft_tok;
  a.u = u;
  a.segsum = static_cast<double*>(ws);
  const int S = (a.nseg + a.segs_per_group - 1) / a.segs_per_group;
  CombineJob cj;
  memset(&cj, 0, sizeof(cj));
  if (combine != nullptr) cj = *combine;
  if (fused) {
    // One launch; the arrival counters were cleared by an earlier launch.
    const int extra = cj.nblocks > 0 ? ((cj.nblocks + 1) / 2 + S - 1) / S : 0;
    hipExtLaunchKernelGGL(accept_fused_kernel, dim3(S, bt.nreq + extra), dim3(kSumWaves * kWave), 0, stream, ev_start,
                          ev_stop, 0, a, bt, warp != nullptr ? nullptr : partials, ntiles, accept_len, out_tok,
                          new_kv_len, accept_arrivals(ws, B, V), cj);
    return hipGetLastError();
  }
  hipExtLaunchKernelGGL(accept_sums_kernel, dim3(S, bt.nreq), dim3(kSumWaves * kWave), 0, stream, ev_start, nullptr,
                        0, a, bt, warp != nullptr ? nullptr : partials, ntiles, accept_len);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(accept_pick_kernel, dim3(bt.nreq + cj.nblocks), dim3(kCombineThreads), 0, stream, nullptr,
                        ev_stop, 0, a, bt, accept_len, out_tok, new_kv_len, cj);
  return hipGetLastError();
}

size_t accept_tree_workspace_bytes(int B, int V) {
  return (accept_workspace_bytes(B, V) + 255) / 256 * 256 + sizeof(TreeFinal) * static_cast<size_t>(B);
}

hipError_t launch_accept_tree(int N, int V, int B, const AcceptBatch& bt, const float* x, const float* row_lse,
                              const int32_t* tokens, const int32_t* parent, const float* u, void* ws,
                              int32_t* accept_len, int32_t* out_tok, int32_t* out_node, int32_t* new_kv_len,
                              hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop, const CombineJob* combine,
                              const float2* partials, int ntiles, bool fused) {
  if (bt.nreq <= 0) return hipSuccess;
  AcceptArgs a;
  a.gamma = N;
  a.V = V;
  a.nseg = (V + kSeg - 1) / kSeg;
  if (a.nseg > kMaxSeg || N + 1 > kWave) return hipErrorInvalidValue;
  const int64_t want = ((int64_t)a.nseg * bt.nreq + kTargetGroups - 1) / kTargetGroups;
  a.segs_per_group = (int)std::min<int64_t>(a.nseg, std::max<int64_t>(kSumWaves, (want + kSumWaves - 1) / kSumWaves * kSumWaves));
  a.x = x;
  a.lse = row_lse;
  a.warp = nullptr;
  a.q = nullptr;
  a.draft = nullptr;
  a.u = u;
  // Workspace: segment totals [B][nseg] and the arrival counters, then one
  // TreeFinal per request (all requests, indexed by the global request number).
  const size_t seg_bytes = (accept_workspace_bytes(B, V) + 255) / 256 * 256;
  a.segsum = static_cast<double*>(ws);
  TreeFinal* fin = reinterpret_cast<TreeFinal*>(static_cast<char*>(ws) + seg_bytes);
  a.tree = fin;
  hipExtLaunchKernelGGL(tree_walk_kernel, dim3(bt.nreq), dim3(kSumWaves * kWave), 0, stream, ev_start, nullptr, 0, a,
                        bt, tokens, parent, fin, accept_len, out_tok, out_node, new_kv_len, partials, ntiles);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int S = (a.nseg + a.segs_per_group - 1) / a.segs_per_group;
  CombineJob cj;
  memset(&cj, 0, sizeof(cj));
  if (combine != nullptr) cj = *combine;
  if (fused) {
    const int extra = cj.nblocks > 0 ? ((cj.nblocks + 1) / 2 + S - 1) / S : 0;
    hipExtLaunchKernelGGL(accept_fused_kernel, dim3(S, bt.nreq + extra), dim3(kSumWaves * kWave), 0, stream, nullptr,
                          ev_stop, 0, a, bt, (const float2*)nullptr, 0, accept_len, out_tok, new_kv_len,
                          accept_arrivals(ws, B, V), cj);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(accept_sums_kernel, dim3(S, bt.nreq), dim3(kSumWaves * kWave), 0, stream, a, bt,
                     (const float2*)nullptr, 0, accept_len);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(accept_pick_kernel, dim3(bt.nreq + cj.nblocks), dim3(kCombineThreads), 0, stream, nullptr, ev_stop, 0, a,
                        bt, accept_len, out_tok, new_kv_len, cj);
  return hipGetLastError();
}

}  // namespace sdv
