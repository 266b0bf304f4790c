// Warped target rows for sampled verification (gfx950).
//
// Sampled decoding replaces the target p of the acceptance test (the
// Leviathan test of Sec. 2) by a warped p': logits scaled by 1/T, then the
// top-k cut (every token tied with the k-th largest logit kept), then the
// top-p cut (the smallest set {logit >= theta} of the top-k-kept tokens whose
// mass reaches top_p of their total), or, at T = 0, one-hot on the first
// largest logit (greedy).  For each row this kernel finds the cut and the
// normaliser; the acceptance kernels then evaluate
//   p'(v) = [key(v) >= theta] exp(logit(v) / T - lse)   (greedy: [v == argmax]).
//
// One workgroup of 1024 threads per row:
//   1. the largest logit and the first index holding it (one pass);
//   2. top-k: a radix descent over the 32-bit order keys of the logits, 11, 11
//      and 10 bits per level, with per-bucket counts and masses in LDS; the
//      bucket where the running count from the top reaches k holds the cut;
//   3. top-p: the same descent over the kept tokens, on masses, against
//      ceil(top_p * kept mass) (with no top-k cut, the kept mass is the
//      total of the first level's histogram, which holds every entry);
//   4. lse = max / T + log(kept mass).
// In either descent over a long row the second level also gathers the keys
// inside the first level's bucket into LDS; when they fit, the third level
// reads those instead of the row (the same entries, so the same integer
// sums).
// Masses are exp((logit - max) / T) in float32, scaled by 2^S and truncated to
// 64-bit integers (S = 62 - ceil(log2 V), so a whole row cannot overflow);
// integer sums make every histogram and total independent of the order of
// the atomic adds, so the cut is deterministic.
#include <hip/hip_ext.h>

#include <cmath>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kWarpThreads = 1024;
constexpr int kWarpWaves = kWarpThreads / kWave;
constexpr int kBuckets = 2048;
static_assert(kBuckets == 2 * kWarpThreads, "the level-0 total reads two buckets per thread");
constexpr int kCand = 2048;  // candidates the small-k path can hold
// Keys of the entries inside the first level's bucket that a descent's
// second level gathers into LDS, so that its third level histograms them
// instead of passing over the row again (when they fit).
constexpr int kKeep = 16384;
constexpr int kKeepMinV = 65536;

__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ unsigned long long fixed_mass(float x, float m, float inv_t, double scale) {
  const float w = expf((x - m) * inv_t);
  return (unsigned long long)((double)w * scale);
}

__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int mask) {
  const uint32_t lo = __shfl_xor((uint32_t)v, mask);
  const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), mask);
  return ((unsigned long long)hi << 32) | lo;
}

// Bitonic sort of one 64-bit key per lane across the wave, largest first.
__device__ __forceinline__ unsigned long long wave_sort_desc(unsigned long long v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int size = 2; size <= kWave; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const unsigned long long o = shfl_xor_u64(v, stride);
      const bool desc = (lane & size) == 0 || size == kWave;
      const bool lower = (lane & stride) == 0;
      v = (lower == desc) ? (o > v ? o : v) : (o < v ? o : v);
    }
  }
  return v;
}

// The 64 largest of two lists sorted largest first, sorted largest first: the
// lane-wise maximum of one list and the other reversed is bitonic and holds
// them; a bitonic merge orders it.
__device__ __forceinline__ unsigned long long wave_merge_desc(unsigned long long a, unsigned long long b) {
  const int lane = threadIdx.x & 63;
  const uint32_t lo = __shfl((uint32_t)b, kWave - 1 - lane);
  const uint32_t hi = __shfl((uint32_t)(b >> 32), kWave - 1 - lane);
  const unsigned long long br = ((unsigned long long)hi << 32) | lo;
  unsigned long long v = a > br ? a : br;
#pragma unroll
  for (int stride = kWave >> 1; stride > 0; stride >>= 1) {
    const unsigned long long o = shfl_xor_u64(v, stride);
    v = ((lane & stride) == 0) ? (o > v ? o : v) : (o < v ? o : v);
  }
  return v;
}

__device__ __forceinline__ unsigned long long shfl_u64(unsigned long long v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src);
  const uint32_t hi = __shfl((uint32_t)(v >> 32), src);
  return ((unsigned long long)hi << 32) | lo;
}

// Rank key of an entry: the float32 order key, then the inverted index, so
// that equal logits rank by increasing index and keys are unique (0: none).
__device__ __forceinline__ unsigned long long entry_key(uint32_t k, int v) {
  return ((unsigned long long)k << 32) | (unsigned long long)(0xffffffffu - (uint32_t)v);
}

// Calls f(v, x[v]) for every element of the row, this thread's share, with
// several loads in flight per thread (4 x float4 when the row is 16-byte
// aligned, else 8 scalars).  The order in which a thread sees its elements is
// unspecified; every reduction built on it is order-independent.
template <typename F>
__device__ __forceinline__ void row_pass(const float* __restrict__ x, int V, F&& f) {
  const int tid = threadIdx.x;
  if ((V & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0) {
    constexpr int U = 4;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    const int V4 = V >> 2;
    int i = tid;
    for (; i + (U - 1) * kWarpThreads < V4; i += U * kWarpThreads) {
      float4 r[U];
#pragma unroll
      for (int u = 0; u < U; ++u) r[u] = x4[i + u * kWarpThreads];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = 4 * (i + u * kWarpThreads);
        f(v, r[u].x);
        f(v + 1, r[u].y);
        f(v + 2, r[u].z);
        f(v + 3, r[u].w);
      }
    }
    for (; i < V4; i += kWarpThreads) {
      const float4 r = x4[i];
      f(4 * i, r.x);
      f(4 * i + 1, r.y);
      f(4 * i + 2, r.z);
      f(4 * i + 3, r.w);
    }
  } else {
    constexpr int U = 8;
    int v = tid;
    for (; v + (U - 1) * kWarpThreads < V; v += U * kWarpThreads) {
      float r[U];
#pragma unroll
      for (int u = 0; u < U; ++u) r[u] = x[v + u * kWarpThreads];
#pragma unroll
      for (int u = 0; u < U; ++u) f(v + u * kWarpThreads, r[u]);
    }
    for (; v < V; v += kWarpThreads) f(v, x[v]);
  }
}

struct Level {
  int shift, nb;
  uint32_t hmask;  // bits above this level's digit
};

__device__ __forceinline__ Level level_of(int level) {
  Level l;
  l.shift = level == 0 ? 21 : (level == 1 ? 10 : 0);
  l.nb = level == 2 ? 1024 : 2048;
  l.hmask = level == 0 ? 0u : (0xffffffffu << (l.shift + (level == 2 ? 10 : 11)));
  return l;
}

// Wave 0: scanning the buckets from the top, the first bucket at which the
// running total (of counts, or of masses with BY_MASS) reaches `need`, and the
// count and mass of the buckets above it.  need >= 1 and the buckets hold at
// least `need` in total (otherwise the lowest bucket is returned).  Lane l
// totals the l-th group of nb/64 buckets from the top (reading them in a
// lane-rotated order, so the lanes hit different LDS banks); a wave scan and
// a ballot find the group, and the same inside the group finds the bucket.
template <bool BY_MASS>
__device__ void select_bucket(const uint32_t* hcnt, const unsigned long long* hmass, int nb, unsigned long long need,
                              uint32_t* s_bucket, uint32_t* s_cnt_above, unsigned long long* s_mass_above) {
  const int lane = threadIdx.x & 63;
  const int per = nb / kWave;  // 32 or 16: a power of two
  const int top = nb - 1 - lane * per;
  uint64_t c = 0, ms = 0;
  for (int i = 0; i < per; ++i) {
    const int b = top - ((i + lane) & (per - 1));
    c += hcnt[b];
    ms += hmass[b];
  }
  const uint64_t inc_c = wave_inclusive_scan_u64(c), inc_m = wave_inclusive_scan_u64(ms);
  const unsigned long long hit = __ballot((BY_MASS ? inc_m : inc_c) >= need);
  const int L = hit ? __ffsll(hit) - 1 : kWave - 1;
  const uint64_t c_above = lane_u64(inc_c, L) - lane_u64(c, L);
  const uint64_t m_above = lane_u64(inc_m, L) - lane_u64(ms, L);
  // Inside group L: lane i < per takes bucket nb - 1 - L*per - i.
  // Loads clamped rather than predicated, and every lane read taken before
  // the single-lane store: with the reads inside that branch, the compiled
  // selection returned a wrong mass above the bucket.
  const int b = max(nb - 1 - L * per - lane, 0);
  const uint64_t in_group = 0ull - (uint64_t)(lane < per);
  const uint64_t cb = (uint64_t)hcnt[b] & in_group;
  const uint64_t mb = (uint64_t)hmass[b] & in_group;
  const uint64_t ic = wave_inclusive_scan_u64(cb), im = wave_inclusive_scan_u64(mb);
  const unsigned long long hit2 = __ballot(lane < per - 1 && (BY_MASS ? m_above + im : c_above + ic) >= need);
  const int I = hit2 ? __ffsll(hit2) - 1 : per - 1;
  const uint32_t bucket = (uint32_t)(nb - 1 - L * per - I);
  const uint32_t cnt_above = (uint32_t)(c_above + lane_u64(ic, I) - lane_u64(cb, I));
  const uint64_t mass_above = m_above + lane_u64(im, I) - lane_u64(mb, I);
  if (lane == 0) {
    *s_bucket = bucket;
    *s_cnt_above = cnt_above;
    *s_mass_above = mass_above;
  }
}

__global__ __launch_bounds__(kWarpThreads)
void warp_kernel(int V, const float* __restrict__ logits, float inv_t, int greedy, int top_k, float top_p,
                 double scale, WarpRow* __restrict__ out, float* __restrict__ row_lse,
                 float* __restrict__ row_min_logit) {
  __shared__ uint32_t hcnt[kBuckets];
  __shared__ unsigned long long hmass[kBuckets];
  __shared__ uint32_t w_key[kWarpWaves];
  __shared__ int w_idx[kWarpWaves];
  __shared__ unsigned long long w_sum[kWarpWaves];
  __shared__ uint32_t s_kmax, s_bucket, s_cnt_above;
  __shared__ int s_amax;
  __shared__ unsigned long long s_mass_above, s_total;
  __shared__ unsigned long long s_list[kWarpWaves][kWave];
  __shared__ unsigned long long s_cand[kCand];
  __shared__ uint32_t s_n, s_bound, s_theta, s_pdone;
  __shared__ unsigned long long s_w;


  const int row = blockIdx.x;
  const float* x = logits + (int64_t)row * V;
  float m_row = 0.f;  // the row's largest logit, once known
  __shared__ uint32_t s_keep[kKeep];
  __shared__ uint32_t s_nkeep;

  // One level of a radix descent: histogram (counts and masses) of the
  // entries whose key is at least `floor` and whose bits above the level's
  // digit equal `prefix`.  Level 1 also gathers those entries' keys; level 2
  // reads the gathered keys when all of them fit.
  auto histogram = [&](int level, const Level& lv, uint32_t prefix, uint32_t floor) {
    for (int i = threadIdx.x; i < lv.nb; i += kWarpThreads) {
      hcnt[i] = 0;
      hmass[i] = 0;
    }
    if (threadIdx.x == 0 && level == 1) s_nkeep = 0;
    __syncthreads();
    const float* xr = logits + (int64_t)blockIdx.x * V;
    auto add = [&](uint32_t k, float xv) {  // xv = key_value(k)
      const int b = (k >> lv.shift) & (lv.nb - 1);
      atomicAdd(&hcnt[b], 1u);
      atomicAdd(&hmass[b], fixed_mass(xv, m_row, inv_t, scale));
    };
    // Rows short enough to stay in L2 are read again instead: the gathered
    // level measured slower at 32,000 entries, faster at 128,256.
    const bool use_keep = V >= kKeepMinV;
    const bool gather = use_keep && level == 1;
    if (use_keep && level == 2 && s_nkeep <= (uint32_t)kKeep) {
      const int n = (int)s_nkeep;
      for (int i = threadIdx.x; i < n; i += kWarpThreads) {
        const uint32_t k = s_keep[i];
        if (k >= floor && (k & lv.hmask) == prefix) add(k, key_value(k));
      }
    } else {
      row_pass(xr, V, [&](int, float xv) {
        const uint32_t k = order_key(xv);
        if (k >= floor && (k & lv.hmask) == prefix) {
          add(k, xv);
          if (gather) {
            const uint32_t i = atomicAdd(&s_nkeep, 1u);
            if (i < (uint32_t)kKeep) s_keep[i] = k;
          }
        }
      });
    }
    __syncthreads();
  };
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // 1. Largest key; among equal keys the smallest index.
  auto merge = [](uint32_t& k, int& i, uint32_t ok, int oi) {
    if (ok > k || (ok == k && oi < i)) {
      k = ok;
      i = oi;
    }
  };
  uint32_t bk = 0;
  int bi = 0x7fffffff;
  row_pass(x, V, [&](int v, float xv) { merge(bk, bi, order_key(xv), v); });
  const unsigned long long tkey = bi == 0x7fffffff ? 0ull : entry_key(bk, bi);  // this thread's best entry
  for (int off = 32; off >= 1; off >>= 1) merge(bk, bi, __shfl_xor(bk, off), __shfl_xor(bi, off));
  if (lane == 0) {
    w_key[wave] = bk;
    w_idx[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t k = w_key[0];
    int i = w_idx[0];
    for (int w = 1; w < kWarpWaves; ++w) merge(k, i, w_key[w], w_idx[w]);
    s_kmax = k;
    s_amax = i;
  }
  __syncthreads();
  const int amax = s_amax;
  if (greedy) {
    if (tid == 0) {
      out[row] = WarpRow{0.f, 0xffffffffu, 0.f, amax};
      row_lse[row] = 0.f;
      row_min_logit[row] = INFINITY;
    }
    return;
  }
  const float m = key_value(s_kmax);
  m_row = m;

  // Mass of the whole row (no top-k), or of the top-k set.
  uint32_t theta = 0;
  unsigned long long W = 0;
  bool have_k = false, have_p = false;
  bool w_known = true;  // W holds the kept mass (false: the first top-p level supplies it)
  if (top_k >= 1 && top_k <= kWave && top_k < V) {
    // Small k: the k-th largest of the threads' best entries bounds the k-th
    // largest logit from below (k threads reach it), so the entries at or
    // above it hold the top-k set and all its ties.  They are collected in
    // LDS and wave 0 sorts them in 64-key batches.
    s_list[wave][lane] = wave_sort_desc(tkey);
    __syncthreads();
    if (wave == 0) {
      unsigned long long acc = s_list[0][lane];
      for (int w = 1; w < kWarpWaves; ++w) acc = wave_merge_desc(acc, s_list[w][lane]);
      const unsigned long long kth = shfl_u64(acc, top_k - 1);
      if (lane == 0) {
        s_bound = (uint32_t)(kth >> 32);
        s_n = 0;
      }
    }
    __syncthreads();
    const uint32_t bound = s_bound;
    row_pass(x, V, [&](int v, float xv) {
      const uint32_t k = order_key(xv);
      if (k >= bound) {
        const uint32_t i = atomicAdd(&s_n, 1u);
        if (i < (uint32_t)kCand) s_cand[i] = entry_key(k, v);
      }
    });
    __syncthreads();
    const uint32_t n = s_n;
    if (n <= (uint32_t)kCand) {  // otherwise (masses of ties at the bound) the radix descent below
      if (wave == 0) {
        unsigned long long lst = 0;
        for (uint32_t base = 0; base < n; base += kWave)
          lst = wave_merge_desc(lst, wave_sort_desc(base + lane < n ? s_cand[base + lane] : 0ull));
        const uint32_t thk = (uint32_t)(shfl_u64(lst, top_k - 1) >> 32);
        // The kept set: every candidate whose key reaches the k-th (ties kept).
        uint32_t cnt = 0;
        unsigned long long ms = 0;
        for (uint32_t i = lane; i < n; i += kWave) {
          const uint32_t k = (uint32_t)(s_cand[i] >> 32);
          if (k >= thk) {
            ++cnt;
            ms += fixed_mass(key_value(k), m, inv_t, scale);
          }
        }
        for (int off = 32; off >= 1; off >>= 1) {
          cnt += __shfl_xor(cnt, off);
          ms += shfl_xor_u64(ms, off);
        }
        // Equal on every lane; as scalars, the branch below is uniform.
        cnt = (uint32_t)__builtin_amdgcn_readfirstlane((int)cnt);
        ms = lane_u64(ms, 0);
        uint32_t th = thk;
        unsigned long long w = ms;
        bool pdone = false;
        if (top_p < 1.f && cnt <= (uint32_t)kWave) {
          // Lanes [0, cnt) of the sorted list are the kept set, largest first:
          // the cut is the first key whose running mass reaches the target.
          unsigned long long target = (unsigned long long)ceil((double)top_p * (double)ms);
          target = target < 1 ? 1 : (target > ms ? ms : target);
          const uint32_t lk = (uint32_t)(lst >> 32);
          const unsigned long long cum =
              wave_inclusive_scan_u64(lane < (int)cnt ? fixed_mass(key_value(lk), m, inv_t, scale) : 0ull);
          const int i = __ffsll(__ballot(lane < (int)cnt && cum >= target)) - 1;
          th = __shfl(lk, i);
          const int c = __popcll(__ballot(lane < (int)cnt && lk >= th));
          w = shfl_u64(cum, c - 1);
          pdone = true;
        }
        if (lane == 0) {
          s_theta = th;
          s_w = w;
          s_pdone = pdone;
        }
      }
      __syncthreads();
      theta = s_theta;
      W = s_w;
      have_k = true;
      have_p = s_pdone != 0;
    }
  }
  if (have_k) {
  } else if (top_k >= 1 && top_k < V) {
    uint32_t prefix = 0, krem = (uint32_t)top_k;
    unsigned long long above = 0;
    for (int level = 0; level < 3; ++level) {
      const Level lv = level_of(level);
      histogram(level, lv, prefix, 0u);
      if (wave == 0) select_bucket<false>(hcnt, hmass, lv.nb, krem, &s_bucket, &s_cnt_above, &s_mass_above);
      __syncthreads();
      const uint32_t b = s_bucket;
      krem -= s_cnt_above;
      above += s_mass_above;
      prefix |= b << lv.shift;
      if (level == 2) W = above + hmass[b];
      __syncthreads();
    }
    theta = prefix;
  } else if (top_p < 1.f) {
    // No top-k cut: the first level of the top-p descent histograms every
    // entry, and W is the total of that histogram (no pass of its own).
    w_known = false;
  } else {
    unsigned long long sum = 0;
    row_pass(x, V, [&](int, float xv) { sum += fixed_mass(xv, m, inv_t, scale); });
    for (int off = 32; off >= 1; off >>= 1) sum += shfl_xor_u64(sum, off);
    if (lane == 0) w_sum[wave] = sum;
    __syncthreads();
    if (tid == 0) {
      unsigned long long t = 0;
      for (int w = 0; w < kWarpWaves; ++w) t += w_sum[w];
      s_total = t;
    }
    __syncthreads();
    W = s_total;
  }

  if (top_p < 1.f && !have_p) {
    unsigned long long target = 0;
    auto set_target = [&]() {
      target = (unsigned long long)ceil((double)top_p * (double)W);
      target = target < 1 ? 1 : (target > W ? W : target);
    };
    if (w_known) set_target();
    uint32_t prefix = 0;
    unsigned long long above = 0;
    for (int level = 0; level < 3; ++level) {
      const Level lv = level_of(level);
      histogram(level, lv, prefix, theta);
      if (!w_known) {  // level 0 over every entry: W = the histogram's total
        unsigned long long t = hmass[tid] + hmass[tid + kWarpThreads];
        for (int off = 32; off >= 1; off >>= 1) t += shfl_xor_u64(t, off);
        if (lane == 0) w_sum[wave] = t;
        __syncthreads();
        if (tid == 0) {
          unsigned long long tt = 0;
          for (int w = 0; w < kWarpWaves; ++w) tt += w_sum[w];
          s_total = tt;
        }
        __syncthreads();
        W = s_total;
        w_known = true;
        set_target();
      }
      if (wave == 0)
        select_bucket<true>(hcnt, hmass, lv.nb, target - above, &s_bucket, &s_cnt_above, &s_mass_above);
      __syncthreads();
      const uint32_t b = s_bucket;
      above += s_mass_above;
      prefix |= b << lv.shift;
      if (level == 2) W = above + hmass[b];
      __syncthreads();
    }
    theta = prefix;
  }

  if (tid == 0) {
    const float lse = (float)((double)m * (double)inv_t + log((double)W / scale));
    out[row] = WarpRow{inv_t, theta, lse, -1};
    row_lse[row] = lse;
    row_min_logit[row] = theta == 0 ? -INFINITY : key_value(theta);
  }
}

}  // namespace

hipError_t launch_warp(int M, int V, const float* logits, float temperature, int top_k, float top_p, WarpRow* out,
                       float* row_lse, float* row_min_logit, hipStream_t stream, hipEvent_t ev_start) {
  if (M <= 0) return hipSuccess;
  const int greedy = temperature == 0.f;
  const float inv_t = greedy ? 0.f : 1.f / temperature;  // float32 division, correctly rounded
  int bits = 0;
  while ((int64_t(1) << bits) < V) ++bits;
  const double scale = std::ldexp(1.0, 62 - bits);
  hipExtLaunchKernelGGL(warp_kernel, dim3(M), dim3(kWarpThreads), 0, stream, ev_start, nullptr, 0, V, logits, inv_t,
                        greedy, top_k, top_p, scale, out, row_lse, row_min_logit);
  return hipGetLastError();
}

}  // namespace sdv
