// Causal multi-query verification attention (split-KV) for gfx950.
//
// Each request b brings G = gamma + 1 queries (root + drafts) per query head;
// query j sees keys 0 .. L_b - G + j of the request's own KV segment.  With
// grouped-query attention the G * group queries that share a KV head form the
// "rows" of one KV head, and every key/value vector is read from HBM once for
// all of them.
//
// Work split: one workgroup per (request chunk of `chunk_keys` keys, KV head).
// Its four waves stream interleaved 32-key tiles straight from HBM:
//   S^T = K Q^T on MFMA 16x16x32 bf16 (K rows are the A operand, loaded in
//       place from the [L][D] layout; the Q fragments stay in registers),
//   online softmax in the log2 domain, each lane owning one query row,
//   O^T += V^T P^T on MFMA, with P used straight from the S^T accumulator
//       layout and V transposed through a wave-private LDS tile.
// The four waves then merge their (max, sum, O) through LDS and one partial
// per workgroup goes to the workspace; a combine kernel merges the chunks of
// each request in fixed order and writes O in the input dtype.
#include <hip/hip_ext.h>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = 4;
constexpr int kTile = 32;


__device__ __forceinline__ int find_request(const AttnBatch& bt, int c) {
  int lo = 0, hi = bt.nreq - 1;  // largest b with chunk_prefix[b] <= c
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (bt.chunk_prefix[mid] <= c) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <int D>
struct VStage {
  static constexpr int kStride = D + 4;  // uint16 per staged row: 4 row groups hit distinct LDS banks
  static constexpr int kWaveElems = kTile * kStride;
};

template <int RB, int D>
struct AttnSmem {
  static constexpr int kRowsPad = 16 * RB;
  static constexpr int kOStride = D + 4;
  static constexpr size_t kStage = sizeof(uint16_t) * kAttnWaves * VStage<D>::kWaveElems;
  static constexpr size_t kMerge = sizeof(float) * (2 * kRowsPad + kRowsPad * kOStride);
  static constexpr size_t kBytes = kStage > kMerge ? kStage : kMerge;
};

template <int RB, int D>
__global__ __launch_bounds__(kAttnThreads, (RB >= 3 ? 1 : 2))
void attn_bf16_kernel(const AttnShape s, const AttnBatch bt, const uint16_t* __restrict__ q,
                      const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
                      AttnPartials parts) {
  constexpr int DS = D / 32;  // 32-wide steps of the q.k contraction
  constexpr int DB = D / 16;  // 16-wide blocks of the output
  constexpr int VS = VStage<D>::kStride;
  using SM = AttnSmem<RB, D>;
  __shared__ __align__(16) unsigned char smem[SM::kBytes];

  const int c_local = blockIdx.x;
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;  // row (or column) within a 16-block
  const int lg = lane >> 4;  // lane group: k-slice of MFMA operands

  const int b = find_request(bt, c_local);
  const int L = bt.kv_len[b];
  const int64_t off = bt.kv_off[b];
  const int req = bt.req0 + b;
  const int k_begin = (c_local - bt.chunk_prefix[b]) * s.chunk_keys;
  const int k_end = min(L, k_begin + s.chunk_keys);
  const uint16_t* Kb = kp + off + (int64_t)g * L * D;
  const uint16_t* Vb = vp + off + (int64_t)g * L * D;

  // Q fragments (B operand of S^T = K Q^T): lane holds row rb*16+lr, d = ds*32 + lg*8 .. +8.
  bf16x8 qf[RB][DS];
  int lim[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = rb * 16 + lr;
    if (row < s.rows) {
      const int j = row / s.group;
      const int h = g * s.group + (row - j * s.group);
      const uint16_t* qrow = q + (((int64_t)req * s.G + j) * s.Hq + h) * D;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = load_bf16x8(qrow + ds * 32 + lg * 8);
      lim[rb] = L - s.G + j;
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = bf16x8{};
      lim[rb] = -1;
    }
  }

  float m[RB], lsum[RB];
  f32x4 o[RB][DB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = kNegBig;
    lsum[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  uint16_t* vst = reinterpret_cast<uint16_t*>(smem) + wave * VStage<D>::kWaveElems;
  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  constexpr int LPR = D / 8;      // lanes per staged V row (16 bytes each)
  constexpr int KPI = 64 / LPR;   // V rows per wave-wide load

  constexpr int NV = kTile / KPI;
  for (int t = wave; t < ntiles; t += kAttnWaves) {
    const int k0 = k_begin + t * kTile;
    // K fragments (A operand): lane holds key k0 + kb*16 + lr; keys past L are clamped and masked.
    bf16x8 kf[2][DS];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int key = min(k0 + kb * 16 + lr, L - 1);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = load_bf16x8(Kb + (int64_t)key * D + ds * 32 + lg * 8);
    }
    // V rows of the tile, coalesced 16-byte loads, staged row-major in LDS below.
    u32x4 vreg[NV];
#pragma unroll
    for (int it = 0; it < NV; ++it) {
      const int key = min(k0 + it * KPI + lane / LPR, L - 1);
      vreg[it] = *reinterpret_cast<const u32x4*>(Vb + (int64_t)key * D + (lane % LPR) * 8);
    }

    f32x4 st[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) acc = mfma16x16x32(kf[kb][ds], qf[rb][ds], acc);
        st[rb][kb] = acc;
      }

#pragma unroll
    for (int it = 0; it < NV; ++it) {
      uint16_t* dst = vst + (it * KPI + lane / LPR) * VS + (lane % LPR) * 8;
      reinterpret_cast<u32x2*>(dst)[0] = u32x2{vreg[it][0], vreg[it][1]};
      reinterpret_cast<u32x2*>(dst)[1] = u32x2{vreg[it][2], vreg[it][3]};
    }

    // Online softmax: lane owns row rb*16+lr and keys k0 + kb*16 + lg*4 + i.
    bf16x8 pf[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float sv[8];
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = k0 + kb * 16 + lg * 4 + i;
          float x = st[rb][kb][i] * s.scale_log2;
          x = key > lim[rb] ? -INFINITY : x;
          sv[kb * 4 + i] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m[rb], mx);
      const float alpha = exp2f(m[rb] - mn);
      m[rb] = mn;
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const __bf16 pb = (__bf16)exp2f(sv[e] - mn);
        pf[rb][e] = pb;
        ps += (float)pb;
      }
      lsum[rb] = lsum[rb] * alpha + ps;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
    }

    lds_wait();
    // V^T fragments (A operand of O^T += V^T P^T): lane holds d = db*16 + lr and the
    // 8 keys {lg*4 .. lg*4+3, 16+lg*4 .. 16+lg*4+3} matching the P fragment's k-slots.
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      bf16x8 vf;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int kl = (e < 4) ? (lg * 4 + e) : (16 + lg * 4 + e - 4);
        vf[e] = __builtin_bit_cast(__bf16, vst[kl * VS + db * 16 + lr]);
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) o[rb][db] = mfma16x16x32(vf, pf[rb], o[rb][db]);
    }
    lds_wait();
  }

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    lsum[rb] += __shfl_xor(lsum[rb], 16);
    lsum[rb] += __shfl_xor(lsum[rb], 32);
  }

  // Merge the four waves through LDS, one after the other (fixed order).
  float* mm = reinterpret_cast<float*>(smem);
  float* ml = mm + SM::kRowsPad;
  float* mo = ml + SM::kRowsPad;
  __syncthreads();
  for (int turn = 0; turn < kAttnWaves; ++turn) {
    if (wave == turn) {
      if (turn > 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int row = rb * 16 + lr;
          const float m2 = mm[row], l2 = ml[row];
          const float mn = fmaxf(m[rb], m2);
          const float a1 = exp2f(m[rb] - mn), a2 = exp2f(m2 - mn);
          m[rb] = mn;
          lsum[rb] = lsum[rb] * a1 + l2 * a2;
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const f32x4 o2 = *reinterpret_cast<const f32x4*>(mo + row * SM::kOStride + db * 16 + lg * 4);
            o[rb][db] = o[rb][db] * a1 + o2 * a2;
          }
        }
      }
      if (turn < kAttnWaves - 1) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int row = rb * 16 + lr;
          if (lg == 0) {
            mm[row] = m[rb];
            ml[row] = lsum[rb];
          }
#pragma unroll
          for (int db = 0; db < DB; ++db)
            *reinterpret_cast<f32x4*>(mo + row * SM::kOStride + db * 16 + lg * 4) = o[rb][db];
        }
      }
    }
    __syncthreads();
  }

  if (wave == kAttnWaves - 1) {
    const int64_t slot = (int64_t)(bt.chunk_base + c_local) * s.Hkv + g;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = rb * 16 + lr;
      if (row < s.rows) {
        if (lg == 0) {
          parts.m[slot * s.rows + row] = m[rb];
          parts.l[slot * s.rows + row] = lsum[rb];
        }
#pragma unroll
        for (int db = 0; db < DB; ++db)
          *reinterpret_cast<f32x4*>(parts.o + (slot * s.rows + row) * D + db * 16 + lg * 4) = o[rb][db];
      }
    }
  }
}

// float32 path (small shapes): one workgroup per (chunk, KV head); scores and
// probabilities staged in LDS, plain FMA arithmetic.
__global__ __launch_bounds__(kAttnThreads)
void attn_f32_kernel(const AttnShape s, const AttnBatch bt, const float* __restrict__ q,
                     const float* __restrict__ kp, const float* __restrict__ vp,
                     AttnPartials parts) {
  extern __shared__ float fsm[];
  const int D = s.D;
  const int C = s.chunk_keys;
  float* qs = fsm;                 // [rows][D]
  float* ps = fsm + s.rows * D;    // [rows][C]
  const int c_local = blockIdx.x;
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int b = find_request(bt, c_local);
  const int L = bt.kv_len[b];
  const int req = bt.req0 + b;
  const int k_begin = (c_local - bt.chunk_prefix[b]) * C;
  const int nk = min(L, k_begin + C) - k_begin;
  const float* Kb = kp + bt.kv_off[b] + (int64_t)g * L * D;
  const float* Vb = vp + bt.kv_off[b] + (int64_t)g * L * D;
  const int64_t slot = (int64_t)(bt.chunk_base + c_local) * s.Hkv + g;

  for (int i = threadIdx.x; i < s.rows * D; i += kAttnThreads) {
    const int row = i / D, d = i - row * D;
    const int j = row / s.group;
    const int h = g * s.group + (row - j * s.group);
    qs[i] = q[(((int64_t)req * s.G + j) * s.Hq + h) * D + d];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < s.rows * nk; i += kAttnThreads) {
    const int row = i / nk, kk = i - row * nk;
    const int key = k_begin + kk;
    const float* kr = Kb + (int64_t)key * D;
    const float* qr = qs + row * D;
    float acc = 0.f;
    for (int d = 0; d < D; ++d) acc = fmaf(qr[d], kr[d], acc);
    const int lim = L - s.G + row / s.group;
    ps[row * C + kk] = key > lim ? -INFINITY : acc * s.scale_log2;
  }
  __syncthreads();
  for (int row = wave; row < s.rows; row += kAttnWaves) {
    float mx = kNegBig;
    for (int kk = lane; kk < nk; kk += kWave) mx = fmaxf(mx, ps[row * C + kk]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int kk = lane; kk < nk; kk += kWave) {
      const float p = exp2f(ps[row * C + kk] - mx);
      ps[row * C + kk] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      parts.m[slot * s.rows + row] = mx;
      parts.l[slot * s.rows + row] = sum;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < s.rows * D; i += kAttnThreads) {
    const int row = i / D, d = i - row * D;
    float acc = 0.f;
    for (int kk = 0; kk < nk; ++kk) acc = fmaf(ps[row * C + kk], Vb[(int64_t)(k_begin + kk) * D + d], acc);
    parts.o[(slot * s.rows + row) * D + d] = acc;
  }
}

template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<uint16_t>(uint16_t* p, float v) {
  *p = __builtin_bit_cast(uint16_t, (__bf16)v);
}

// Merge the chunk partials of one (request, KV head) in chunk order.  One
// thread per (row, 4 consecutive d); chunk loads are unrolled so they are in
// flight together.
template <typename OutT>
__global__ __launch_bounds__(kAttnThreads)
void attn_combine_kernel(const AttnShape s, const AttnBatch bt, AttnPartials parts, OutT* __restrict__ out) {
  const int b = blockIdx.x;
  const int g = blockIdx.y;
  const int req = bt.req0 + b;
  const int c0 = bt.chunk_base + bt.chunk_prefix[b];
  const int c1 = bt.chunk_base + bt.chunk_prefix[b + 1];
  const int D4 = s.D / 4;
  const int i = blockIdx.z * kAttnThreads + threadIdx.x;
  if (i >= s.rows * D4) return;
  const int row = i / D4, d = (i - row * D4) * 4;
  float mx = kNegBig;
#pragma unroll 8
  for (int c = c0; c < c1; ++c) mx = fmaxf(mx, parts.m[((int64_t)c * s.Hkv + g) * s.rows + row]);
  float den = 0.f;
  f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int c = c0; c < c1; ++c) {
    const int64_t slot = (int64_t)c * s.Hkv + g;
    const float a = exp2f(parts.m[slot * s.rows + row] - mx);
    den = fmaf(a, parts.l[slot * s.rows + row], den);
    const f32x4 o = *reinterpret_cast<const f32x4*>(parts.o + (slot * s.rows + row) * s.D + d);
    num += a * o;
  }
  const int j = row / s.group;
  const int h = g * s.group + (row - j * s.group);
  OutT* dst = out + (((int64_t)req * s.G + j) * s.Hq + h) * s.D + d;
#pragma unroll
  for (int e = 0; e < 4; ++e) store_out(dst + e, num[e] / den);
}

template <int RB, int D>
hipError_t launch_bf16(const AttnShape& s, const AttnBatch& bt, int nchunks, const void* q, const void* k,
                       const void* v, AttnPartials parts, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  hipExtLaunchKernelGGL((attn_bf16_kernel<RB, D>), dim3(nchunks, s.Hkv), dim3(kAttnThreads), 0, stream, e0, e1, 0,
                        s, bt, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                        static_cast<const uint16_t*>(v), parts);
  return hipGetLastError();
}

template <int D>
hipError_t dispatch_rb(int rb, const AttnShape& s, const AttnBatch& bt, int nchunks, const void* q, const void* k,
                       const void* v, AttnPartials parts, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  switch (rb) {
    case 1: return launch_bf16<1, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 2: return launch_bf16<2, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 3: return launch_bf16<3, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 4: return launch_bf16<4, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 5: return launch_bf16<5, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 6: return launch_bf16<6, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 7: return launch_bf16<7, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 8: return launch_bf16<8, D>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int attn_chunk_keys(int dtype, int rows, int head_dim) {
  (void)head_dim;
  if (dtype == 0) return 128;
  // Larger row groups write larger partials; longer chunks amortise them.
  if (rows <= 16) return 512;
  if (rows <= 32) return 1024;
  return 2048;
}

size_t attn_partial_bytes(int64_t total_chunks, int Hkv, int rows, int D) {
  const size_t slots = static_cast<size_t>(total_chunks) * Hkv;
  return slots * rows * sizeof(float) * (2 + static_cast<size_t>(D)) + 256;
}

AttnPartials attn_carve(void* ws, int64_t total_chunks, int Hkv, int rows, int D) {
  const size_t slots = static_cast<size_t>(total_chunks) * Hkv;
  float* base = static_cast<float*>(ws);
  AttnPartials p;
  p.o = base;                                  // 16-byte aligned rows: D % 4 == 0
  p.m = base + slots * rows * D;
  p.l = p.m + slots * rows;
  return p;
}

hipError_t launch_attention(int dtype, const AttnShape& s, const AttnBatch& bt, int nchunks,
                            const void* q, const void* k, const void* v, AttnPartials parts,
                            hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if (nchunks <= 0) return hipSuccess;
  if (dtype == 0) {
    const size_t shm = sizeof(float) * static_cast<size_t>(s.rows) * (s.D + s.chunk_keys);
    hipExtLaunchKernelGGL(attn_f32_kernel, dim3(nchunks, s.Hkv), dim3(kAttnThreads), shm, stream, e0, e1, 0, s, bt,
                          static_cast<const float*>(q), static_cast<const float*>(k),
                          static_cast<const float*>(v), parts);
    return hipGetLastError();
  }
  const int rb = (s.rows + 15) / 16;
  if (s.D == 128) return dispatch_rb<128>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
  if (s.D == 64) return dispatch_rb<64>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
  return hipErrorInvalidValue;
}

hipError_t launch_attention_combine(int dtype, const AttnShape& s, const AttnBatch& bt,
                                    AttnPartials parts, void* out, hipStream_t stream) {
  if (bt.nreq <= 0) return hipSuccess;
  const dim3 grid(bt.nreq, s.Hkv, (s.rows * (s.D / 4) + kAttnThreads - 1) / kAttnThreads);
  if (dtype == 0)
    hipLaunchKernelGGL(attn_combine_kernel<float>, grid, dim3(kAttnThreads), 0, stream, s, bt, parts,
                       static_cast<float*>(out));
  else
    hipLaunchKernelGGL(attn_combine_kernel<uint16_t>, grid, dim3(kAttnThreads), 0, stream, s, bt, parts,
                       static_cast<uint16_t*>(out));
  return hipGetLastError();
}

}  // namespace sdv
