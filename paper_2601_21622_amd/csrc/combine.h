// Merge of the split-KV attention partials: for one (request, KV head), the
// chunk partials (running maximum m, sum l, unnormalised o) are merged in
// chunk order, O = sum_c 2^(m_c - M) o_c / sum_c 2^(m_c - M) l_c.  Used by
// the standalone combine kernel and by launches that carry the merge beside
// other work (the verification step folds it into its last launch when the
// projection reads the caller's hidden rows rather than the attention output).
#pragma once

#include "common.h"
#include "launch.h"

namespace sdv {

// Threads per combine block: one per (row, 4 consecutive d) of a pair.
constexpr int kCombineThreads = 256;
// Chunks per pair whose partials a thread loads in one round.
constexpr int kCombineBatch = 8;

inline int combine_zblocks(const AttnShape& s) {
  return (s.rows * (s.D / 4) + kCombineThreads - 1) / kCombineThreads;
}

template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) {
  *p = v;
}
template <>
__device__ __forceinline__ void store_out<uint16_t>(uint16_t* p, float v) {
  *p = __builtin_bit_cast(uint16_t, (__bf16)v);
}

// Block z of pair (request b of the launch, KV head g); thread t of
// kCombineThreads.  Chunk loads are unrolled so that they are in flight together.
template <typename OutT>
__device__ __forceinline__ void combine_block(const AttnShape& s, const AttnBatch& bt, const AttnPartials& parts,
                                              OutT* __restrict__ out, int b, int g, int z, int t) {
  const int req = bt.req0 + b;
  const int c0 = bt.chunk_base + bt.chunk_prefix[b];
  const int c1 = bt.chunk_base + bt.chunk_prefix[b + 1];
  const int D4 = s.D / 4;
  const int i = z * kCombineThreads + t;
  if (i >= s.rows * D4) return;
  const int row = i / D4, d = (i - row * D4) * 4;
  float mx = kNegBig;
  float den = 0.f;
  f32x4 num = {0.f, 0.f, 0.f, 0.f};
  if (c1 - c0 <= kCombineBatch) {
    // Every chunk's (m, l, o) loaded in one round, then the same arithmetic
    // in the same order as below.
    float mv[kCombineBatch], lv[kCombineBatch];
    f32x4 ov[kCombineBatch];
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k) {
      const int64_t slot = (int64_t)min(c0 + k, c1 - 1) * s.Hkv + g;
      mv[k] = parts.m[slot * s.rows + row];
      lv[k] = parts.l[slot * s.rows + row];
      ov[k] = *reinterpret_cast<const f32x4*>(parts.o + (slot * s.rows + row) * s.D + d);
    }
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k)
      if (c0 + k < c1) mx = fmaxf(mx, mv[k]);
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k)
      if (c0 + k < c1) {
        const float a = exp2f(mv[k] - mx);
        den = fmaf(a, lv[k], den);
        num += a * ov[k];
      }
  } else {
#pragma unroll 8
    for (int c = c0; c < c1; ++c) mx = fmaxf(mx, parts.m[((int64_t)c * s.Hkv + g) * s.rows + row]);
#pragma unroll 4
    for (int c = c0; c < c1; ++c) {
      const int64_t slot = (int64_t)c * s.Hkv + g;
      const float a = exp2f(parts.m[slot * s.rows + row] - mx);
      den = fmaf(a, parts.l[slot * s.rows + row], den);
      const f32x4 o = *reinterpret_cast<const f32x4*>(parts.o + (slot * s.rows + row) * s.D + d);
      num += a * o;
    }
  }
  const int j = row / s.group;
  const int h = g * s.group + (row - j * s.group);
  OutT* dst = out + (((int64_t)req * s.G + j) * s.Hq + h) * s.D + d;
#pragma unroll
  for (int e = 0; e < 4; ++e) store_out(dst + e, num[e] / den);
}

// A merge carried by another launch: nblocks blocks over (request, KV head,
// z) of one attention launch's requests; out is bf16 when bf16 != 0.
struct CombineJob {
  AttnShape s;
  AttnBatch bt;
  AttnPartials parts;
  void* out;
  int bf16;
  int nblocks;
};

// Block k (< nblocks) of a carried merge, on threads [0, kCombineThreads).
__device__ __forceinline__ void combine_job_block(const CombineJob& cj, int k, int t) {
  const int zb = (cj.s.rows * (cj.s.D / 4) + kCombineThreads - 1) / kCombineThreads;
  const int z = k % zb;
  const int bg = k / zb;
  const int g = bg % cj.s.Hkv;
  const int b = bg / cj.s.Hkv;
  if (cj.bf16)
    combine_block<uint16_t>(cj.s, cj.bt, cj.parts, static_cast<uint16_t*>(cj.out), b, g, z, t);
  else
    combine_block<float>(cj.s, cj.bt, cj.parts, static_cast<float*>(cj.out), b, g, z, t);
}

}  // namespace sdv
