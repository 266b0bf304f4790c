// Device helpers shared by the verification kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sdv {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kWave = 64;
// Finite stand-in for -infinity in running maxima: masked scores are -inf,
// so exp2(-inf - m) is exactly 0 for any finite running maximum m.
constexpr float kNegBig = -1.0e30f;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// 16-byte global load reinterpreted as 8 bf16 (the MFMA operand of one lane).
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// Streaming (read-once) 16-byte load: the nontemporal hint keeps single-use
// data such as weights and KV caches from displacing reused lines in L2 and
// the Infinity Cache, and sustains a markedly higher HBM read rate.
__device__ __forceinline__ bf16x8 load_bf16x8_stream(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}
__device__ __forceinline__ u32x4 load_u32x4_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// LDS DMA: lane l copies 16 bytes from its global address g into LDS at
// lds + 16*l (lds is wave-uniform).  Counted by vmcnt like any global load;
// the reader must wait for it (vmcnt, then a barrier across waves) itself.
__device__ __forceinline__ void dma_16B_to_lds(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Transposing LDS read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane j supplies the address of 4 consecutive 16-bit elements x_j[0..3];
// lane i receives {x_{i/4}[i%4], x_{4+i/4}[i%4], x_{8+i/4}[i%4], x_{12+i/4}[i%4]}.
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4;
__device__ __forceinline__ s16x4 lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D[32x32] += A[32x16] B[16x32].  Lane l holds A[l%32][8*(l/32) .. +8] and
// B[8*(l/32) .. +8][l%32]; result register r of lane l is
// D[8*(r/4) + 4*(l/32) + r%4][l%32].
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Cross-lane moves inside rows of 16 lanes (DPP; GFX9 control codes) and
// reads of single lanes.  The wave reductions and the scan below are built
// from them rather than from LDS-routed shuffles (ds_bpermute), which cost an
// LDS round trip per step on the latency-bound paths.  The order of
// operations is fixed, and every lane of a reduction ends with the same bits
// (pairs are combined commutatively inside a row, and the four row results
// are read into scalars and combined once).
constexpr int kDppXor1 = 0xB1;           // quad_perm [1,0,3,2]: lane i <- i ^ 1
constexpr int kDppXor2 = 0x4E;           // quad_perm [2,3,0,1]: lane i <- i ^ 2
constexpr int kDppRowHalfMirror = 0x141;  // lane i <- 7 - i within each 8 lanes
constexpr int kDppRowMirror = 0x140;      // lane i <- 15 - i within each row
constexpr int kDppRowShr = 0x110;         // + n: lane i <- i - n inside the row, 0 before its start
constexpr int kDppWaveShr1 = 0x138;       // lane i <- i - 1 across the wave, lane 0 <- 0

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, dpp_u32<CTRL>(__builtin_bit_cast(uint32_t, v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint64_t lo = dpp_u32<CTRL>((uint32_t)b), hi = dpp_u32<CTRL>((uint32_t)(b >> 32));
  return __builtin_bit_cast(double, (hi << 32) | lo);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const uint64_t lo = dpp_u32<CTRL>((uint32_t)v), hi = dpp_u32<CTRL>((uint32_t)(v >> 32));
  return (hi << 32) | lo;
}
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int l) {
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return (hi << 32) | lo;
}
__device__ __forceinline__ float lane_f32(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __builtin_bit_cast(double, (hi << 32) | lo);
}

// Reductions over the 64 lanes of a wave; every lane must be active.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppRowHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppRowMirror>(v));
  return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppRowHalfMirror>(v);
  v += dpp_f32<kDppRowMirror>(v);
  return (lane_f32(v, 0) + lane_f32(v, 16)) + (lane_f32(v, 32) + lane_f32(v, 48));
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppRowHalfMirror>(v);
  v += dpp_f64<kDppRowMirror>(v);
  return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}

// Inclusive prefix sum across the 64 lanes, fixed order: Hillis-Steele inside
// each row of 16, then the totals of the rows before are added.
__device__ __forceinline__ double wave_inclusive_scan_f64(double v) {
  v += dpp_f64<kDppRowShr + 1>(v);
  v += dpp_f64<kDppRowShr + 2>(v);
  v += dpp_f64<kDppRowShr + 4>(v);
  v += dpp_f64<kDppRowShr + 8>(v);
  const double t0 = lane_f64(v, 15), t1 = lane_f64(v, 31), t2 = lane_f64(v, 47);
  // Rows before this lane's, without branches (as in the integer scan): the
  // 0/1 factors are exact, so row r adds ((t0 + t1) + t2) truncated to its
  // first r terms, and row 0 adds +0.
  const int row = (threadIdx.x & 63) >> 4;
  const double before = (t0 * (double)(row > 0) + t1 * (double)(row > 1)) + t2 * (double)(row > 2);
  return v + before;
}

// Inclusive prefix sum of 64-bit integers across the 64 lanes (exact, so the
// order does not matter): inside each row of 16, then the rows before.
__device__ __forceinline__ uint64_t wave_inclusive_scan_u64(uint64_t v) {
  v += dpp_u64<kDppRowShr + 1>(v);
  v += dpp_u64<kDppRowShr + 2>(v);
  v += dpp_u64<kDppRowShr + 4>(v);
  v += dpp_u64<kDppRowShr + 8>(v);
  const uint64_t t0 = lane_u64(v, 15), t1 = lane_u64(v, 31), t2 = lane_u64(v, 47);
  // Rows before this lane's, without branches: compiled as divergent
  // branches, this tail followed by further DPP scans gave wrong sums.
  const int row = (threadIdx.x & 63) >> 4;
  const uint64_t m1 = 0ull - (uint64_t)(row > 0), m2 = 0ull - (uint64_t)(row > 1), m3 = 0ull - (uint64_t)(row > 2);
  return v + ((t0 & m1) + (t1 & m2) + (t2 & m3));
}

__device__ __forceinline__ void lds_wait() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// exp(a - b), with a - b carried exactly as s + err (TwoSum), so that the
// result is within a few float32 ulp of the exact exp(a - b).  A masked
// entry (a = -inf, finite b) gives exactly 0: there s = -inf and err is NaN
// ((-inf) - (-inf)), so the correction is skipped whenever exp(s) is 0.
__device__ __forceinline__ float exp_diff(float a, float b) {
  const float s = a - b;
  const float bb = s - a;
  const float err = (a - (s - bb)) + (-b - bb);
  const float e = expf(s);
  return e == 0.f ? 0.f : fmaf(e, err, e);
}

// 32-bit key whose unsigned order is the order of the float32 values (-0
// below +0): negative values bit-inverted, the others with the sign bit set.
__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Workgroup barrier that orders LDS traffic only.  __syncthreads() also waits
// for every outstanding global load (vmcnt(0) on gfx9-family parts), which
// would drain the prefetch pipeline of the streaming kernels.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Row log-sum-exp from per-tile (maximum, sum of exp(x - maximum)) pairs, one
// wave: the row maximum m, then sum_t S_t * exp(M_t - m) accumulated in
// float64, lse = m + log(sum).  Each lane holds tiles lane, lane + 64, ...;
// loads take clamped indexes and masks so a round of kR per lane is in flight
// at once (rows of up to kR * 64 tiles are read once), the lane sums are added
// by the fixed-order wave reduction, so the result is deterministic and
// every lane returns the same bits.  ntiles >= 1.
template <int kR>  // tiles per lane held in registers per round
__device__ __forceinline__ float row_lse_from_partials_r(const float2* p, int ntiles) {
  const int lane = threadIdx.x & 63;
  float2 v[kR];
  auto load = [&](int base) {
#pragma unroll
    for (int j = 0; j < kR; ++j) v[j] = p[min(base + j * kWave + lane, ntiles - 1)];
#pragma unroll
    for (int j = 0; j < kR; ++j)
      if (base + j * kWave + lane >= ntiles) v[j] = make_float2(-INFINITY, 0.f);
  };
  float mx = -INFINITY;
  for (int base = 0; base < ntiles; base += kR * kWave) {
    load(base);
#pragma unroll
    for (int j = 0; j < kR; ++j) mx = fmaxf(mx, v[j].x);
  }
  mx = wave_max(mx);
  const bool one_round = ntiles <= kR * kWave;
  double s = 0.0;
  for (int base = 0; base < ntiles; base += kR * kWave) {
    if (!one_round) load(base);
#pragma unroll
    for (int j = 0; j < kR; ++j) s += (double)v[j].y * (double)expf(v[j].x - mx);
  }
  s = wave_sum_f64(s);
  return (float)((double)mx + log(s));  // mx and s are the same on every lane
}

// Rows of at most 512 tiles (vocabularies up to 131072 at 256-wide tiles)
// take one round of 8 loads per lane; longer rows rounds of 16.
__device__ __forceinline__ float row_lse_from_partials(const float2* p, int ntiles) {
  return ntiles <= 8 * kWave ? row_lse_from_partials_r<8>(p, ntiles) : row_lse_from_partials_r<16>(p, ntiles);
}

}  // namespace sdv
