// Vocabulary projection with a fused softmax-statistics epilogue (gfx950).
//
// logits^T = W hidden^T on MFMA 16x16x32 bf16: a W fragment (16 vocabulary
// rows x 32 k, loaded in place from the [V][K] layout) is the A operand and a
// hidden fragment (16 rows x 32 k) the B operand.  Each lane then holds four
// consecutive vocabulary entries of one hidden row, which is what the logits
// store and the row statistics want.
//
// One workgroup owns a tile of 64 vocabulary rows for all M hidden rows of its
// M-tile, so W (the dominant stream, K*V*2 bytes) is read from HBM once; the
// hidden rows, shared by every workgroup, are staged per K-chunk in LDS in
// MFMA-fragment order (double-buffered) and stay L2-resident.  The epilogue
// writes the float32 logits and, per (row, tile), the tile maximum and the sum
// of exp(logit - maximum); a second kernel combines the tiles of each row in
// fixed order into the row's log-sum-exp.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kVThreads = 256;
constexpr int kTileN = 64;  // vocabulary rows per workgroup (4 waves x 16)

template <int MB, int KC>
struct VocabCfg {
  static constexpr int kSteps = KC / 32;                  // MFMA k-steps per chunk
  static constexpr int kFragBytes = 1024;                 // one 16x32 bf16 fragment
  static constexpr int kBufBytes = MB * kSteps * kFragBytes;
  static constexpr int kPieces = 16 * MB * KC / 8;        // 16-byte pieces per A chunk
  static constexpr int kPiecesPerThread = (kPieces + kVThreads - 1) / kVThreads;
};

template <int MB, int KC, bool PACKED>
__global__ __launch_bounds__(kVThreads)
void vocab_bf16_kernel(int M, int K, int V, int ntiles, const uint16_t* __restrict__ hidden,
                       const uint16_t* __restrict__ w, float* __restrict__ logits,
                       float2* __restrict__ partials) {
  using C = VocabCfg<MB, KC>;
  __shared__ __align__(16) unsigned char abuf[2][C::kBufBytes];
  __shared__ float red[4][16 * MB];

  const int tile = blockIdx.x;
  const int m0 = blockIdx.y * 16 * MB;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;
  // W fragment stream of this wave: 16 vocabulary rows (clamped; masked in the
  // epilogue).  Row-major: the lane's row from column lg*8.  Packed: fragment
  // (k-step s, block) at ((s * nblk + block) * 64 + lane) * 8.
  const int nblk = (V + 15) / 16;
  const uint16_t* wrow;
  int64_t wstep;  // elements between consecutive k-steps
  if (PACKED) {
    wrow = w + ((int64_t)min(nblk - 1, tile * 4 + wave) * 64 + lane) * 8;
    wstep = (int64_t)nblk * 64 * 8;
  } else {
    wrow = w + (int64_t)min(V - 1, tile * kTileN + wave * 16 + lr) * K + lg * 8;
    wstep = 32;
  }
  const int nchunks = K / KC;

  // Cooperative A-chunk load: piece p -> (row, 16-byte k piece), coalesced along k.
  u32x4 areg[C::kPiecesPerThread];
  auto load_a = [&](int kc) {
#pragma unroll
    for (int i = 0; i < C::kPiecesPerThread; ++i) {
      const int p = threadIdx.x + i * kVThreads;
      const int row = p / (KC / 8);
      const int kp = p - row * (KC / 8);
      u32x4 v = {0u, 0u, 0u, 0u};
      if (p < C::kPieces && m0 + row < M)
        v = *reinterpret_cast<const u32x4*>(hidden + (int64_t)(m0 + row) * K + kc * KC + kp * 8);
      areg[i] = v;
    }
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < C::kPiecesPerThread; ++i) {
      const int p = threadIdx.x + i * kVThreads;
      if (p < C::kPieces) {
        const int row = p / (KC / 8);
        const int kp = p - row * (KC / 8);
        const int mb = row >> 4, r = row & 15, ks = kp >> 2, g = kp & 3;
        const int slot = (mb * C::kSteps + ks) * 64 + r + 16 * g;
        *reinterpret_cast<u32x4*>(abuf[buf] + slot * 16) = areg[i];
      }
    }
  };

  bf16x8 wcur[C::kSteps], wnext[C::kSteps];
  auto load_w = [&](bf16x8* dst, int kc) {
#pragma unroll
    for (int ks = 0; ks < C::kSteps; ++ks) dst[ks] = load_bf16x8(wrow + (int64_t)(kc * C::kSteps + ks) * wstep);
  };

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_a(0);
  load_w(wcur, 0);
  store_a(0);
  lds_barrier();
  for (int kc = 0; kc < nchunks; ++kc) {
    const int buf = kc & 1;
    const bool more = kc + 1 < nchunks;
    if (more) {
      load_a(kc + 1);
      load_w(wnext, kc + 1);
    }
#pragma unroll
    for (int ks = 0; ks < C::kSteps; ++ks) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(abuf[buf] + ((mb * C::kSteps + ks) * 64 + lane) * 16));
        acc[mb] = mfma16x16x32(wcur[ks], a, acc[mb]);
      }
    }
    if (more) {
      store_a(buf ^ 1);
#pragma unroll
      for (int ks = 0; ks < C::kSteps; ++ks) wcur[ks] = wnext[ks];
    }
    lds_barrier();
  }

  // Epilogue.  Lane holds hidden row m0 + mb*16 + lr, vocabulary v0 .. v0+3.
  const int v0 = tile * kTileN + wave * 16 + lg * 4;
  const bool vec_ok = (V % 4 == 0) && (v0 + 3 < V);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 16 + lr;
    if (m < M) {
      float* dst = logits + (int64_t)m * V + v0;
      if (vec_ok) {
        *reinterpret_cast<f32x4*>(dst) = acc[mb];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (v0 + i < V) dst[i] = acc[mb][i];
      }
    }
  }
  float tmax[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    float x = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) x = (v0 + i < V) ? fmaxf(x, acc[mb][i]) : x;
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    if (lg == 0) red[wave][mb * 16 + lr] = x;
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int r = mb * 16 + lr;
    tmax[mb] = fmaxf(fmaxf(red[0][r], red[1][r]), fmaxf(red[2][r], red[3][r]));
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) s += (v0 + i < V) ? expf(acc[mb][i] - tmax[mb]) : 0.f;
    s += __shfl_xor(s, 16);
    s += __shfl_xor(s, 32);
    if (lg == 0) red[wave][mb * 16 + lr] = s;
  }
  __syncthreads();
  if (wave == 0 && lg == 0) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = mb * 16 + lr;
      const int m = m0 + r;
      if (m < M) {
        const float s = (red[0][r] + red[1][r]) + (red[2][r] + red[3][r]);
        partials[(int64_t)m * ntiles + tile] = make_float2(tmax[mb], s);
      }
    }
  }
}

// float32 path: 64 rows x 64 vocabulary entries per workgroup, LDS-tiled FMA.
constexpr int kF32KC = 32;
__global__ __launch_bounds__(kVThreads)
void vocab_f32_kernel(int M, int K, int V, int ntiles, const float* __restrict__ hidden,
                      const float* __restrict__ w, float* __restrict__ logits,
                      float2* __restrict__ partials) {
  __shared__ float wt[kF32KC][kTileN + 1];  // [k][vocab]
  __shared__ float ht[64][kF32KC + 1];      // [row][k]
  const int tile = blockIdx.x;
  const int m0 = blockIdx.y * 64;
  const int col = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int v = tile * kTileN + col;
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  for (int k0 = 0; k0 < K; k0 += kF32KC) {
    for (int i = threadIdx.x; i < kTileN * kF32KC; i += kVThreads) {
      const int r = i / kF32KC, k = i - r * kF32KC;
      const int vv = min(V - 1, tile * kTileN + r);
      wt[k][r] = (k0 + k < K) ? w[(int64_t)vv * K + k0 + k] : 0.f;
    }
    for (int i = threadIdx.x; i < 64 * kF32KC; i += kVThreads) {
      const int r = i / kF32KC, k = i - r * kF32KC;
      ht[r][k] = (m0 + r < M && k0 + k < K) ? hidden[(int64_t)(m0 + r) * K + k0 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int k = 0; k < kF32KC; ++k) {
      const float wv = wt[k][col];
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = fmaf(ht[wave + 4 * i][k], wv, acc[i]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int m = m0 + wave + 4 * i;
    if (m >= M) continue;  // uniform across the wave
    if (v < V) logits[(int64_t)m * V + v] = acc[i];
    const float x = v < V ? acc[i] : -INFINITY;
    const float mx = wave_max(x);
    const float s = wave_sum(v < V ? expf(x - mx) : 0.f);
    if (col == 0) partials[(int64_t)m * ntiles + tile] = make_float2(mx, s);
  }
}

// One wave per row: maximum over tiles, then a float64 sum of the rescaled tile sums.
__global__ __launch_bounds__(kVThreads)
void lse_combine_kernel(int M, int ntiles, const float2* __restrict__ partials, float* __restrict__ row_lse) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const float v = row_lse_from_partials(partials + (int64_t)row * ntiles, ntiles);
  if (lane == 0) row_lse[row] = v;
}

// Repack W [V][K] into fragment order [K/32][ceil(V/16)][64][8]: one thread
// per 16-byte piece, writes coalesced; rows past V are zero.
__global__ __launch_bounds__(kVThreads)
void pack_vocab_kernel(int K, int V, const uint16_t* __restrict__ w, uint16_t* __restrict__ out) {
  const int nblk = (V + 15) / 16;
  const int64_t pieces = (int64_t)(K / 32) * nblk * 64;
  for (int64_t i = (int64_t)blockIdx.x * kVThreads + threadIdx.x; i < pieces; i += (int64_t)gridDim.x * kVThreads) {
    const int lane = (int)(i & 63);
    const int64_t f = i >> 6;
    const int blk = (int)(f % nblk);
    const int s = (int)(f / nblk);
    const int row = blk * 16 + (lane & 15);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < V) v = *reinterpret_cast<const u32x4*>(w + (int64_t)row * K + s * 32 + (lane >> 4) * 8);
    *reinterpret_cast<u32x4*>(out + i * 8) = v;
  }
}

template <int MB, int KC>
hipError_t launch_mb_kc(const VocabPlan& p, int mtiles, const void* hidden, const void* w, float* logits,
                        float2* partials, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, true>), dim3(p.ntiles, mtiles), dim3(kVThreads), 0, stream, e0,
                          e1, 0, p.M, p.K, p.V, p.ntiles, static_cast<const uint16_t*>(hidden),
                          static_cast<const uint16_t*>(w), logits, partials);
  else
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, false>), dim3(p.ntiles, mtiles), dim3(kVThreads), 0, stream, e0,
                          e1, 0, p.M, p.K, p.V, p.ntiles, static_cast<const uint16_t*>(hidden),
                          static_cast<const uint16_t*>(w), logits, partials);
  return hipGetLastError();
}

// K-chunk: as long as the double-buffered hidden chunk fits comfortably in LDS;
// 32 (one MFMA step) whenever K is not a multiple of the preferred chunk.
template <int MB>
hipError_t launch_mb(const VocabPlan& p, int mtiles, const void* hidden, const void* w, float* logits,
                     float2* partials, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  constexpr int KC = MB <= 4 ? 256 : (MB <= 8 ? 128 : (MB <= 16 ? 64 : 32));
  if (p.K % KC == 0) return launch_mb_kc<MB, KC>(p, mtiles, hidden, w, logits, partials, stream, e0, e1);
  if (p.K % 32 == 0) return launch_mb_kc<MB, 32>(p, mtiles, hidden, w, logits, partials, stream, e0, e1);
  return hipErrorInvalidValue;
}

}  // namespace

size_t vocab_packed_bytes(int K, int V) {
  return sizeof(uint16_t) * static_cast<size_t>(K) * ((static_cast<size_t>(V) + 15) / 16) * 16;
}

hipError_t launch_pack_vocab(int K, int V, const void* w, void* out, hipStream_t stream) {
  const int64_t pieces = (int64_t)(K / 32) * ((V + 15) / 16) * 64;
  const int64_t blocks = std::min<int64_t>((pieces + kVThreads - 1) / kVThreads, 65536);
  hipLaunchKernelGGL(pack_vocab_kernel, dim3((unsigned)blocks), dim3(kVThreads), 0, stream, K, V,
                     static_cast<const uint16_t*>(w), static_cast<uint16_t*>(out));
  return hipGetLastError();
}

VocabPlan vocab_plan(int dtype, int M, int K, int V, bool packed) {
  (void)dtype;
  VocabPlan p;
  p.packed = packed;
  p.M = M;
  p.K = K;
  p.V = V;
  p.tile_n = kTileN;
  p.ntiles = (V + kTileN - 1) / kTileN;
  return p;
}

size_t vocab_partial_bytes(const VocabPlan& p) {
  return sizeof(float2) * static_cast<size_t>(p.M) * p.ntiles + 256;
}

hipError_t launch_vocab(int dtype, const VocabPlan& p, const void* hidden, const void* w, float* logits,
                        float2* partials, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if (dtype == 0) {
    const int mtiles = (p.M + 63) / 64;
    hipExtLaunchKernelGGL(vocab_f32_kernel, dim3(p.ntiles, mtiles), dim3(kVThreads), 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, static_cast<const float*>(hidden), static_cast<const float*>(w), logits,
                          partials);
    return hipGetLastError();
  }
  const int blocks = (p.M + 15) / 16;
  // Rows per M-tile: up to 20 blocks of 16 (320 rows) so that W is streamed
  // once for every pooled batch up to that size.
  const int mtiles = (blocks + 19) / 20;
  const int mb = (blocks + mtiles - 1) / mtiles;
  switch (mb) {
#define SDV_MB(n) case n: return launch_mb<n>(p, mtiles, hidden, w, logits, partials, stream, e0, e1);
    SDV_MB(1) SDV_MB(2) SDV_MB(3) SDV_MB(4) SDV_MB(5) SDV_MB(6) SDV_MB(7) SDV_MB(8) SDV_MB(9) SDV_MB(10)
    SDV_MB(11) SDV_MB(12) SDV_MB(13) SDV_MB(14) SDV_MB(15) SDV_MB(16) SDV_MB(17) SDV_MB(18) SDV_MB(19)
    SDV_MB(20)
#undef SDV_MB
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_lse_combine(const VocabPlan& p, const float2* partials, float* row_lse, hipStream_t stream) {
  hipLaunchKernelGGL(lse_combine_kernel, dim3((p.M + 3) / 4), dim3(kVThreads), 0, stream, p.M, p.ntiles,
                     partials, row_lse);
  return hipGetLastError();
}

}  // namespace sdv
