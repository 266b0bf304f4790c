// Vocabulary projection with a fused softmax-statistics epilogue (gfx950).
//
// logits^T = W hidden^T on MFMA 16x16x32 bf16: a W fragment (16 vocabulary
// rows x 32 k) is the A operand and a hidden fragment (16 rows x 32 k) the B
// operand.  Each lane then holds four consecutive vocabulary entries of one
// hidden row, which is what the logits store and the row statistics want.
//
// A workgroup (4 waves) owns a tile of vocabulary rows for all hidden rows of
// its M-tile, so W (the dominant stream, K*V*2 bytes) is read from HBM once.
// Every wave streams its own W fragments straight into registers; the hidden
// rows, shared by every workgroup and L2-resident, are staged per K-chunk in
// LDS in MFMA-fragment order and read by all four waves.  Two schedules:
//   * shallow (at most 64 hidden rows): one 16-entry vocabulary block per
//     wave, 256-wide K-chunks, one chunk of prefetch; several workgroups per
//     CU keep enough W in flight.
//   * deep (more rows): the accumulators of up to 320 rows pin one workgroup
//     to a CU, so W and hidden are prefetched through a 4-deep register ring
//     of 32-wide K-chunks (three chunks in flight while one is multiplied),
//     and each wave owns 2 or 4 vocabulary blocks, so that one LDS read of a
//     hidden fragment feeds 2 or 4 MFMAs.
// The epilogue writes the float32 logits and, per (row, tile), the tile
// maximum and the sum of exp(logit - maximum); a second kernel combines the
// tiles of each row in fixed order into the row's log-sum-exp.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kVThreads = 256;
constexpr int kTileN = 64;  // vocabulary rows per workgroup (4 waves x 16)

// Epilogue of one workgroup.  acc[mb][nb] of a lane holds hidden row
// m0 + mb*16 + (lane & 15) and vocabulary entries (blk0 + nb)*16 + (lane>>4)*4
// .. +3, where blk0 is the wave's first 16-entry block.  Writes the logits,
// then the tile's per-row maximum and sum of exponentials, combined over the
// four waves through `red` ([4][MBW*16] floats).
template <int MBW, int NBW>
__device__ __forceinline__ void tile_epilogue(const f32x4 (&acc)[MBW][NBW], int M, int V, int ntiles, int tile,
                                              int m0, int blk0, float* __restrict__ logits,
                                              float2* __restrict__ partials, float (*red)[MBW * 16]) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;
  const bool v4 = (V % 4) == 0;
  float tmax[MBW];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) {
    const int m = m0 + mb * 16 + lr;
    float x = -INFINITY;
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int v0 = (blk0 + nb) * 16 + lg * 4;
      if (m < M) {
        float* dst = logits + (int64_t)m * V + v0;
        if (v4 && v0 + 3 < V) {
          *reinterpret_cast<f32x4*>(dst) = acc[mb][nb];
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (v0 + i < V) dst[i] = acc[mb][nb][i];
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) x = (v0 + i < V) ? fmaxf(x, acc[mb][nb][i]) : x;
    }
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    if (lg == 0) red[wave][mb * 16 + lr] = x;
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) {
    const int r = mb * 16 + lr;
    tmax[mb] = fmaxf(fmaxf(red[0][r], red[1][r]), fmaxf(red[2][r], red[3][r]));
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) {
    float sm = 0.f;
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int v0 = (blk0 + nb) * 16 + lg * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) sm += (v0 + i < V) ? expf(acc[mb][nb][i] - tmax[mb]) : 0.f;
    }
    sm += __shfl_xor(sm, 16);
    sm += __shfl_xor(sm, 32);
    if (lg == 0) red[wave][mb * 16 + lr] = sm;
  }
  __syncthreads();
  if (wave == 0 && lg == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
      const int r = mb * 16 + lr;
      const int m = m0 + r;
      if (m < M) {
        const float sm = (red[0][r] + red[1][r]) + (red[2][r] + red[3][r]);
        partials[(int64_t)m * ntiles + tile] = make_float2(tmax[mb], sm);
      }
    }
  }
}

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

  f32x4 acc[MB][1];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb][0] = f32x4{0.f, 0.f, 0.f, 0.f};

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
        acc[mb][0] = mfma16x16x32(wcur[ks], a, acc[mb][0]);
      }
    }
    if (more) {
      store_a(buf ^ 1);
#pragma unroll
      for (int ks = 0; ks < C::kSteps; ++ks) wcur[ks] = wnext[ks];
    }
    lds_barrier();
  }

  tile_epilogue<MB, 1>(acc, M, V, ntiles, tile, m0, tile * 4 + wave, logits, partials, red);
}

// Deep schedule: the workgroup's hidden rows (MBW blocks of 16) times
// 4 waves x NBW vocabulary blocks, K in 32-wide chunks.  W fragments go
// through a register ring of 4 slots and hidden pieces through one of 2
// slots.  At chunk c a wave issues the hidden loads of chunk c+2 and the W
// loads of chunk c+3, multiplies chunk c (W from the ring, hidden from LDS
// buffer c&1) and writes hidden chunk c+1 from its ring slot into the other
// LDS buffer.  Loads complete in issue order, so while chunk c is multiplied
// the W of chunks c+1..c+3 and the hidden of c+1..c+2 are in flight, and the
// wait for hidden c+1 never waits for W past c+2.  Loads past the last chunk
// re-read the last chunk (in bounds) and chunks past the end multiply a zero
// W, which keeps the loop free of branches around memory operations.
template <int MBW, int NBW>
struct DeepCfg {
  static constexpr int kRows = MBW * 16;
  static constexpr int kBufBytes = MBW * 1024;  // one 32-wide hidden chunk, fragment order
  static constexpr int kPieces = kRows * 4;     // 16-byte pieces per chunk
  static constexpr int kPiecesPerThread = (kPieces + kVThreads - 1) / kVThreads;
};

template <int MBW, int NBW, bool PACKED>
__global__ __launch_bounds__(kVThreads, 1)
void vocab_bf16_deep_kernel(int M, int K, int V, int ntiles, const uint16_t* __restrict__ hidden,
                            const uint16_t* __restrict__ w, float* __restrict__ logits,
                            float2* __restrict__ partials) {
  using C = DeepCfg<MBW, NBW>;
  constexpr int PPT = C::kPiecesPerThread;
  __shared__ __align__(16) unsigned char abuf[2][C::kBufBytes];
  __shared__ float red[4][C::kRows];

  const int tile = blockIdx.x;
  const int m0 = blockIdx.y * C::kRows;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;
  const int nblk = (V + 15) / 16;
  const int blk0 = (tile * 4 + wave) * NBW;
  const uint16_t* wrow[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb) {
    if (PACKED)
      wrow[nb] = w + ((int64_t)min(nblk - 1, blk0 + nb) * 64 + lane) * 8;
    else
      wrow[nb] = w + (int64_t)min(V - 1, (blk0 + nb) * 16 + lr) * K + lg * 8;
  }
  const int64_t wstep = PACKED ? (int64_t)nblk * 64 * 8 : 32;
  const int nchunks = K / 32;

  // Hidden piece p of a chunk: row p/4 (clamped to M-1; such rows are never
  // stored), 16-byte k piece p%4; pieces past kPieces repeat the last one.
  const uint16_t* hsrc[PPT];
  int hslot[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int p = min((int)threadIdx.x + i * kVThreads, C::kPieces - 1);
    const int row = p >> 2, kp = p & 3;
    hsrc[i] = hidden + (int64_t)min(M - 1, m0 + row) * K + kp * 8;
    hslot[i] = ((row >> 4) * 64 + (row & 15) + 16 * kp) * 16;
  }

  u32x4 hreg[2][PPT];
  bf16x8 wreg[4][NBW];
  auto issue_h = [&](int slot, int c) {
    c = min(c, nchunks - 1);
#pragma unroll
    for (int i = 0; i < PPT; ++i) hreg[slot][i] = *reinterpret_cast<const u32x4*>(hsrc[i] + c * 32);
  };
  auto issue_w = [&](int slot, int c) {
    c = min(c, nchunks - 1);
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) wreg[slot][nb] = load_bf16x8(wrow[nb] + (int64_t)c * wstep);
  };
  auto stage = [&](int slot, int buf) {
#pragma unroll
    for (int i = 0; i < PPT; ++i)
      if (i + 1 < PPT || (int)threadIdx.x + i * kVThreads < C::kPieces)
        *reinterpret_cast<u32x4*>(abuf[buf] + hslot[i]) = hreg[slot][i];
  };

  f32x4 acc[MBW][NBW];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  issue_h(0, 0);
  issue_w(0, 0);
  issue_h(1, 1);
  issue_w(1, 1);
  issue_w(2, 2);
  stage(0, 0);
  lds_barrier();
  for (int c0 = 0; c0 < nchunks; c0 += 4) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int c = c0 + s;
      issue_h(s & 1, c + 2);
      issue_w((s + 3) & 3, c + 3);
      bf16x8 wv[NBW];
      const bool live = c < nchunks;
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) wv[nb] = live ? wreg[s][nb] : bf16x8{};
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb) {
        const bf16x8 a =
            __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(abuf[s & 1] + (mb * 64 + lane) * 16));
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] = mfma16x16x32(wv[nb], a, acc[mb][nb]);
      }
      stage((s + 1) & 1, (s + 1) & 1);
      lds_barrier();
    }
  }
  tile_epilogue<MBW, NBW>(acc, M, V, ntiles, tile, m0, blk0, logits, partials, red);
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
hipError_t launch_shallow(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                          hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid(p.ntiles, p.mtiles), block(kVThreads);
  const uint16_t* h = static_cast<const uint16_t*>(hidden);
  const uint16_t* wv = static_cast<const uint16_t*>(w);
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, true>), grid, block, 0, stream, e0, e1, 0, p.M, p.K, p.V,
                          p.ntiles, h, wv, logits, partials);
  else
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, false>), grid, block, 0, stream, e0, e1, 0, p.M, p.K, p.V,
                          p.ntiles, h, wv, logits, partials);
  return hipGetLastError();
}

template <int MB>
hipError_t launch_shallow_mb(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                             hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if (p.K % 256 == 0) return launch_shallow<MB, 256>(p, hidden, w, logits, partials, stream, e0, e1);
  return launch_shallow<MB, 32>(p, hidden, w, logits, partials, stream, e0, e1);
}

template <int MBW, int NBW>
hipError_t launch_deep(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                       hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid(p.ntiles, p.mtiles), block(kVThreads);
  const uint16_t* h = static_cast<const uint16_t*>(hidden);
  const uint16_t* wv = static_cast<const uint16_t*>(w);
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_deep_kernel<MBW, NBW, true>), grid, block, 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, h, wv, logits, partials);
  else
    hipExtLaunchKernelGGL((vocab_bf16_deep_kernel<MBW, NBW, false>), grid, block, 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, h, wv, logits, partials);
  return hipGetLastError();
}

// Largest row-block count per M-tile of the deep schedule: the accumulators
// (MBW x NBW x 4 registers) stay within the 256 accumulation registers.
constexpr int kDeepMaxBlocks2 = 20;
constexpr int kDeepMaxBlocks4 = 16;
constexpr int kShallowMaxBlocks = 4;

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
  VocabPlan p;
  p.packed = packed;
  p.M = M;
  p.K = K;
  p.V = V;
  const int blocks = (M + 15) / 16;
  if (dtype == 0) {
    p.deep = false;
    p.mblocks = 4;
    p.nbw = 1;
    p.mtiles = (M + 63) / 64;
  } else if (blocks <= kShallowMaxBlocks) {
    p.deep = false;
    p.mblocks = blocks;
    p.nbw = 1;
    p.mtiles = 1;
  } else {
    // Four blocks per wave once the vocabulary still gives at least one
    // 256-wide tile per CU; two otherwise.
    p.deep = true;
    p.nbw = V >= 256 * 256 ? 4 : 2;
    const int cap = p.nbw == 4 ? kDeepMaxBlocks4 : kDeepMaxBlocks2;
    p.mtiles = (blocks + cap - 1) / cap;
    p.mblocks = (blocks + p.mtiles - 1) / p.mtiles;
  }
  p.tile_n = 64 * p.nbw;
  p.ntiles = (V + p.tile_n - 1) / p.tile_n;
  return p;
}

size_t vocab_partial_bytes(const VocabPlan& p) {
  return sizeof(float2) * static_cast<size_t>(p.M) * p.ntiles + 256;
}

hipError_t launch_vocab(int dtype, const VocabPlan& p, const void* hidden, const void* w, float* logits,
                        float2* partials, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if (dtype == 0) {
    hipExtLaunchKernelGGL(vocab_f32_kernel, dim3(p.ntiles, p.mtiles), dim3(kVThreads), 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, static_cast<const float*>(hidden), static_cast<const float*>(w), logits,
                          partials);
    return hipGetLastError();
  }
  if (!p.deep) {
    switch (p.mblocks) {
      case 1: return launch_shallow_mb<1>(p, hidden, w, logits, partials, stream, e0, e1);
      case 2: return launch_shallow_mb<2>(p, hidden, w, logits, partials, stream, e0, e1);
      case 3: return launch_shallow_mb<3>(p, hidden, w, logits, partials, stream, e0, e1);
      case 4: return launch_shallow_mb<4>(p, hidden, w, logits, partials, stream, e0, e1);
      default: return hipErrorInvalidValue;
    }
  }
#define SDV_D(B, N) \
  case B: return launch_deep<B, N>(p, hidden, w, logits, partials, stream, e0, e1);
  if (p.nbw == 4) {
    switch (p.mblocks) {
      SDV_D(5, 4) SDV_D(6, 4) SDV_D(7, 4) SDV_D(8, 4) SDV_D(9, 4) SDV_D(10, 4) SDV_D(11, 4) SDV_D(12, 4)
      SDV_D(13, 4) SDV_D(14, 4) SDV_D(15, 4) SDV_D(16, 4)
      default: return hipErrorInvalidValue;
    }
  }
  switch (p.mblocks) {
    SDV_D(5, 2) SDV_D(6, 2) SDV_D(7, 2) SDV_D(8, 2) SDV_D(9, 2) SDV_D(10, 2) SDV_D(11, 2) SDV_D(12, 2)
    SDV_D(13, 2) SDV_D(14, 2) SDV_D(15, 2) SDV_D(16, 2) SDV_D(17, 2) SDV_D(18, 2) SDV_D(19, 2) SDV_D(20, 2)
    default: return hipErrorInvalidValue;
  }
#undef SDV_D
}

hipError_t launch_lse_combine(const VocabPlan& p, const float2* partials, float* row_lse, hipStream_t stream) {
  hipLaunchKernelGGL(lse_combine_kernel, dim3((p.M + 3) / 4), dim3(kVThreads), 0, stream, p.M, p.ntiles,
                     partials, row_lse);
  return hipGetLastError();
}

}  // namespace sdv
