// Vocabulary projection with a fused softmax-statistics epilogue (gfx950).
//
// logits^T = W hidden^T: a W fragment (vocabulary rows x k) is the MFMA A
// operand and a hidden fragment the B operand, so each lane ends up holding
// four consecutive vocabulary entries of one hidden row, which is what the
// logits store and the row statistics want.
//
// A workgroup owns a tile of vocabulary rows for all hidden rows of its
// M-tile, so W (the dominant stream, K*V*2 bytes) is read from HBM once.
// Every wave streams its own W fragments, either from the [V][K] layout or
// from the fragment-ordered copy sd_pack_vocab makes at weight-load time (1 KB
// contiguous per fragment).  The hidden rows, shared by every workgroup and
// L2-resident, are staged per K-chunk in LDS in fragment order and read by
// all waves.  Three schedules:
//   * shallow (at most 64 hidden rows), MFMA 16x16x32: one 16-entry
//     vocabulary block per wave, 256-wide K-chunks, one chunk of prefetch;
//     several workgroups per CU keep enough W in flight.
//   * deep (more rows), MFMA 32x32x16: the hidden rows are first repacked
//     (pack_hidden_kernel) into 32-row fragments that LDS DMA moves 1 KB at a
//     time; a workgroup's accumulators pin it to a CU.  Three shapes: four
//     waves (one per SIMD) with 1 or 2 blocks of 32 vocabulary entries each,
//     W in a 6-slot register ring and hidden in 6 LDS stages; or eight waves
//     (two per SIMD) with 2 blocks each, a 512-wide tile on a 3-stage ring.
//   * wide (deep rows, large vocabularies): four waves with four blocks of
//     32 vocabulary entries each, a 512-wide tile whose accumulators fill
//     both register files; W and hidden both go to LDS by buffer DMA.
//     vocab_plan picks, among the deep shapes and the wide one, the one whose
//     per-CU inflow (W misses plus hidden hits) is smallest.  Workgroups that
//     share a vocabulary tile (several M-tiles) are dealt to the same XCD.
// W fragments are loaded with the nontemporal hint in every schedule: W is
// read once per launch and should not evict the hidden rows or the logits.
// The epilogue writes the float32 logits and, per (row, tile), the tile
// maximum and the sum of exp(logit - maximum); the row log-sum-exp is folded
// from those in fixed order (lse_combine_kernel, or the acceptance kernel in
// a whole step).
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kVThreads = 256;

// Counters a later launch on the stream expects at zero (the acceptance's
// arrival counters): cleared by the first workgroup of a vocabulary launch.
__device__ __forceinline__ void clear_counters(int* __restrict__ clear, int nclear) {
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < nclear; i += blockDim.x) clear[i] = 0;
}
constexpr int kTileN = 64;  // vocabulary rows per workgroup (4 waves x 16)

// Epilogue of one workgroup of WM x WN waves.  Wave (wm, wn) = (wave / WN,
// wave % WN) holds in acc[mb][nb] hidden row m0 + r0 + mb*16 + (lane & 15),
// with r0 = wm*MBW*16, and vocabulary entries (blk0 + nb)*16 + (lane>>4)*4
// .. +3, where blk0 is the wave's first 16-entry block.  Writes the logits,
// then the tile's per-row maximum and sum of exponentials, combined over the
// WN waves that share the rows through `red` ([WN][WM*MBW*16] floats).
template <int MBW, int NBW, int WM, int WN>
__device__ __forceinline__ void tile_epilogue(const f32x4 (&acc)[MBW][NBW], int M, int V, int ntiles, int tile,
                                              int m0, int blk0, float* __restrict__ logits,
                                              float2* __restrict__ partials, float (*red)[WM * MBW * 16]) {
  const int wave = threadIdx.x >> 6;
  const int wn = wave % WN;
  const int r0 = (wave / WN) * MBW * 16;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;
  const bool v4 = (V % 4) == 0;
  float tmax[MBW];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) {
    const int m = m0 + r0 + mb * 16 + lr;
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
    if (lg == 0) red[wn][r0 + mb * 16 + lr] = x;
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb) {
    const int r = r0 + mb * 16 + lr;
    float x = red[0][r];
#pragma unroll
    for (int w = 1; w < WN; ++w) x = fmaxf(x, red[w][r]);
    tmax[mb] = x;
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
    if (lg == 0) red[wn][r0 + mb * 16 + lr] = sm;
  }
  __syncthreads();
  if (wn == 0 && lg == 0) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
      const int r = r0 + mb * 16 + lr;
      const int m = m0 + r;
      if (m < M) {
        float sm;
        if (WN == 8)
          sm = ((red[0][r] + red[1][r]) + (red[2][r] + red[3][r])) + ((red[4][r] + red[5][r]) + (red[6][r] + red[7][r]));
        else if (WN == 4)
          sm = (red[0][r] + red[1][r]) + (red[2][r] + red[3][r]);
        else if (WN == 2)
          sm = red[0][r] + red[1][r];
        else
          sm = red[0][r];
        partials[(int64_t)m * ntiles + tile] = make_float2(tmax[mb], sm);
      }
    }
  }
}

// Shallow schedule: waves per workgroup.  Every wave of a workgroup multiplies
// the same hidden chunk; eight waves halve the L2 requests that stage it but
// measured slower than four (half as many workgroups in flight per CU).
constexpr int kShallowWaves = 4;

template <int MB, int KC, int NW>
struct VocabCfg {
  static constexpr int kThreads = NW * kWave;
  static constexpr int kSteps = KC / 32;                  // MFMA k-steps per chunk
  static constexpr int kFragBytes = 1024;                 // one 16x32 bf16 fragment
  static constexpr int kBufBytes = MB * kSteps * kFragBytes;
  static constexpr int kPieces = 16 * MB * KC / 8;        // 16-byte pieces per A chunk
  static constexpr int kPiecesPerThread = (kPieces + kThreads - 1) / kThreads;
};

// LDS slot (16 bytes) of lane s of hidden fragment ks in the shallow
// schedule's chunk buffer: the lane holds row s % 16 and k piece g = s / 16;
// the low four bits of the slot are XORed with 2g + (ks & 1) + 8 ((ks >> 1) &
// 1).  Consecutive threads store consecutive 16-byte pieces of one row (g
// fastest, then ks); without the XOR every store of a row lands on the same
// bank group.  With it, any 8 consecutive stores, and any 8 consecutive
// lanes' reads, cover 8 distinct 16-byte slots of a 128-byte span.
__device__ __forceinline__ int shallow_slot(int s, int ks) {
  const int t = 8 * ((ks >> 1) & 1) + 2 * ((s >> 4) & 3) + (ks & 1);
  return (s & 48) | ((s & 15) ^ t);
}

template <int MB, int KC, int NW, bool PACKED>
__global__ __launch_bounds__(NW * kWave)
void vocab_bf16_kernel(int M, int K, int V, int ntiles, const uint16_t* __restrict__ hidden,
                       const uint16_t* __restrict__ w, float* __restrict__ logits,
                       float2* __restrict__ partials, int* __restrict__ clear, int nclear) {
  using C = VocabCfg<MB, KC, NW>;
  clear_counters(clear, nclear);
  __shared__ __align__(16) unsigned char abuf[2][C::kBufBytes];
  __shared__ float red[NW][16 * MB];

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
    wrow = w + ((int64_t)min(nblk - 1, tile * NW + wave) * 64 + lane) * 8;
    wstep = (int64_t)nblk * 64 * 8;
  } else {
    wrow = w + (int64_t)min(V - 1, (tile * NW + wave) * 16 + lr) * K + lg * 8;
    wstep = 32;
  }
  const int nchunks = K / KC;

  // Cooperative A-chunk load: piece p -> (row, 16-byte k piece), coalesced along k.
  u32x4 areg[C::kPiecesPerThread];
  auto load_a = [&](int kc) {
#pragma unroll
    for (int i = 0; i < C::kPiecesPerThread; ++i) {
      const int p = threadIdx.x + i * C::kThreads;
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
      const int p = threadIdx.x + i * C::kThreads;
      if (p < C::kPieces) {
        const int row = p / (KC / 8);
        const int kp = p - row * (KC / 8);
        const int mb = row >> 4, r = row & 15, ks = kp >> 2, g = kp & 3;
        const int slot = (mb * C::kSteps + ks) * 64 + shallow_slot(r + 16 * g, ks);
        *reinterpret_cast<u32x4*>(abuf[buf] + slot * 16) = areg[i];
      }
    }
  };

  // W is read once per launch: the nontemporal hint keeps it from displacing
  // the hidden rows, which every workgroup re-reads from L2 (5.4 -> 5.9 TB/s
  // measured at 48 x 4096 x 32000).
  bf16x8 wcur[C::kSteps], wnext[C::kSteps];
  auto load_w = [&](bf16x8* dst, int kc) {
#pragma unroll
    for (int ks = 0; ks < C::kSteps; ++ks)
      dst[ks] = load_bf16x8_stream(wrow + (int64_t)(kc * C::kSteps + ks) * wstep);
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
            bf16x8, *reinterpret_cast<const u32x4*>(abuf[buf] + ((mb * C::kSteps + ks) * 64 + shallow_slot(lane, ks)) * 16));
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

  tile_epilogue<MB, 1, 1, NW>(acc, M, V, ntiles, tile, m0, tile * NW + wave, logits, partials, red);
}

// Deep schedule (more than 64 rows) on MFMA 32x32x16: the accumulators of up
// to 384 rows pin one workgroup of four waves to a CU, and a single wave per
// SIMD keeps the 32x32 MFMA pipe full where the 16x16 one would stall.  The
// workgroup covers MB blocks of 32 hidden rows and 4 x NB blocks of 32
// vocabulary entries; wave w owns blocks (tile*4 + w)*NB .. +NB, i.e.
// MB x NB accumulators of 16 registers (at most 320).  K goes in 32-wide
// chunks of two 16-wide MFMA steps.
//
// The rate that bounds this kernel is how fast one CU pulls lines in: a CU
// keeps a bounded number of line misses in flight, so its inflow is that
// number over the latency, and a W line (a miss to HBM) holds its place about
// twice as long as a hidden line (an L2 hit).  Every workgroup reads its W
// slice once and the whole M-tile of hidden rows once, so wider vocabulary
// tiles cut the hidden bytes per CU; vocab_plan picks NB per shape.
//
// Pipeline over S stages, chunk c of the loop:
//   * issue chunk c+S-1: its hidden chunk goes straight from global memory
//     into LDS stage (c-1) % S (LDS DMA, no registers), its W fragments into
//     register ring slot (c-1) % S; both slots last served chunk c-1, which
//     every wave finished before the previous step's barrier;
//   * multiply chunk c (ring slot c % S); its hidden fragments were read from
//     LDS stage c % S during the previous step (one wave per SIMD), or are
//     read now, a few MFMAs ahead of their first use (two waves per SIMD);
//   * in the first case, read the fragments of chunk c+1 and wait until this
//     wave's DMA of chunk c+2 has landed; in the second, wait until its loads
//     of chunk c+1 have landed; then barrier, so that chunk is readable by
//     every wave in the next step.
// Memory operations complete in issue order, so the wait leaves the later
// chunks in flight while the next one is multiplied, and no MFMA waits on an
// LDS read issued in the same step when registers allow the read ahead.
// Loads past the last chunk re-read the last chunk (in bounds) and chunks past
// the end multiply a zero W, which keeps the loop free of branches around
// memory operations.
//
// The hidden rows are first repacked (pack_hidden_kernel) into fragments of 32
// rows x 16 k in lane order (lane l: row l%32, k 8*(l/32) .. +8), so every
// DMA instruction moves 1 KB of contiguous memory into one LDS fragment.  W
// fragments (32 vocabulary rows x 16 k, same lane order) are read either from
// the row-major [V][K] layout or gathered from the packed 16x16x32 fragment
// layout.
template <int MB, int NB, int S, int NW>
struct Deep32Cfg {
  static constexpr int kRows = MB * 32;
  static constexpr int kFrags = 2 * MB;                     // hidden fragments per chunk
  static constexpr int kDmaPerWave = (kFrags + NW - 1) / NW;  // the same count on every wave
  static constexpr int kBufBytes = NW * kDmaPerWave * 1024;
  static constexpr int kAhead = S - 1;  // chunks issued ahead of the one multiplied
  // With one wave per SIMD the hidden fragments of chunk c+1 are read into
  // registers while chunk c is multiplied (two register sets of 2*MB
  // fragments); with two waves per SIMD, whose registers hold no second
  // set, each fragment is read a few MFMAs ahead of its first use and the
  // other wave of the SIMD covers what latency is left.
  static constexpr bool kNextChunk = NW == 4;
  // Memory operations a wave issues per chunk, and the most that may still be
  // outstanding at the end of step c: once the hidden chunk c+2 has landed
  // (its W, then chunks c+3 .. c+kAhead) when the next chunk's fragments are
  // read ahead, else once chunk c+1 has landed (chunks c+2 .. c+kAhead).
  static constexpr int kOpsPerChunk = kDmaPerWave + 2 * NB;
  static constexpr int kInFlight = kNextChunk ? 2 * NB + (kAhead - 2) * kOpsPerChunk : (kAhead - 1) * kOpsPerChunk;
  static constexpr int kMfmas = 2 * MB * NB;  // per chunk and wave
  // Just-in-time reads: fragments read ahead of the MFMA that first uses one.
  static constexpr int kReadAhead = NB >= 4 ? 2 : (NB == 2 ? 3 : 5);
  static_assert(S >= (kNextChunk ? 4 : 3) && S <= 6, "LDS stages");
  static_assert(NW == 4 || NW == 8, "one or two waves per SIMD");
  static_assert(kInFlight <= 63, "vmcnt holds 6 bits");
  static_assert(kOpsPerChunk <= kMfmas, "memory operations ride between MFMAs");
};

// Fixed-order combination of the NW per-wave values of row r.
template <int NW, int R>
__device__ __forceinline__ float waves_max(const float (*red)[R], int r) {
  float x = fmaxf(fmaxf(red[0][r], red[1][r]), fmaxf(red[2][r], red[3][r]));
  if (NW == 8) x = fmaxf(x, fmaxf(fmaxf(red[4][r], red[5][r]), fmaxf(red[6][r], red[7][r])));
  return x;
}
template <int NW, int R>
__device__ __forceinline__ float waves_sum(const float (*red)[R], int r) {
  float x = (red[0][r] + red[1][r]) + (red[2][r] + red[3][r]);
  if (NW == 8) x += (red[4][r] + red[5][r]) + (red[6][r] + red[7][r]);
  return x;
}

template <int MB, int NB, int NW>
__device__ __forceinline__ void tile_epilogue32(const f32x16 (&acc)[MB][NB], int M, int V, int ntiles, int tile,
                                                int m0, int blk0, float* __restrict__ logits,
                                                float2* __restrict__ partials, float (*red)[MB * 32]) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int j = lane & 31;
  const int h = lane >> 5;
  const bool v4 = (V % 4) == 0;
  float tmax[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 32 + j;
    float x = -INFINITY;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int v0 = (blk0 + nb) * 32 + 8 * g + 4 * h;
        const f32x4 q = {acc[mb][nb][4 * g], acc[mb][nb][4 * g + 1], acc[mb][nb][4 * g + 2], acc[mb][nb][4 * g + 3]};
        if (m < M) {
          float* dst = logits + (int64_t)m * V + v0;
          if (v4 && v0 + 3 < V) {
            *reinterpret_cast<f32x4*>(dst) = q;
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (v0 + i < V) dst[i] = q[i];
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) x = (v0 + i < V) ? fmaxf(x, q[i]) : x;
      }
    }
    x = fmaxf(x, __shfl_xor(x, 32));
    if (h == 0) red[wave][mb * 32 + j] = x;
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int r = mb * 32 + j;
    tmax[mb] = waves_max<NW, MB * 32>(red, r);
  }
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    float sm = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = (blk0 + nb) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        sm += (v < V) ? expf(acc[mb][nb][r] - tmax[mb]) : 0.f;
      }
    sm += __shfl_xor(sm, 32);
    if (h == 0) red[wave][mb * 32 + j] = sm;
  }
  __syncthreads();
  if (wave == 0 && h == 0) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = mb * 32 + j;
      const int m = m0 + r;
      if (m < M) {
        const float sm = waves_sum<NW, MB * 32>(red, r);
        partials[(int64_t)m * ntiles + tile] = make_float2(tmax[mb], sm);
      }
    }
  }
}

template <int MB, int NB, int S, int NW, bool PACKED>
__global__ __launch_bounds__(NW * kWave, 1)
void vocab_bf16_deep_kernel(int M, int K, int V, int ntiles, int mtiles, const uint16_t* __restrict__ hpacked,
                            const uint16_t* __restrict__ w, float* __restrict__ logits,
                            float2* __restrict__ partials) {
  using C = Deep32Cfg<MB, NB, S, NW>;
  constexpr int ND = C::kDmaPerWave;
  constexpr int kA = C::kAhead;
  constexpr int kB = C::kBufBytes;
  // One LDS object per stage: the compiler then sees that a fragment read
  // and a DMA into another stage cannot alias, and leaves the ordering to the
  // explicit vmcnt waits below.
  __shared__ __align__(1024) unsigned char lds0[kB], lds1[kB], lds2[kB], lds3[S > 3 ? kB : 16],
      lds4[S > 4 ? kB : 16], lds5[S > 5 ? kB : 16];
  __shared__ float red[NW][C::kRows];
  auto abuf = [&](int stage) -> unsigned char* {
    switch (stage) {
      case 0: return lds0;
      case 1: return lds1;
      case 2: return lds2;
      case 3: return lds3;
      case 4: return lds4;
      default: return lds5;
    }
  };

  // Workgroup id -> (tile, M-tile): ids are dealt to the 8 XCDs round-robin,
  // so the M-tiles of one vocabulary tile take ids 8 apart and share an XCD
  // (and its L2), where the second reader of each W line finds it.
  const int grp = 8 * mtiles;
  const int tile = (blockIdx.x / grp) * 8 + (blockIdx.x & 7);
  if (tile >= ntiles) return;
  const int m0 = ((blockIdx.x % grp) >> 3) * C::kRows;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int nblk = (V + 15) / 16;
  const int blk0 = (tile * NW + wave) * NB;  // first 32-entry vocabulary block of the wave
  // W source of this lane for 16-wide k-step ks of chunk 0; chunk c adds c*wstep.
  const uint16_t* wsrc[NB][2];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int row = (blk0 + nb) * 32 + (lane & 31);
      if (PACKED) {
        // Row `row` lives in 16-row block row/16 at lane row%16 + 16*g, where
        // g = 2*ks + lane/32 selects the 8-wide k piece of the 32-wide step.
        const int n16 = min(nblk - 1, row >> 4);
        const int l16 = (row & 15) + 16 * (2 * ks + (lane >> 5));
        wsrc[nb][ks] = w + ((int64_t)n16 * 64 + l16) * 8;
      } else {
        wsrc[nb][ks] = w + (int64_t)min(V - 1, row) * K + ks * 16 + (lane >> 5) * 8;
      }
    }
  const int64_t wstep = PACKED ? (int64_t)nblk * 64 * 8 : 32;
  const int nchunks = K / 32;

  // DMA i of this wave moves fragment f = wave + NW*i (2*mb + ks) of a chunk:
  // 1 KB contiguous in the packed hidden (lane l: row mb*32 + l%32, k
  // 16*ks + 8*(l/32) .. +8).  Fragment numbers past the chunk's 2*MB keep
  // every wave's operation count equal: all their lanes read the same 16
  // bytes of the last fragment (one cache line, one request) into spare LDS
  // space.  Blocks past the packed rows (last M-tile) re-read the last
  // block, whose rows are never stored.  In the last block, lanes of rows
  // past M (zero padding) read the last row's 16 bytes instead: those lines
  // are already requested by the same instruction, so the padding costs no
  // inflow, and the rows it feeds are never stored either.
  const int mbt = (M + 31) / 32;
  const int64_t hstep = (int64_t)2 * mbt * 512;  // elements per 32-wide chunk
  const uint16_t* hsrc[ND];
  int hoff[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) {
    const int f = wave + NW * i;
    const int fs = min(f, C::kFrags - 1);
    const int mbg = min(mbt - 1, m0 / 32 + (fs >> 1));
    const int rlast = M - 1 - mbg * 32;  // last real row of the block (>= 0)
    const int hl = (lane & 32) + min(lane & 31, rlast);
    hsrc[i] = hpacked + (((int64_t)(fs & 1) * mbt + mbg) * 64 + (f < C::kFrags ? hl : 0)) * 8;
    hoff[i] = f * 1024;
  }

  bf16x8 wreg[S][NB][2];
  // Memory operation j (0 <= j < kOpsPerChunk) of chunk c: the hidden DMAs
  // first, then the W loads, always in this order (the vmcnt accounting
  // relies on it).
  auto issue_op = [&](int j, int slot, int c) {
    c = min(c, nchunks - 1);
    if (j < ND) {
      dma_16B_to_lds(hsrc[j] + c * hstep, abuf(slot) + hoff[j]);
    } else {
      const int nb = (j - ND) >> 1, ks = (j - ND) & 1;
      wreg[slot][nb][ks] = load_bf16x8_stream(wsrc[nb][ks] + (int64_t)c * wstep);  // read once
    }
  };
  // Hidden fragment number q of a chunk in MFMA order (q = ks*MB + mb) is
  // LDS fragment 2*mb + ks.
  auto read_frag = [&](int stage, int q) -> bf16x8 {
    const int f = 2 * (q % MB) + q / MB;
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(abuf(stage) + f * 1024 + lane * 16));
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

#pragma unroll
  for (int c = 0; c < kA; ++c)
#pragma unroll
    for (int j = 0; j < C::kOpsPerChunk; ++j) issue_op(j, c, c);
  if constexpr (C::kNextChunk) {
    bf16x8 af[2][C::kFrags];
    wait_vmcnt<2 * NB + (kA - 2) * C::kOpsPerChunk>();  // chunks 0 and 1 have landed
    lds_barrier();
#pragma unroll
    for (int q = 0; q < C::kFrags; ++q) af[0][q] = read_frag(0, q);
    for (int c0 = 0; c0 < nchunks; c0 += S) {
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int c = c0 + s;
        const bool live = c < nchunks;
        // One MFMA, then one other instruction: the loads of chunk c+S-1 and
        // the fragment reads of chunk c+1 fill the issue slots between MFMAs,
        // so a single wave keeps the matrix pipe busy while they go out.
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          bf16x8 wv[NB];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) wv[nb] = live ? wreg[s][nb][ks] : bf16x8{};
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              const int q = ks * MB + mb;
              const int i = q * NB + nb;
              acc[mb][nb] = mfma32x32x16(wv[nb], af[s & 1][q], acc[mb][nb]);
              if (i < C::kOpsPerChunk)
                issue_op(i, (s + kA) % S, c + kA);
              else if (i - C::kOpsPerChunk < C::kFrags)
                af[(s + 1) & 1][i - C::kOpsPerChunk] = read_frag((s + 1) % S, i - C::kOpsPerChunk);
              __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int q = C::kMfmas - C::kOpsPerChunk; q < C::kFrags; ++q)
          if (q >= 0) af[(s + 1) & 1][q] = read_frag((s + 1) % S, q);
        wait_vmcnt<C::kInFlight>();
        lds_barrier();
      }
    }
  } else {
    wait_vmcnt<(kA - 1) * C::kOpsPerChunk>();  // chunk 0 has landed
    lds_barrier();
    for (int c0 = 0; c0 < nchunks; c0 += S) {
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int c = c0 + s;
        const bool live = c < nchunks;
        bf16x8 hf[C::kFrags];
#pragma unroll
        for (int q = 0; q < C::kReadAhead && q < C::kFrags; ++q) hf[q] = read_frag(s, q);
        // One MFMA, then at most one other instruction: the loads of chunk
        // c+S-1 and the fragment reads fill the issue slots between MFMAs.
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          bf16x8 wv[NB];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) wv[nb] = live ? wreg[s][nb][ks] : bf16x8{};
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            const int q = ks * MB + mb;
            if (q + C::kReadAhead < C::kFrags) hf[q + C::kReadAhead] = read_frag(s, q + C::kReadAhead);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              const int i = q * NB + nb;
              acc[mb][nb] = mfma32x32x16(wv[nb], hf[q], acc[mb][nb]);
              if (i < C::kOpsPerChunk) issue_op(i, (s + kA) % S, c + kA);
              __builtin_amdgcn_sched_barrier(0);
            }
          }
        }
        wait_vmcnt<C::kInFlight>();
        lds_barrier();
      }
    }
  }
  tile_epilogue32<MB, NB, NW>(acc, M, V, ntiles, tile, m0, blk0, logits, partials, red);
}

// Wide deep schedule: four waves (one per SIMD), four blocks of 32 vocabulary
// entries per wave (a 512-wide tile) and up to seven 32-row blocks, so a CU
// pulls its M-tile of hidden rows once per 512 vocabulary entries instead of
// once per 256.  A wave then holds up to 28 accumulators (448 registers): the
// compiler keeps MFMA accumulators in the 256 accumulation registers only, so
// the first 16 accumulators are left to it and the MFMAs of the others are
// written out with their accumulators in VGPRs.  With the VGPRs taken by
// accumulators, no load lands in registers: W and the hidden fragments both go
// to LDS by buffer DMA (a 32-bit lane offset per operation, the chunk in a
// scalar), three 48 KB stages, chunks issued two ahead; each wave DMAs and
// reads its own W fragments and a quarter of the shared hidden ones.  The
// loop runs a multiple of three chunks; chunks past the end are read through
// an empty buffer range, which returns zeros, so they add nothing.
constexpr int kWideNB = 4;     // 32-entry vocabulary blocks per wave
constexpr int kWideAgpr = 16;  // accumulators kept in the accumulation registers
constexpr int kWideMaxMB = 7;  // 16 + 12 accumulators of 16 registers

__device__ __forceinline__ void mfma32x32x16_vgpr(f32x16& c, bf16x8 a, bf16x8 b) {
  asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
// The MFMAs above are opaque to the compiler's hazard tracking: separate the
// zeroing of their accumulators before the loop, and the reads of the
// epilogue, from them by more wait states than an XDL op of 8 passes needs.
__device__ __forceinline__ void mfma_asm_fence() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}
// Copy of an accumulator held in accumulation registers, read where it is
// used: left to itself the compiler copies every such accumulator to VGPRs
// at the end of the loop, which does not fit next to the VGPR accumulators.
__device__ __forceinline__ f32x16 agpr_take(const f32x16& a) {
  f32x16 v;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float t;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(t) : "a"(a[r]));
    v[r] = t;
  }
  return v;
}

typedef __amdgpu_buffer_rsrc_t BufRsrc;
constexpr int kRawBufferWord3 = 0x00020000;  // gfx9 raw buffer: 32-bit data format, no swizzle
__device__ __forceinline__ BufRsrc raw_buffer(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRawBufferWord3);
}
// Buffer DMA: lane l copies 16 bytes at byte offset voff + soff of the buffer
// into LDS at lds + 16*l; offsets past the buffer's size read zeros.  NT sets
// the nontemporal hint (read-once data, as for the register loads of W).
template <bool NT>
__device__ __forceinline__ void dma_16B_buffer_to_lds(BufRsrc r, uint32_t voff, uint32_t soff, void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, (int)voff, (int)soff,
                                           0, NT ? 2 : 0);
}

// Epilogue of the wide schedule, one 32-row block at a time (the blocks with
// VGPR accumulators first, which frees their registers): store the block's
// logits, form the wave's maximum and sum of exponentials per row, then
// combine the four waves' (maximum, sum) pairs of a row in wave order, each
// sum rescaled to the tile maximum.
template <int MB, int NB, int NW>
__device__ __forceinline__ void tile_epilogue_wide(const f32x16 (&acc)[MB][NB], int M, int V, int ntiles, int tile,
                                                   int m0, int blk0, float* __restrict__ logits,
                                                   float2* __restrict__ partials, float2 (*red)[MB * 32]) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int j = lane & 31;
  const int h = lane >> 5;
  const bool full = (V % 4) == 0 && (blk0 + NB) * 32 <= V;  // wave-uniform
#pragma unroll
  for (int mb = MB - 1; mb >= 0; --mb) {
    f32x16 av[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) av[nb] = (mb * NB + nb < kWideAgpr) ? agpr_take(acc[mb][nb]) : acc[mb][nb];
    const int m = m0 + mb * 32 + j;
    float x = -INFINITY;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int v0 = (blk0 + nb) * 32 + 8 * g + 4 * h;
        const f32x4 q = {av[nb][4 * g], av[nb][4 * g + 1], av[nb][4 * g + 2], av[nb][4 * g + 3]};
        float* dst = logits + (int64_t)m * V + v0;
        if (full) {
          if (m < M) *reinterpret_cast<f32x4*>(dst) = q;
          x = fmaxf(x, fmaxf(fmaxf(q[0], q[1]), fmaxf(q[2], q[3])));
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (m < M && v0 + i < V) dst[i] = q[i];
            x = (v0 + i < V) ? fmaxf(x, q[i]) : x;
          }
        }
      }
    }
    x = fmaxf(x, __shfl_xor(x, 32));
    float sm = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = (blk0 + nb) * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        sm += (full || v < V) ? expf(av[nb][r] - x) : 0.f;
      }
    sm += __shfl_xor(sm, 32);
    if (h == 0) red[wave][mb * 32 + j] = make_float2(x, sm);
  }
  __syncthreads();
  if (wave == 0 && h == 0) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = mb * 32 + j;
      const int m = m0 + r;
      if (m < M) {
        float mx = red[0][r].x;
#pragma unroll
        for (int w = 1; w < NW; ++w) mx = fmaxf(mx, red[w][r].x);
        float sm = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const float2 e = red[w][r];
          sm += e.y > 0.f ? e.y * expf(e.x - mx) : 0.f;  // a wave wholly past V holds (-inf, 0)
        }
        partials[(int64_t)m * ntiles + tile] = make_float2(mx, sm);
      }
    }
  }
}

template <int MB, bool PACKED>
__global__ __launch_bounds__(4 * kWave, 1)
void vocab_bf16_wide_kernel(int M, int K, int V, int ntiles, int mtiles, const uint16_t* __restrict__ hpacked,
                            const uint16_t* __restrict__ w, float* __restrict__ logits,
                            float2* __restrict__ partials) {
  constexpr int NB = kWideNB, NW = 4, S = 3;
  constexpr int kFrags = 2 * MB;               // hidden fragments per chunk
  constexpr int kHd = (kFrags + NW - 1) / NW;  // hidden DMAs per wave and chunk
  constexpr int kWd = 2 * NB;                  // W DMAs per wave and chunk
  constexpr int kOps = kHd + kWd;              // memory operations per wave and chunk
  constexpr int kHBytes = NW * kHd * 1024;
  constexpr int kStage = kHBytes + NW * kWd * 1024;
  static_assert(MB >= 2 && MB <= kWideMaxMB, "accumulators: 16 + 12 of 16 registers");
  static_assert(kOps <= 2 * MB * NB, "memory operations ride between MFMAs");
  __shared__ __align__(1024) unsigned char lds0[kStage], lds1[kStage], lds2[kStage];
  __shared__ float2 red[NW][MB * 32];

  // Workgroup id -> (tile, M-tile) as in the deep kernel: the M-tiles of one
  // vocabulary tile share an XCD.
  const int grp = 8 * mtiles;
  const int tile = (blockIdx.x / grp) * 8 + (blockIdx.x & 7);
  if (tile >= ntiles) return;
  const int m0 = ((blockIdx.x % grp) >> 3) * MB * 32;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int blk0 = (tile * NW + wave) * NB;  // first 32-entry vocabulary block of the wave
  const int nchunks = K / 32;

  // W fragment (nb, ks) of chunk c: byte woff[nb][ks] + c*wstep of W.
  // Packed layout: 32-entry block b is 16-row blocks 2b (lanes with bit 4
  // clear) and 2b+1, 512 B each per 16-wide k-step; blocks past the packed
  // rows read the last one, and a block whose upper half is past them reads
  // its lower half twice (rows past V are never stored).  Row-major: lane l
  // reads row 32b + l%32 (clamped to V-1), k 8*(l/32) .. +8 of the step.
  // The plan takes this schedule only for W under 4 GB.
  const int nblk = (V + 15) / 16;
  uint32_t woff[NB][2];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int b = blk0 + nb;
    uint32_t o;
    if (PACKED) {
      const int lo16 = min(2 * b, nblk - 1);
      const bool upper = 2 * b + 1 < nblk;
      o = (uint32_t)lo16 * 1024u + 2u * ((upper ? ((lane >> 4) & 1) * 512 : 0) + (lane & 15) * 8 + (lane >> 5) * 128);
    } else {
      const int r0 = min(b * 32, V - 1);
      o = 2u * ((uint32_t)(r0 + min(lane & 31, V - 1 - r0)) * (uint32_t)K + (lane >> 5) * 8);
    }
    woff[nb][0] = o;
    woff[nb][1] = o + (PACKED ? 512u : 32u);
  }
  const uint32_t wstep = PACKED ? (uint32_t)nblk * 1024u : 64u;  // bytes per 32-wide chunk
  const uint32_t wbytes = PACKED ? (uint32_t)nchunks * wstep : (uint32_t)V * (uint32_t)K * 2u;

  // Hidden DMA i of this wave moves fragment f = wave + 4i of a chunk into
  // LDS fragment f, as the deep kernel's do: numbers past 2*MB are dummies
  // (every lane reads the last fragment's first 16 bytes), blocks past the
  // packed rows re-read the last one, and lanes of rows past M in the last
  // block read the last row's bytes.
  const int mbt = (M + 31) / 32;
  const uint32_t hstep = 2u * mbt * 1024u;  // bytes per 32-wide chunk
  uint32_t hoff[kHd];
#pragma unroll
  for (int i = 0; i < kHd; ++i) {
    const int f = wave + NW * i;
    const int fs = min(f, kFrags - 1);
    const int mbg = min(mbt - 1, m0 / 32 + (fs >> 1));
    const int rlast = M - 1 - mbg * 32;
    hoff[i] = (uint32_t)((fs & 1) * mbt + mbg) * 1024u +
              (f < kFrags ? 16u * ((lane & 32) + min(lane & 31, rlast)) : 0u);
  }
  const BufRsrc wbuf = raw_buffer(w, wbytes);
  const BufRsrc hbuf = raw_buffer(hpacked, (uint32_t)nchunks * hstep);
  const BufRsrc nobuf = raw_buffer(w, 0u);  // every read past its end: zeros

  // Operation j of chunk c into LDS stage dst.
  auto issue_op = [&](int j, unsigned char* dst, int c) {
    const bool live = c < nchunks;  // uniform
    if (j < kHd) {
      dma_16B_buffer_to_lds<false>(live ? hbuf : nobuf, hoff[j], live ? (uint32_t)c * hstep : 0u,
                                   dst + (wave + NW * j) * 1024);
    } else {
      const int nb = (j - kHd) >> 1, ks = (j - kHd) & 1;
      dma_16B_buffer_to_lds<true>(live ? wbuf : nobuf, woff[nb][ks], live ? (uint32_t)c * wstep : 0u,
                                  dst + kHBytes + (wave * kWd + 2 * nb + ks) * 1024);
    }
  };
  auto read_h = [&](const unsigned char* src, int q) -> bf16x8 {  // q = ks*MB + mb
    const int f = 2 * (q % MB) + q / MB;
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(src + f * 1024 + lane * 16));
  };
  auto read_w = [&](const unsigned char* src, int nb, int ks) -> bf16x8 {
    return __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(src + kHBytes + (wave * kWd + 2 * nb + ks) * 1024 + lane * 16));
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;
  mfma_asm_fence();

#pragma unroll
  for (int c = 0; c < S - 1; ++c)
#pragma unroll
    for (int j = 0; j < kOps; ++j) issue_op(j, c == 0 ? lds0 : lds1, c);
  // A wave's W fragments are its own (only its own DMA writes them), so it
  // reads those of the first k-step of the next chunk as soon as its own
  // loads have landed, before the barrier the hidden fragments need.
  bf16x8 wf[2][NB];
  wait_vmcnt<kOps>();  // chunk 0 has landed
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) wf[0][nb] = read_w(lds0, nb, 0);
  lds_barrier();
  for (int c0 = 0; c0 < nchunks; c0 += S) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
      const int c = c0 + s;
      const unsigned char* cur = s == 0 ? lds0 : (s == 1 ? lds1 : lds2);
      unsigned char* nxt = s == 0 ? lds2 : (s == 1 ? lds0 : lds1);  // chunk c+2 goes where chunk c-1 was
      bf16x8 hf[2];
      hf[0] = read_h(cur, 0);
      // One MFMA, then at most a DMA and a fragment read: the hidden
      // fragment of the next (ks, mb) is read four MFMAs before its first
      // use, the W fragments of the second k-step during the first.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int q = ks * MB + mb;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const int i = q * NB + nb;
            if (mb * NB + nb < kWideAgpr)
              acc[mb][nb] = mfma32x32x16(wf[ks][nb], hf[q & 1], acc[mb][nb]);
            else
              mfma32x32x16_vgpr(acc[mb][nb], wf[ks][nb], hf[q & 1]);
            if (i < kOps) issue_op(i, nxt, c + S - 1);
            if (nb == 0 && q + 1 < kFrags) hf[(q + 1) & 1] = read_h(cur, q + 1);
            if (ks == 0 && mb == MB - 2) wf[1][nb] = read_w(cur, nb, 1);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      wait_vmcnt<kOps>();  // chunk c+1 has landed; chunk c+2 stays in flight
      const unsigned char* after = s == 0 ? lds1 : (s == 1 ? lds2 : lds0);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) wf[0][nb] = read_w(after, nb, 0);
      lds_barrier();
    }
  }
  wait_vmcnt<0>();
  mfma_asm_fence();
  tile_epilogue_wide<MB, NB, NW>(acc, M, V, ntiles, tile, m0, blk0, logits, partials, red);
}

// Hidden rows [M][K] -> fragments [K/16][ceil(M/32)][64 lanes][8]: lane l of
// fragment (k16, mb) holds row mb*32 + l%32, k 16*k16 + 8*(l/32) .. +8; rows
// past M are zero.  One thread per 16-byte piece, writes coalesced.
__global__ __launch_bounds__(kVThreads)
void pack_hidden_kernel(int M, int K, const uint16_t* __restrict__ hidden, uint16_t* __restrict__ out,
                        int* __restrict__ clear, int nclear) {
  clear_counters(clear, nclear);
  const int mbt = (M + 31) / 32;
  const int64_t pieces = (int64_t)(K / 16) * mbt * 64;
  for (int64_t i = (int64_t)blockIdx.x * kVThreads + threadIdx.x; i < pieces; i += (int64_t)gridDim.x * kVThreads) {
    const int lane = (int)(i & 63);
    const int64_t f = i >> 6;
    const int mb = (int)(f % mbt);
    const int k16 = (int)(f / mbt);
    const int row = mb * 32 + (lane & 31);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < M) v = *reinterpret_cast<const u32x4*>(hidden + (int64_t)row * K + k16 * 16 + (lane >> 5) * 8);
    *reinterpret_cast<u32x4*>(out + i * 8) = v;
  }
}

// float32 path: 64 rows x 64 vocabulary entries per workgroup, LDS-tiled FMA.
constexpr int kF32KC = 32;
__global__ __launch_bounds__(kVThreads)
void vocab_f32_kernel(int M, int K, int V, int ntiles, const float* __restrict__ hidden,
                      const float* __restrict__ w, float* __restrict__ logits,
                      float2* __restrict__ partials, int* __restrict__ clear, int nclear) {
  clear_counters(clear, nclear);
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
                          hipStream_t stream, hipEvent_t e0, hipEvent_t e1, int* clear, int nclear) {
  const dim3 grid(p.ntiles, p.mtiles), block(kShallowWaves * kWave);
  const uint16_t* h = static_cast<const uint16_t*>(hidden);
  const uint16_t* wv = static_cast<const uint16_t*>(w);
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, kShallowWaves, true>), grid, block, 0, stream, e0, e1, 0, p.M,
                          p.K, p.V, p.ntiles, h, wv, logits, partials, clear, nclear);
  else
    hipExtLaunchKernelGGL((vocab_bf16_kernel<MB, KC, kShallowWaves, false>), grid, block, 0, stream, e0, e1, 0, p.M,
                          p.K, p.V, p.ntiles, h, wv, logits, partials, clear, nclear);
  return hipGetLastError();
}

template <int MB>
hipError_t launch_shallow_mb(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                             hipStream_t stream, hipEvent_t e0, hipEvent_t e1, int* clear, int nclear) {
  if (p.K % 256 == 0) return launch_shallow<MB, 256>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
  return launch_shallow<MB, 32>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
}

template <int MB, int NB, int NW, int S = (NW == 8 ? 3 : 6)>
hipError_t launch_deep(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                       uint16_t* hpacked, hipStream_t stream, hipEvent_t e0, hipEvent_t e1, int* clear, int nclear) {
  const int64_t pieces = (int64_t)(p.K / 16) * ((p.M + 31) / 32) * 64;
  const int pblocks = (int)std::min<int64_t>((pieces + kVThreads - 1) / kVThreads, 4096);
  // The events bracket the projection kernel alone (the repacking is a few
  // microseconds of latency before it), so that they time the same launch a
  // kernel trace lists.
  hipExtLaunchKernelGGL(pack_hidden_kernel, dim3(pblocks), dim3(kVThreads), 0, stream, nullptr, nullptr, 0, p.M, p.K,
                        static_cast<const uint16_t*>(hidden), hpacked, clear, nclear);
  const dim3 grid((p.ntiles + 7) / 8 * 8 * p.mtiles), block(NW * kWave);
  const uint16_t* wv = static_cast<const uint16_t*>(w);
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_deep_kernel<MB, NB, S, NW, true>), grid, block, 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, p.mtiles, hpacked, wv, logits, partials);
  else
    hipExtLaunchKernelGGL((vocab_bf16_deep_kernel<MB, NB, S, NW, false>), grid, block, 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, p.mtiles, hpacked, wv, logits, partials);
  return hipGetLastError();
}

template <int MB>
hipError_t launch_wide(const VocabPlan& p, const void* hidden, const void* w, float* logits, float2* partials,
                       uint16_t* hpacked, hipStream_t stream, hipEvent_t e0, hipEvent_t e1, int* clear, int nclear) {
  const int64_t pieces = (int64_t)(p.K / 16) * ((p.M + 31) / 32) * 64;
  const int pblocks = (int)std::min<int64_t>((pieces + kVThreads - 1) / kVThreads, 4096);
  hipExtLaunchKernelGGL(pack_hidden_kernel, dim3(pblocks), dim3(kVThreads), 0, stream, nullptr, nullptr, 0, p.M, p.K,
                        static_cast<const uint16_t*>(hidden), hpacked, clear, nclear);
  const dim3 grid((p.ntiles + 7) / 8 * 8 * p.mtiles), block(4 * kWave);
  const uint16_t* wv = static_cast<const uint16_t*>(w);
  if (p.packed)
    hipExtLaunchKernelGGL((vocab_bf16_wide_kernel<MB, true>), grid, block, 0, stream, e0, e1, 0, p.M, p.K, p.V,
                          p.ntiles, p.mtiles, hpacked, wv, logits, partials);
  else
    hipExtLaunchKernelGGL((vocab_bf16_wide_kernel<MB, false>), grid, block, 0, stream, e0, e1, 0, p.M, p.K, p.V,
                          p.ntiles, p.mtiles, hpacked, wv, logits, partials);
  return hipGetLastError();
}

// Deep schedules: NB blocks of 32 vocabulary entries per wave, NW waves per
// workgroup (one or two per SIMD), and the most 32-row blocks per M-tile
// that keep a wave's accumulators (MB x NB x 16) in its share of the
// accumulation registers (256 with one wave per SIMD, 160 of the 256
// registers of each of two) next to the W ring (S x NB x 8 registers).
struct DeepShape {
  int nb, nw, cap;
};
constexpr DeepShape kDeepShapes[4] = {{1, 4, 12}, {2, 4, 7}, {2, 8, 5}, {kWideNB, 4, kWideMaxMB}};
constexpr int kShallowMaxBlocks = 4;  // 16-row blocks of the shallow schedule

// Per-CU cost of a deep plan in the inflow model of the deep kernel: the
// workgroups a CU runs one after another (CUs of the MI355X: 256), each
// pulling its M-tile of hidden rows (L2 hits) and its W slice, per unit of K.
// The M-tiles of one vocabulary tile run on one XCD at the same time, so the
// first reader of a W line misses to HBM (weight 2.1 against an L2 hit) and
// the others find it in L2.
constexpr int kModelCUs = 256;
constexpr double kMissWeight = 2.1;

double deep_cost(int blocks32, int V, const DeepShape& d, int* mtiles, int* mblocks) {
  *mtiles = (blocks32 + d.cap - 1) / d.cap;
  *mblocks = (blocks32 + *mtiles - 1) / *mtiles;
  const int tile_n = 32 * d.nb * d.nw;
  const long long wgs = (long long)((V + tile_n - 1) / tile_n) * *mtiles;
  const long long rounds = (wgs + kModelCUs - 1) / kModelCUs;
  const double w_weight = (kMissWeight + (*mtiles - 1)) / *mtiles;
  return (double)rounds * (w_weight * tile_n + 32.0 * *mblocks);
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
    p.waves = 4;
    p.mtiles = (M + 63) / 64;
  } else if (blocks <= kShallowMaxBlocks) {
    p.deep = false;
    p.mblocks = blocks;
    p.nbw = kShallowWaves / 4;  // a 16-entry block per wave
    p.waves = 4;
    p.mtiles = 1;
  } else {
    // The deep shape the inflow model prices lowest (ties go to the
    // narrower tile).
    const int blocks32 = (M + 31) / 32;
    p.deep = true;
    double best = 0.0;
    // The wide schedule addresses W and the hidden rows with 32-bit offsets.
    const bool small = (uint64_t)K * (((uint64_t)V + 31) / 32 * 32) * 2 < (1ull << 32) &&
                       (uint64_t)K * (uint64_t)blocks32 * 64 < (1ull << 32);
    for (int i = 0; i < 4; ++i) {
      if (kDeepShapes[i].nb == kWideNB && !small) continue;
      int mt, mb;
      const double cost = deep_cost(blocks32, V, kDeepShapes[i], &mt, &mb);
      if (i == 0 || cost < best) {
        best = cost;
        p.nbw = 2 * kDeepShapes[i].nb;
        p.waves = kDeepShapes[i].nw;
        p.mtiles = mt;
        p.mblocks = mb;
      }
    }
  }
  p.tile_n = 16 * p.waves * p.nbw;
  p.ntiles = (V + p.tile_n - 1) / p.tile_n;
  return p;
}

static size_t partial_bytes(const VocabPlan& p) {
  return (sizeof(float2) * static_cast<size_t>(p.M) * p.ntiles + 255) / 256 * 256;
}

size_t vocab_workspace_bytes(const VocabPlan& p) {
  size_t b = partial_bytes(p);
  if (p.deep) b += sizeof(uint16_t) * static_cast<size_t>(p.K) * ((static_cast<size_t>(p.M) + 31) / 32) * 32;
  return b;
}

hipError_t launch_vocab(int dtype, const VocabPlan& p, const void* hidden, const void* w, float* logits,
                        void* workspace, hipStream_t stream, hipEvent_t e0, hipEvent_t e1, int* clear, int nclear) {
  if (clear == nullptr) nclear = 0;
  float2* partials = static_cast<float2*>(workspace);
  uint16_t* hpacked = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + partial_bytes(p));
  if (dtype == 0) {
    hipExtLaunchKernelGGL(vocab_f32_kernel, dim3(p.ntiles, p.mtiles), dim3(kVThreads), 0, stream, e0, e1, 0, p.M, p.K,
                          p.V, p.ntiles, static_cast<const float*>(hidden), static_cast<const float*>(w), logits,
                          partials, clear, nclear);
    return hipGetLastError();
  }
  if (!p.deep) {
    switch (p.mblocks) {
      case 1: return launch_shallow_mb<1>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
      case 2: return launch_shallow_mb<2>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
      case 3: return launch_shallow_mb<3>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
      case 4: return launch_shallow_mb<4>(p, hidden, w, logits, partials, stream, e0, e1, clear, nclear);
      default: return hipErrorInvalidValue;
    }
  }
#define SDV_D(B, N, W) \
  case B: return launch_deep<B, N, W>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
  if (p.nbw == 2 * kWideNB) {
    switch (p.mblocks) {
      case 2: return launch_wide<2>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      case 3: return launch_wide<3>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      case 4: return launch_wide<4>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      case 5: return launch_wide<5>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      case 6: return launch_wide<6>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      case 7: return launch_wide<7>(p, hidden, w, logits, partials, hpacked, stream, e0, e1, clear, nclear);
      default: return hipErrorInvalidValue;
    }
  }
  if (p.waves == 8) {
    switch (p.mblocks) {
      SDV_D(2, 2, 8) SDV_D(3, 2, 8) SDV_D(4, 2, 8) SDV_D(5, 2, 8)
      default: return hipErrorInvalidValue;
    }
  }
  if (p.nbw == 4) {
    switch (p.mblocks) {
      SDV_D(2, 2, 4) SDV_D(3, 2, 4) SDV_D(4, 2, 4) SDV_D(5, 2, 4) SDV_D(6, 2, 4) SDV_D(7, 2, 4)
      default: return hipErrorInvalidValue;
    }
  }
  switch (p.mblocks) {
    SDV_D(2, 1, 4) SDV_D(3, 1, 4) SDV_D(4, 1, 4) SDV_D(5, 1, 4) SDV_D(6, 1, 4) SDV_D(7, 1, 4) SDV_D(8, 1, 4)
    SDV_D(9, 1, 4) SDV_D(10, 1, 4) SDV_D(11, 1, 4) SDV_D(12, 1, 4)
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
