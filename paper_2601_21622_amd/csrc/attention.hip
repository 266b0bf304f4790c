// Causal multi-query verification attention (split-KV) for gfx950.
//
// Each request b brings G = gamma + 1 queries (root + drafts) per query head;
// query j sees keys 0 .. L_b - G + j of the request's own KV segment.  With
// grouped-query attention the G * group queries that share a KV head form the
// "rows" of one KV head, and every key/value vector is read from HBM once for
// all of them.
//
// Work split: one wave per work item (request chunk of `chunk_keys` keys, KV
// head); a workgroup holds four independent items, so no wave waits on
// another.  The host picks the chunk length from the total work and the
// number of workgroups a launch round holds (attn_chunk_keys).  Two bf16
// kernels:
//   * one 16-row block (multi-head attention: the G queries of one head):
//     each wave loads the next 32-key tile's K rows (before it folds in the
//     current tile) and V rows (in the middle of the fold) into its other
//     register set; K and V then pass through wave-private LDS tiles, so that
//     the transposing read ds_read_b64_tr_b16 hands each lane its V^T
//     fragment;
//   * several 16-row blocks (grouped-query attention): K and V tiles go from
//     HBM into wave-private LDS stages by DMA (no registers, completion
//     tracked with explicit vmcnt waits), one tile ahead, the next tile's
//     DMAs spread over the current tile's fold.
// Both compute S^T = K Q^T and O^T += V^T P^T on MFMA 16x16x32 bf16 (the Q
// fragments stay in registers, P comes straight from the S^T accumulator
// layout) with the online softmax in the log2 domain, each lane owning one
// query row.  The one-block kernel moves a row's reference maximum lazily
// (O is rescaled only when the maximum grows by more than 2^8); the
// several-block kernel never rescales O: its first tile sets the maxima, and
// a later growth beyond 2^64 restarts the item with the grown maxima.  Each
// item writes one partial (max, sum, O) to the workspace; a combine kernel
// (or, in a whole step, the acceptance's last launch) merges the chunks of
// each request in fixed order and writes O in the input dtype.  LDS tiles keep
// rows whole but rotate their 16-byte pieces so that the fragment reads
// mostly avoid bank conflicts (rocprofv3 counts 0.8 conflict cycles per LDS
// instruction in the one-block kernel, 1.3 in the other).
#include <hip/hip_ext.h>

#include <atomic>
#include <climits>
#include <type_traits>

#include "combine.h"
#include "common.h"
#include "launch.h"

namespace sdv {

namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = 4;
constexpr int kTile = 32;
constexpr int kF32ChunkKeys = 128;
constexpr int kMinChunkKeys = 512;
constexpr int kMaxChunkKeys = 4096;
// Work items aimed for: about one per resident wave of the one-block kernel
// (2048 slots), about four per resident wave of the multi-block kernel
// (1024 slots, whose row groups come with long, uneven contexts).
constexpr int64_t kAttnTargetItemsOne = 2048;
constexpr int64_t kAttnTargetItemsMany = 4096;
// Small batches of the one-block kernel: when the default split leaves CUs
// without a workgroup, the shortest chunk (>= kRoundMinKeys) whose
// workgroups fit one round of one per CU is taken instead (shorter chunks
// that spill into a second workgroup on some CUs were measured slower).
constexpr int kRoundMinKeys = 160;
constexpr int64_t kRoundWorkgroups = 256;
// Start-up cost of one work item (query rows, pipeline fill, partial write),
// in keys of streaming, for the round estimate of the multi-block kernel.
constexpr int64_t kItemStartKeys = 256;
// Most 16-row blocks one wave holds at head dimension 128: O takes 32
// accumulator registers per block and the Q fragments 16, and at six blocks
// the several-block kernel spills to scratch.  Wider row sets split over
// row groups (each wave re-reads the item's K and V tiles, mostly from cache,
// since the waves of one KV head share a workgroup).
constexpr int kMaxRowBlocks = 5;

// Compute units of the current device (cached per device; 256 on MI355X).
int64_t device_cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}


__device__ __forceinline__ int find_request(const AttnBatch& bt, int c) {
  int lo = 0, hi = bt.nreq - 1;  // largest b with chunk_prefix[b] <= c
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (bt.chunk_prefix[mid] <= c) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Visibility of key `key` to a row: every prefix key up to pend, then the G
// tail positions (root, then drafts or tree nodes) whose bit is set in anc.
// A chain row j has anc = bits 0..j (causal); a padding row has pend = -1 and
// anc = 0 (nothing visible).
__device__ __forceinline__ bool key_visible(int key, int pend, uint64_t anc) {
  const unsigned off = (unsigned)(key - pend - 1);
  return key <= pend || (off < 64u && ((anc >> off) & 1ull));
}

__device__ __forceinline__ uint64_t chain_mask(int j) { return j >= 63 ? ~0ull : ((2ull << j) - 1ull); }

// Online softmax over a 32-key tile, in the log2 domain, for RB 16-row
// blocks at once: in block rb the lane owns row lr and keys
// k0 + kb*16 + lg*4 + e.  The reference maximum m of each row moves lazily:
// only when some row's tile maximum exceeds its m by more than kLazyLog2 does
// the wave (one uniform branch for all blocks) move every m to the new maxima
// and rescale the sums and O (rows whose maximum did not grow get alpha = 1).
// Otherwise p = 2^(s*scale - m) stays below 2^kLazyLog2, well inside float32
// and bfloat16 range, and O and the sum share the same m, so the normalised
// result is unchanged.  The branch is rarely taken after the first tiles of a
// chunk, so O's accumulators are normally touched by the MFMAs alone.
// Masking (key_visible) depends on MK: never (tiles every row sees whole),
// always (tiles that reach past some row's causal limit), or at run time
// when `masked` is set; a fully masked row gives p = 0.
// Requires scale_log2 > 0 (the row maximum is taken before scaling).
constexpr float kLazyLog2 = 8.f;
// Growth of a row's maximum (log2 domain) that makes the multi-block kernel
// restart an item (it never rescales O in place).
constexpr float kRestartLog2 = 64.f;
enum { kMaskNever = 0, kMaskAlways = 1, kMaskRuntime = 2 };

__device__ __forceinline__ float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }

// max over the four 16-lane groups of a wave (lanes l, l^16, l^32, l^48),
// with the gfx950 lane-swap moves (VALU, no LDS round trip).
__device__ __forceinline__ float max_over_lane_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

// The phases of folding one 32-key tile into the running state of a wave's
// rows.  TREE = false promises chain rows, whose test is one comparison with
// the row's last visible key lim (-1: nothing visible); pend and anc are then
// unused.

// Scores of the tile (masked per MK) and each row's scaled tile maximum;
// returns whether some row's maximum exceeds its reference by more than
// kLazyLog2 (the same answer on every lane).
template <int RB, int MK, bool TREE>
__device__ __forceinline__ bool tile_scores(const f32x4 (&sc)[RB][2], float scale_log2, bool masked, int k0,
                                            const int (&pend)[RB], const uint64_t (&anc)[RB], const int (&lim)[RB],
                                            const float (&m)[RB], float (&raw)[RB][8], float (&mx)[RB],
                                            float thr = kLazyLog2) {
  const int lg = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) raw[rb][kb * 4 + e] = sc[rb][kb][e];
  if (MK == kMaskAlways || (MK == kMaskRuntime && masked)) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = k0 + kb * 16 + lg * 4 + e;
          if (TREE ? !key_visible(key, pend[rb], anc[rb]) : key > lim[rb]) raw[rb][kb * 4 + e] = -INFINITY;
        }
  }
  bool grow = false;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float* r = raw[rb];
    float t = fmaxf(fmaxf(fmaxf(r[0], r[1]), r[2]), fmaxf(fmaxf(r[3], r[4]), r[5]));
    t = fmaxf(t, fmaxf(r[6], r[7]));
    mx[rb] = max_over_lane_groups(t) * scale_log2;
    grow |= mx[rb] > m[rb] + thr;
  }
  return __ballot(grow) != 0;
}

// Move each row's reference maximum to its new maximum and rescale its sum
// and O (alpha = 1 for rows whose maximum did not grow).
template <int RB, int DB>
__device__ __forceinline__ void tile_rescale(const float (&mx)[RB], float (&m)[RB], float (&lsum)[RB],
                                             f32x4 (&o)[RB][DB]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float mn = fmaxf(m[rb], mx[rb]);
    const float alpha = exp2_raw(m[rb] - mn);
    m[rb] = mn;
    lsum[rb] *= alpha;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
  }
}

// p = 2^(s*scale - m) rounded to bfloat16 (the P fragments, B operand of
// O^T += V^T P^T); the rounded p of the lane's keys are added to lsum, so
// the normaliser matches the weights O accumulates.
template <int RB>
__device__ __forceinline__ void tile_probs(const float (&raw)[RB][8], float scale_log2, const float (&m)[RB],
                                           float (&lsum)[RB], bf16x8 (&pf)[RB]) {
  const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float mneg = -m[rb];
    float acc = lsum[rb];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const f32x2 x = {exp2_raw(fmaf(raw[rb][e], scale_log2, mneg)), exp2_raw(fmaf(raw[rb][e + 1], scale_log2, mneg))};
      const bf16x2 pb = __builtin_convertvector(x, bf16x2);
      pf[rb][e] = pb[0];
      pf[rb][e + 1] = pb[1];
      acc = __builtin_amdgcn_fdot2_f32_bf16(pb, ones, acc, false);
    }
    lsum[rb] = acc;
  }
}

// Staging layout of a 32-key tile of K or V in LDS.  The tile is split into
// 1 KB blocks n = q * kHalves + h: keys 8q .. 8q + 7 of the tile, bytes
// 128h .. 128h + 127 of each key row (one 128-byte line per row).  A wave
// fills a block with one 16-byte load (or DMA) per lane, lane l bringing a
// 16-byte unit of row l / 8, so every load instruction reads eight whole
// cache lines.  In the block, row r sits at byte 128r and its unit u at slot
// (u + rot) mod 8:
//   K: rot = r + (q & 1), so the 16 keys one fragment read touches (two
//      blocks, one unit each) fall on 16 distinct 16-byte bank groups;
//   V: rot = r & ~1, which keeps the two units of a 32-byte column block
//      adjacent, and the 8 rows one half-wave of the transposing read
//      ds_read_b64_tr_b16 touches (32 bytes each) cover all 256 bytes of
//      the bank space once.
// The per-lane offsets below depend on the lane and at most two bits of
// the block or fragment index, so loads and reads take a few fixed per-lane
// registers plus scalar or immediate offsets.
template <int D>
struct Tile {
  static constexpr int kRow = D * 2;            // bytes per key row
  static constexpr int kHalves = D / 64;        // 128-byte half rows per row
  static constexpr int kBlocks = 4 * kHalves;   // blocks per tile of K (or V)
  static constexpr int kBytes = kBlocks * 1024;
  static_assert(kBytes == kTile * kRow, "a tile is 32 rows");
  // Global byte offset of block n in the tile.
  __device__ static constexpr int block_global(int n) { return (n / kHalves) * 8 * kRow + (n % kHalves) * 128; }
  // Global byte offset (from block_global) of the unit lane l loads for a
  // K block with q & 1 == qodd, and for any V block.
  __device__ static uint32_t k_load(int l, int qodd) {
    const int r = l >> 3;
    return r * kRow + (((l & 7) - r - qodd) & 7) * 16;
  }
  __device__ static uint32_t v_load(int l) {
    const int r = l >> 3;
    return r * kRow + (((l & 7) - (r & ~1)) & 7) * 16;
  }
  // The same with the row clamped to the tile's last existing row `last`
  // (global offset from the tile start).
  __device__ static uint32_t k_load_clamped(int l, int n, int last) {
    const int q = n / kHalves, r = l >> 3;
    return min(8 * q + r, last) * kRow + (n % kHalves) * 128 + (((l & 7) - r - (q & 1)) & 7) * 16;
  }
  __device__ static uint32_t v_load_clamped(int l, int n, int last) {
    const int q = n / kHalves, r = l >> 3;
    return min(8 * q + r, last) * kRow + (n % kHalves) * 128 + (((l & 7) - (r & ~1)) & 7) * 16;
  }
  // K fragment (16-key block kb, 32-wide step ds) of lane (lg, lr): key
  // 16kb + lr, elements 32ds + 8lg .. +8.  LDS offset = k_read(lane, ds & 1)
  // + k_read_imm(kb, ds).
  __device__ static uint32_t k_read(int lane, int dsodd) {
    const int lg = lane >> 4, lr = lane & 15, r = lr & 7, qodd = lr >> 3;
    return qodd * kHalves * 1024 + r * 128 + ((4 * dsodd + lg + r + qodd) & 7) * 16;
  }
  __device__ static constexpr int k_read_imm(int kb, int ds) { return kb * 2 * kHalves * 1024 + (ds / 2) * 1024; }
  // Transposing read of V for output block db and key half hk: lane (lg, j)
  // addresses key 16hk + 4lg + j/4, elements 16db + 4(j%4) .. +3.  LDS
  // offset = v_read(lane, db % 4) + v_read_imm(db, hk).
  __device__ static uint32_t v_read(int lane, int dbm) {
    const int lg = lane >> 4, j = lane & 15, r = 4 * (lg & 1) + (j >> 2);
    return (lg >> 1) * kHalves * 1024 + r * 128 + ((2 * dbm + ((j >> 1) & 1) + (r & ~1)) & 7) * 16 + 8 * (j & 1);
  }
  __device__ static constexpr int v_read_imm(int db, int hk) { return hk * 2 * kHalves * 1024 + (db / 4) * 1024; }
};

// Per-lane offsets of the staging layout, computed once per wave.
template <int D>
struct TileLane {
  uint32_t kload[2], vload, kread[2], vread[4];
  __device__ explicit TileLane(int lane) {
    using T = Tile<D>;
    kload[0] = T::k_load(lane, 0);
    kload[1] = T::k_load(lane, 1);
    vload = T::v_load(lane);
    kread[0] = T::k_read(lane, 0);
    kread[1] = T::k_read(lane, 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) vread[i] = T::v_read(lane, i);
  }
};

// LDS DMA of one 1 KB block: lane l copies the 16 bytes at gbase + voff into
// LDS bytes lds + 16l .. +15.  gbase and lds are wave-uniform (scalar
// registers).  Issued from inline assembly, so the compiler neither tracks it
// nor inserts waits for it: the kernel's own vmcnt waits order it against the
// LDS reads.  It sets M0 itself, so the kernel uses M0 for nothing else.  The
// load carries the nontemporal hint (every row is read once).
// Both scalars pass through readfirstlane (free when the compiler already
// holds them in scalar registers), since the instruction takes them only
// from scalar registers.
__device__ __forceinline__ void dma_block(uint32_t lds, const void* gbase, uint32_t voff) {
  const uint64_t g = (uint64_t)(uintptr_t)gbase;
  const uint64_t gu = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(g >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)g);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"((const void*)(uintptr_t)gu)
               : "memory");
}

// DMA of blocks N0 .. N1-1 of one tile's K (ISV false) or V rows at t into
// the wave's LDS stage at l; `last` as for dma_tile.
template <int D, bool ISV, int N0, int N1>
__device__ __forceinline__ void dma_tile_part(const uint16_t* t, uint32_t l, const TileLane<D>& tl, int last) {
  using T = Tile<D>;
  const int lane = threadIdx.x & 63;
  const char* b = reinterpret_cast<const char*>(t);
  if (last >= kTile - 1) {
#pragma unroll
    for (int n = N0; n < N1; ++n)
      dma_block(l + n * 1024, b + T::block_global(n), ISV ? tl.vload : tl.kload[(n / T::kHalves) & 1]);
  } else {
#pragma unroll
    for (int n = N0; n < N1; ++n)
      dma_block(l + n * 1024, b, ISV ? T::v_load_clamped(lane, n, last) : T::k_load_clamped(lane, n, last));
  }
}

// DMA of one tile (rows at kt / vt) into the wave's LDS stage (kl / vl);
// `last` >= 31 when every row of the tile exists, else its last row.
template <int D>
__device__ __forceinline__ void dma_tile(const uint16_t* kt, const uint16_t* vt, uint32_t kl, uint32_t vl,
                                         const TileLane<D>& tl, int last) {
  using T = Tile<D>;
  const int lane = threadIdx.x & 63;
  const char* kb = reinterpret_cast<const char*>(kt);
  const char* vb = reinterpret_cast<const char*>(vt);
  if (last >= kTile - 1) {
#pragma unroll
    for (int n = 0; n < T::kBlocks; ++n) {
      dma_block(kl + n * 1024, kb + T::block_global(n), tl.kload[(n / T::kHalves) & 1]);
      dma_block(vl + n * 1024, vb + T::block_global(n), tl.vload);
    }
  } else {
#pragma unroll
    for (int n = 0; n < T::kBlocks; ++n) {
      dma_block(kl + n * 1024, kb, T::k_load_clamped(lane, n, last));
      dma_block(vl + n * 1024, vb, T::v_load_clamped(lane, n, last));
    }
  }
}

// Where the K and V rows of one (request, KV head) live.  Contiguous: the
// request's segment [Hkv][L][D] at kv_off.  Paged: pages [num_pages][Hkv][P][D]
// (P = 2^shift keys) named by the request's block table; each wave loads the
// page ids of its chunk once (lane j: the chunk's page j) and reads them back
// per tile with readlane.  A 32-key tile never crosses a page (P is a multiple
// of 32), so tile(k0) + (key - k0) * D addresses every key of the tile.
template <int D, bool PAGED>
struct KVSrc {
  const uint16_t* k;
  const uint16_t* v;
  int64_t page_elems = 0;  // paged: Hkv * P * D
  int64_t head_off = 0;    // paged: g * P * D
  int shift = 0, page0 = 0, ids = 0;
  __device__ int64_t tile(int k0) const {
    if (!PAGED) return (int64_t)k0 * D;
    const int page = __builtin_amdgcn_readlane(ids, (k0 >> shift) - page0);
    return (int64_t)page * page_elems + head_off + (int64_t)(k0 & ((1 << shift) - 1)) * D;
  }
};

// The rows of (request b of the launch, KV head g) for the item whose chunk
// starts at key k_begin (a multiple of the page size when paged).
template <int D, bool PAGED>
__device__ __forceinline__ KVSrc<D, PAGED> kv_src(const AttnShape& s, const AttnBatch& bt, const uint16_t* kp,
                                                  const uint16_t* vp, int b, int g, int L, int k_begin) {
  KVSrc<D, PAGED> src;
  if (!PAGED) {
    const int64_t base = bt.kv_off[b] + (int64_t)g * L * D;
    src.k = kp + base;
    src.v = vp + base;
    return src;
  }
  src.k = kp;
  src.v = vp;
  src.shift = bt.page_shift;
  src.page0 = k_begin >> bt.page_shift;
  src.page_elems = ((int64_t)s.Hkv << bt.page_shift) * D;
  src.head_off = ((int64_t)g << bt.page_shift) * D;
  const int npages = (L + (1 << bt.page_shift) - 1) >> bt.page_shift;
  const int j = min(src.page0 + (int)(threadIdx.x & 63), npages - 1);
  const int id = bt.pages[(int64_t)(bt.req0 + b) * bt.max_pages + j];
  src.ids = min(max(id, 0), bt.num_pages - 1);
  return src;
}

// Per-wave running state of the online softmax over its query rows.
template <int RB, int D>
struct AttnRows {
  bf16x8 qf[RB][D / 32];  // Q fragments, B operand of S^T = K Q^T
  int pend[RB];           // last visible prefix key of the lane's row (-1: padding row)
  uint64_t anc[RB];       // visible tail positions of the lane's row
  int lim[RB];            // chain rows: last visible key (-1: padding row)
  float m[RB], lsum[RB];  // running maximum (log2 domain) and sum
  f32x4 o[RB][D / 16];    // running O^T blocks
};

// S^T = K Q^T for the tile's 32 keys (K fragments kf) and the wave's rows.
template <int RB, int D>
__device__ __forceinline__ void tile_qk(const AttnRows<RB, D>& st, const bf16x8 (&kf)[2][D / 32], f32x4 (&sc)[RB][2]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < D / 32; ++ds) acc = mfma16x16x32(kf[kb][ds], st.qf[rb][ds], acc);
      sc[rb][kb] = acc;
    }
}

// O^T += V^T P^T with V staged at vsrc.  V^T fragments (A operand): lane
// (lg, lr) receives d = db*16 + lr and keys {lg*4 .. +3} (first half),
// {16 + lg*4 .. +3} (second half), the P fragment's k-slots.
// V^T fragments (A operand of O^T += V^T P^T) of a tile staged in LDS:
// vf[db] of lane (lg, lr) holds d = db*16 + lr and keys {lg*4 .. +3}, then
// {16 + lg*4 .. +3}, the P fragment's k-slots.
template <int D>
__device__ __forceinline__ void read_v_frags(const unsigned char* __restrict__ vsrc, const TileLane<D>& tl,
                                             bf16x8 (&vf)[D / 16]) {
  using T = Tile<D>;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const s16x4 lo = lds_read_tr16(vsrc + tl.vread[db & 3] + T::v_read_imm(db, 0));
    const s16x4 hi = lds_read_tr16(vsrc + tl.vread[db & 3] + T::v_read_imm(db, 1));
    vf[db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }
}

// O^T += V^T P^T.
template <int RB, int D>
__device__ __forceinline__ void tile_pv(AttnRows<RB, D>& st, const bf16x8 (&pf)[RB], const bf16x8 (&vf)[D / 16]) {
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) st.o[rb][db] = mfma16x16x32(vf[db], pf[rb], st.o[rb][db]);
}

// Fold one 32-key tile (keys from k0; K fragments kf, V staged at vsrc)
// into the running state, the rescale inline.  `masked` says whether some
// key of the tile may lie past a row's causal limit (used when MK is
// kMaskRuntime); a tile with live == false contributes nothing.
// attn_fold's hook, run between the scores and the probabilities: the
// register-staged kernel issues the next tile's V loads there.
struct NoHook {
  __device__ void operator()() const {}
};
template <int RB, int D, bool TREE, int MK, typename Hook = NoHook>
__device__ __forceinline__ void attn_fold(AttnRows<RB, D>& st, float scale_log2, int k0, bool masked,
                                          const bf16x8 (&kf)[2][D / 32], const unsigned char* __restrict__ vsrc,
                                          const TileLane<D>& tl, bool live = true, Hook mid = Hook()) {
  f32x4 sc[RB][2];
  tile_qk<RB, D>(st, kf, sc);
  float raw[RB][8], mx[RB];
  bool grow;
  if (MK == kMaskRuntime && !live) {
    // A dead tile: every key masked.
    int pend[RB], lim[RB];
    uint64_t anc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      pend[rb] = -1;
      lim[rb] = -1;
      anc[rb] = 0ull;
    }
    grow = tile_scores<RB, kMaskAlways, TREE>(sc, scale_log2, true, k0, pend, anc, lim, st.m, raw, mx);
  } else {
    grow = tile_scores<RB, MK, TREE>(sc, scale_log2, masked, k0, st.pend, st.anc, st.lim, st.m, raw, mx);
  }
  if (__builtin_expect(grow, 0)) tile_rescale<RB, D / 16>(mx, st.m, st.lsum, st.o);
  mid();
  bf16x8 pf[RB];
  tile_probs<RB>(raw, scale_log2, st.m, st.lsum, pf);
  bf16x8 vf[D / 16];
  read_v_frags<D>(vsrc, tl, vf);
  tile_pv<RB, D>(st, pf, vf);
}

// K fragments of a tile staged in LDS.
template <int D>
__device__ __forceinline__ void read_k_frags(const unsigned char* __restrict__ ksrc, const TileLane<D>& tl,
                                             bf16x8 (&kf)[2][D / 32]) {
  using T = Tile<D>;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ds = 0; ds < D / 32; ++ds)
      kf[kb][ds] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(ksrc + tl.kread[ds & 1] + T::k_read_imm(kb, ds)));
}

// Item of wave `wave` in workgroup blockIdx.x: (chunk, KV head, row group),
// row group fastest, then KV head, so the waves that split one head's rows
// share a workgroup (and read the same K and V tiles at the same time).
// Returns false past the last item.
__device__ __forceinline__ bool attn_item(const AttnShape& s, const AttnBatch& bt, int& c_local, int& g, int& rg) {
  const int item = blockIdx.x * kAttnWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pair = item / s.row_groups;
  rg = item - pair * s.row_groups;
  c_local = pair / s.Hkv;
  g = pair - c_local * s.Hkv;
  return c_local < bt.chunk_prefix[bt.nreq];
}

// Partial of one item: row r of slot (chunk_base + c_local)*Hkv + g.
template <int RB, int D>
__device__ __forceinline__ void write_partial(const AttnShape& s, const AttnBatch& bt, AttnPartials parts, int c_local,
                                              int g, const float (&m)[RB], float (&lsum)[RB],
                                              const f32x4 (&o)[RB][D / 16], int row0 = 0) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t slot = (int64_t)(bt.chunk_base + c_local) * s.Hkv + g;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    lsum[rb] += __shfl_xor(lsum[rb], 16);
    lsum[rb] += __shfl_xor(lsum[rb], 32);
    const int row = row0 + rb * 16 + lr;
    if (row < s.rows) {
      if (lg == 0) {
        parts.m[slot * s.rows + row] = m[rb];
        parts.l[slot * s.rows + row] = lsum[rb];
      }
#pragma unroll
      for (int db = 0; db < D / 16; ++db)
        *reinterpret_cast<f32x4*>(parts.o + (slot * s.rows + row) * D + db * 16 + lg * 4) = o[rb][db];
    }
  }
}

// Running state of rows row0 .. row0 + 16*RB - 1 of KV head g: Q fragments
// (B operand of S^T = K Q^T; lane holds row row0 + rb*16 + lr, d = ds*32 +
// lg*8 .. +8), causal limits, empty sums.  Rows past s.rows are padding.
template <int RB, int D>
__device__ __forceinline__ void init_rows(AttnRows<RB, D>& st, const AttnShape& s, const uint64_t* __restrict__ anc,
                                          const uint16_t* __restrict__ q, int req, int g, int L, int row0) {
  constexpr int DS = D / 32;
  constexpr int DB = D / 16;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = row0 + rb * 16 + lr;
    if (row < s.rows) {
      const int j = row / s.group;
      const int h = g * s.group + (row - j * s.group);
      const uint16_t* qrow = q + (((int64_t)req * s.G + j) * s.Hq + h) * D;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) st.qf[rb][ds] = load_bf16x8(qrow + ds * 32 + lg * 8);
      st.pend[rb] = L - s.G - 1;
      st.anc[rb] = anc != nullptr ? anc[(int64_t)req * s.G + j] : chain_mask(j);
      st.lim[rb] = L - s.G + j;
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) st.qf[rb][ds] = bf16x8{};
      st.pend[rb] = -1;
      st.anc[rb] = 0ull;
      st.lim[rb] = -1;
    }
    st.m[rb] = kNegBig;
    st.lsum[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) st.o[rb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

template <int RB, int D, bool TREE, bool PAGED>
__global__ __launch_bounds__(kAttnThreads, 1)
void attn_bf16_kernel(const AttnShape s, const AttnBatch bt, const uint16_t* __restrict__ q,
                      const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
                      AttnPartials parts) {
  using T = Tile<D>;
  constexpr int kStage = kAttnWaves * T::kBytes;  // one stage of K or V, all waves
  // Two stages of K and V tiles.
  __shared__ __align__(1024) unsigned char kst[2 * kStage];
  __shared__ __align__(1024) unsigned char vst[2 * kStage];

  int c_local, g, rg;
  if (!attn_item(s, bt, c_local, g, rg)) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;

  // The item's scalars are wave-uniform; readfirstlane lets the compiler
  // keep them (and the loop control and tile pointers built from them) in
  // scalar registers.
  const int b = __builtin_amdgcn_readfirstlane(find_request(bt, c_local));
  const int L = __builtin_amdgcn_readfirstlane(bt.kv_len[b]);
  const int req = bt.req0 + b;
  const int k_begin = __builtin_amdgcn_readfirstlane((c_local - bt.chunk_prefix[b]) * s.chunk_keys);
  const int k_end = min(L, k_begin + s.chunk_keys);
  const KVSrc<D, PAGED> src = kv_src<D, PAGED>(s, bt, kp, vp, b, g, L, k_begin);

  AttnRows<RB, D> st;
  const int row0 = __builtin_amdgcn_readfirstlane(rg * RB * 16);
  init_rows<RB, D>(st, s, bt.anc, q, req, g, L, row0);

  // Tile i of the item starts at key k_begin + 32i and is staged in stage
  // i & 1; tile i + 1 loads while tile i is folded in, its DMAs spread over
  // the fold in four groups (half the K blocks after the K fragments are
  // read, the other half after S = K Q^T, half the V blocks after the
  // scores, the rest after the probabilities).  A wave that issued all of a
  // tile's DMAs at once stalled at issue while the CU's queue of line misses
  // was full and then left the queue idle while it computed; spread out, the
  // same requests keep the queue fuller (70B-shaped share: 287 -> 260 us).
  // (Loading two tiles ahead, with the fragments moved to registers first to
  // free the stage, measured slower.)  Every row sees every key up to L - G (the root's
  // position), so the tiles that end there or before take no mask; the rest
  // (the last few tiles of the request's last chunk, including a partial tile
  // reaching past L - 1, whose missing rows repeat row L - 1 and are masked)
  // do.
  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  const int nplain = min(ntiles, max(0, (L - s.G + 1 - k_begin) / kTile));
  const uint32_t kl0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)kst + wave * T::kBytes;
  const uint32_t vl0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)vst + wave * T::kBytes;
  const TileLane<D> tl(lane);
  auto issue = [&](int i) {
    const int k0 = k_begin + i * kTile;
    const int64_t t = src.tile(k0);
    const uint32_t so = (uint32_t)(i & 1) * kStage;
    dma_tile<D>(src.k + t, src.v + t, kl0 + so, vl0 + so, tl, L - 1 - k0);
  };
  // The reference maxima never move by a rescale of O here (a rescale branch
  // in this loop made the compiler copy O between register files on every
  // tile).  The first tile sets them (nothing is accumulated yet); after
  // that p = 2^(s*scale - m) may exceed 1 by up to 2^kRestartLog2, far inside
  // float32 range for O and the sums.  A row whose maximum grows beyond that
  // restarts the item from its first tile with the grown maxima and O, sums
  // cleared.  Each restart raises a reference by more than kRestartLog2, so
  // restarts are finitely many (none for scores of any ordinary range).
  for (;;) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      st.lsum[rb] = 0.f;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) st.o[rb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    issue(0);
    bool fresh = true, restart = false;
    constexpr int kB = T::kBlocks;
    for (int i = 0; i < ntiles; ++i) {
      wait_vmcnt<0>();  // tile i landed
      const bool more = i + 1 < ntiles;
      const int k0n = k_begin + (i + 1) * kTile;
      const int64_t tn = src.tile(min(k0n, k_begin + (ntiles - 1) * kTile));
      const uint32_t son = (uint32_t)((i + 1) & 1) * kStage;
      const int lastn = L - 1 - k0n;
      const int so = (i & 1) * kStage + wave * T::kBytes;
      bf16x8 kf[2][D / 32];
      read_k_frags<D>(kst + so, tl, kf);
      if (more) dma_tile_part<D, false, 0, kB / 2>(src.k + tn, kl0 + son, tl, lastn);
      f32x4 sc[RB][2];
      tile_qk<RB, D>(st, kf, sc);
      if (more) dma_tile_part<D, false, kB / 2, kB>(src.k + tn, kl0 + son, tl, lastn);
      float raw[RB][8], mx[RB];
      const bool grow = tile_scores<RB, kMaskRuntime, TREE>(sc, s.scale_log2, i >= nplain, k_begin + i * kTile,
                                                            st.pend, st.anc, st.lim, st.m, raw, mx,
                                                            fresh ? 0.f : kRestartLog2);
      if (grow) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) st.m[rb] = fmaxf(st.m[rb], mx[rb]);
        if (!fresh) {
          restart = true;
          break;
        }
      }
      fresh = false;
      if (more) dma_tile_part<D, true, 0, kB / 2>(src.v + tn, vl0 + son, tl, lastn);
      bf16x8 pf[RB], vf[D / 16];
      tile_probs<RB>(raw, s.scale_log2, st.m, st.lsum, pf);
      read_v_frags<D>(vst + so, tl, vf);
      if (more) dma_tile_part<D, true, kB / 2, kB>(src.v + tn, vl0 + son, tl, lastn);
      tile_pv<RB, D>(st, pf, vf);
    }
    if (!restart) break;
    wait_vmcnt<0>();  // the tile after the one that restarted may still be in flight
  }
  write_partial<RB, D>(s, bt, parts, c_local, g, st.m, st.lsum, st.o, row0);
}

// Register-staged variant: K and V blocks go HBM -> registers -> the wave's
// LDS tiles in the staging layout -> MFMA fragments.  All loads land in
// registers, so the compiler's own vmcnt accounting covers the pipeline.  The
// next tile's K loads go out before a tile is folded and its V loads in the
// middle of the fold, which keeps the CU's queue of line misses fuller than
// issuing both at once (vicuna7b: 24.0 -> 23.5 us).  With one 16-row block
// (multi-head attention) two workgroups share a CU.
template <int RB, int D, bool TREE, bool PAGED>
__global__ __launch_bounds__(kAttnThreads, (RB == 1 ? 2 : 1))
void attn_bf16_reg_kernel(const AttnShape s, const AttnBatch bt, const uint16_t* __restrict__ q,
                          const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
                          AttnPartials parts) {
  using T = Tile<D>;
  constexpr int NB = T::kBlocks;
  __shared__ __align__(1024) unsigned char ksm[kAttnWaves * T::kBytes];
  __shared__ __align__(1024) unsigned char vsm[kAttnWaves * T::kBytes];

  int c_local, g, rg;
  if (!attn_item(s, bt, c_local, g, rg)) return;
  (void)rg;  // a single 16-row block: one row group
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;

  // The item's scalars are wave-uniform; readfirstlane lets the compiler
  // keep them (and the loop control and tile pointers built from them) in
  // scalar registers.
  const int b = __builtin_amdgcn_readfirstlane(find_request(bt, c_local));
  const int L = __builtin_amdgcn_readfirstlane(bt.kv_len[b]);
  const int req = bt.req0 + b;
  const int k_begin = __builtin_amdgcn_readfirstlane((c_local - bt.chunk_prefix[b]) * s.chunk_keys);
  const int k_end = min(L, k_begin + s.chunk_keys);
  const KVSrc<D, PAGED> src = kv_src<D, PAGED>(s, bt, kp, vp, b, g, L, k_begin);

  AttnRows<RB, D> st;
  init_rows<RB, D>(st, s, bt.anc, q, req, g, L, 0);

  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  unsigned char* kt = ksm + wave * T::kBytes;
  unsigned char* vt = vsm + wave * T::kBytes;
  auto key0 = [&](int i) { return k_begin + min(i, ntiles - 1) * kTile; };
  const TileLane<D> tl(lane);

  // Blocks of two tiles, streamed with the nontemporal hint (every row is
  // read once).  A dead tile (past the item's last) has every lane read the
  // tile's first 16 bytes (one cache line per load); rows past L - 1 repeat
  // row L - 1.
  u32x4 kr[2][NB], vr[2][NB];
  auto issue_part = [&](int set, int i, bool isv) {
    const int k0 = key0(i);
    const bool dead = i >= ntiles;
    const int last = L - 1 - k0;
    const char* base = reinterpret_cast<const char*>((isv ? src.v : src.k) + src.tile(k0));
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const uint32_t kvo = isv ? (last >= kTile - 1 ? T::block_global(n) + tl.vload : T::v_load_clamped(lane, n, last))
                               : (last >= kTile - 1 ? T::block_global(n) + tl.kload[(n / T::kHalves) & 1]
                                                    : T::k_load_clamped(lane, n, last));
      const uint32_t o = dead ? 0u : kvo;
      if (isv)
        vr[set][n] = load_u32x4_stream(base + o);
      else
        kr[set][n] = load_u32x4_stream(base + o);
    }
  };
  // Fold tile (set, k0) into the running state; live == false masks it.
  // The V loads of the next tile (set nset, tile inext) go out in the middle.
  auto fold = [&](int set, int k0, bool live, int nset, int inext) {
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      *reinterpret_cast<u32x4*>(kt + n * 1024 + lane * 16) = kr[set][n];
      *reinterpret_cast<u32x4*>(vt + n * 1024 + lane * 16) = vr[set][n];
    }
    bf16x8 kf[2][D / 32];
    read_k_frags<D>(kt, tl, kf);
    attn_fold<RB, D, TREE, kMaskRuntime>(st, s.scale_log2, k0, k0 + kTile - 1 > L - s.G, kf, vt, tl, live,
                                         [&]() {
                                           __builtin_amdgcn_sched_barrier(0);
                                           issue_part(nset, inext, true);
                                           __builtin_amdgcn_sched_barrier(0);
                                         });
  };

  // Tile i+1 loads while tile i is folded in (K before, V in the middle);
  // the body always folds two tiles (the second masked when the count is
  // odd), so no branch separates a load from its use.
  issue_part(0, 0, false);
  issue_part(0, 0, true);
  for (int i = 0; i < ntiles; i += 2) {
    issue_part(1, i + 1, false);
    __builtin_amdgcn_sched_barrier(0);  // keep the next tile's loads ahead of this tile's work
    fold(0, key0(i), true, 1, i + 1);
    issue_part(0, i + 2, false);
    __builtin_amdgcn_sched_barrier(0);
    fold(1, key0(i + 1), i + 1 < ntiles, 0, i + 2);
  }
  write_partial<RB, D>(s, bt, parts, c_local, g, st.m, st.lsum, st.o);
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
    const int j = row / s.group;
    const uint64_t anc = bt.anc != nullptr ? bt.anc[(int64_t)req * s.G + j] : chain_mask(j);
    ps[row * C + kk] = key_visible(key, L - s.G - 1, anc) ? acc * s.scale_log2 : -INFINITY;
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

// Standalone merge: grid (requests, KV heads, combine blocks per pair).
template <typename OutT>
__global__ __launch_bounds__(kCombineThreads)
void attn_combine_kernel(const AttnShape s, const AttnBatch bt, AttnPartials parts, OutT* __restrict__ out) {
  combine_block<OutT>(s, bt, parts, out, blockIdx.x, blockIdx.y, blockIdx.z, threadIdx.x);
}

template <int RB, int D, bool TREE, bool PAGED>
hipError_t launch_bf16(const AttnShape& s, const AttnBatch& bt, int nchunks, const void* q, const void* k,
                       const void* v, AttnPartials parts, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  const int items = nchunks * s.Hkv * s.row_groups;
  hipExtLaunchKernelGGL((attn_bf16_kernel<RB, D, TREE, PAGED>), dim3((items + kAttnWaves - 1) / kAttnWaves), dim3(kAttnThreads), 0,
                        stream, e0, e1, 0, s, bt, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                        static_cast<const uint16_t*>(v), parts);
  return hipGetLastError();
}

template <int RB, int D, bool TREE, bool PAGED>
hipError_t launch_reg(const AttnShape& s, const AttnBatch& bt, int nchunks, const void* q, const void* k,
                      const void* v, AttnPartials parts, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  hipExtLaunchKernelGGL((attn_bf16_reg_kernel<RB, D, TREE, PAGED>), dim3((nchunks * s.Hkv + kAttnWaves - 1) / kAttnWaves),
                        dim3(kAttnThreads), 0, stream, e0, e1, 0, s, bt, static_cast<const uint16_t*>(q),
                        static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), parts);
  return hipGetLastError();
}

template <int D, bool TREE, bool PAGED>
hipError_t dispatch_rb(int rb, const AttnShape& s, const AttnBatch& bt, int nchunks, const void* q, const void* k,
                       const void* v, AttnPartials parts, hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  switch (rb) {
    case 1: return launch_reg<1, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 2: return launch_bf16<2, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 3: return launch_bf16<3, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 4: return launch_bf16<4, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 5: return launch_bf16<5, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    default: break;
  }
  // Six to eight blocks per wave only at head dimension 64 (at 128 the rows
  // split over row groups first).
  if constexpr (D == 64) {
    switch (rb) {
      case 6: return launch_bf16<6, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
      case 7: return launch_bf16<7, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
      case 8: return launch_bf16<8, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

// Tree commit: move the K and V rows of request b's accepted nodes (tail
// positions out_node[j] + 1, increasing in j) to positions j + 1 after the
// root, in place.  Every thread moves one 16-byte piece of one (KV head, row)
// for all j in increasing order; since out_node[j] + 1 >= j + 1 and the
// sources increase with j, no source is overwritten before it is read.
// Accept lengths and node numbers outside their ranges end the move (every
// access stays inside the request's cache).  Grid (requests, Hkv).
__global__ __launch_bounds__(kAttnThreads)
void tree_commit_kernel(CommitBatch cb, int G, int D, int esz, const int32_t* __restrict__ out_node,
                        const int32_t* __restrict__ accept_len, unsigned char* __restrict__ kp,
                        unsigned char* __restrict__ vp) {
  const int b = blockIdx.x;
  const int req = cb.req0 + b;
  const int g = blockIdx.y;
  const int L = cb.kv_len[b];
  const int l = min(max(accept_len[req], 0), G - 1);
  const int row_bytes = D * esz;
  const int pieces = row_bytes / 16;
  const int64_t head0 = (cb.kv_off[b] + (int64_t)g * L * D) * esz;  // byte offset of the head's row 0
  const int tail0 = L - G;
  for (int t = threadIdx.x; t < 2 * pieces; t += blockDim.x) {
    unsigned char* base = (t < pieces ? kp : vp) + head0 + (t % pieces) * 16;
    for (int j = 0; j < l; ++j) {
      const int n = out_node[(int64_t)req * G + j];
      if (n < j || n >= G - 1) break;
      const int src = tail0 + n + 1;
      const int dst = tail0 + j + 1;
      if (src != dst) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(base + (int64_t)src * row_bytes);
        *reinterpret_cast<u32x4*>(base + (int64_t)dst * row_bytes) = v;
      }
    }
  }
}

// One workgroup per request, one thread per position: walk up the parents
// (each step moves to a strictly smaller position, so at most g steps).
__global__ __launch_bounds__(kWave)
void tree_masks_kernel(int N, const int32_t* __restrict__ parent, uint64_t* __restrict__ masks) {
  const int b = blockIdx.x;
  const int G = N + 1;
  for (int g = threadIdx.x; g < G; g += kWave) {
    uint64_t m = 1ull;
    int pos = g;
    while (pos > 0) {
      m |= 1ull << pos;
      const int pp = parent[(int64_t)b * N + pos - 1];
      pos = (pp >= -1 && pp < pos - 1) ? pp + 1 : 0;
    }
    masks[(int64_t)b * G + g] = m;
  }
}

}  // namespace

int attn_row_groups(int dtype, int rows, int D) {
  const int rb = (rows + 15) / 16;
  if (dtype == 0 || D != 128 || rb <= kMaxRowBlocks) return 1;
  return (rb + kMaxRowBlocks - 1) / kMaxRowBlocks;
}

int attn_chunk_keys(int dtype, int rows, int row_groups, int Hkv, const int32_t* kv_len, int B) {
  if (dtype == 0) return kF32ChunkKeys;
  int64_t total_keys = 0;
  if (kv_len != nullptr)
    for (int b = 0; b < B; ++b) total_keys += kv_len[b];
  // A whole number of 32-key tiles; never so short that an item's start-up
  // (query rows, first tile) outweighs its streaming.
  const int64_t target = rows <= 16 ? kAttnTargetItemsOne : kAttnTargetItemsMany;
  const int64_t per = (total_keys * Hkv + target - 1) / target;
  const int64_t c = (per + kTile - 1) / kTile * kTile;
  const int def = (int)std::min<int64_t>(kMaxChunkKeys, std::max<int64_t>(kMinChunkKeys, c));
  if (rows <= 16 && kv_len != nullptr) {
    for (int r = kRoundMinKeys; r < def; r += kTile) {
      int64_t items = 0;
      for (int b = 0; b < B; ++b) items += (kv_len[b] + r - 1) / r;
      if ((items * Hkv + kAttnWaves - 1) / kAttnWaves <= kRoundWorkgroups) return r;
    }
  }
  if (rows > 16 && kv_len != nullptr) {
    // The multi-block kernel runs one workgroup (four near-equal items) per
    // CU, so a launch takes ceil(workgroups / CUs) rounds of one item each:
    // a chunk count just past a multiple of the CU count leaves most CUs idle
    // in the last round.  Among chunks at least as long as the default (so
    // the workspace bound still holds), take the one with the shortest
    // rounds * (chunk + per-item start-up) estimate.
    const int64_t cus = device_cu_count();
    int best = def;
    int64_t best_t = INT64_MAX;
    for (int c2 = def; c2 <= kMaxChunkKeys; c2 += kTile) {
      int64_t chunks = 0;
      for (int b = 0; b < B; ++b) chunks += (kv_len[b] + c2 - 1) / c2;
      const int64_t wgs = (chunks * Hkv * row_groups + kAttnWaves - 1) / kAttnWaves;
      const int64_t t = (wgs + cus - 1) / cus * (c2 + kItemStartKeys);
      if (t < best_t) {
        best_t = t;
        best = c2;
      }
    }
    return best;
  }
  return def;
}

int64_t attn_max_chunks(int dtype, int Hkv, int B, int64_t max_kv_len) {
  if (dtype == 0) return (int64_t)B * ((max_kv_len + kF32ChunkKeys - 1) / kF32ChunkKeys);
  // chunks = sum_b ceil(L_b / C) <= sum(L)/C + B, with C >= sum(L)*Hkv/target
  // unless C is capped at kMaxChunkKeys, and never more than with C at its floor.
  const int64_t by_floor = (int64_t)B * ((max_kv_len + kRoundMinKeys - 1) / kRoundMinKeys);
  const int64_t target = std::max(kAttnTargetItemsOne, kAttnTargetItemsMany);
  const int64_t by_target = std::max<int64_t>((target + Hkv - 1) / Hkv,
                                              (int64_t)B * ((max_kv_len + kMaxChunkKeys - 1) / kMaxChunkKeys)) + B;
  return std::min(by_floor, by_target);
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
    if (bt.pages != nullptr) return hipErrorInvalidValue;  // paged caches are bf16 only
    const size_t shm = sizeof(float) * static_cast<size_t>(s.rows) * (s.D + s.chunk_keys);
    hipExtLaunchKernelGGL(attn_f32_kernel, dim3(nchunks, s.Hkv), dim3(kAttnThreads), shm, stream, e0, e1, 0, s, bt,
                          static_cast<const float*>(q), static_cast<const float*>(k),
                          static_cast<const float*>(v), parts);
    return hipGetLastError();
  }
  // 16-row blocks per wave: a KV head's blocks split over its row groups.
  const int rb = ((s.rows + 15) / 16 + s.row_groups - 1) / s.row_groups;
  // Mask kinds: chain or tree; cache layouts: segments or pages (chain only).
  const bool tree = bt.anc != nullptr;
  const bool paged = bt.pages != nullptr;
  if (tree && paged) return hipErrorInvalidValue;
  if (s.D == 128) {
    if (paged) return dispatch_rb<128, false, true>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    return tree ? dispatch_rb<128, true, false>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1)
                : dispatch_rb<128, false, false>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
  }
  if (s.D == 64) {
    if (paged) return dispatch_rb<64, false, true>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    return tree ? dispatch_rb<64, true, false>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1)
                : dispatch_rb<64, false, false>(rb, s, bt, nchunks, q, k, v, parts, stream, e0, e1);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention_combine(int dtype, const AttnShape& s, const AttnBatch& bt,
                                    AttnPartials parts, void* out, hipStream_t stream) {
  if (bt.nreq <= 0) return hipSuccess;
  const dim3 grid(bt.nreq, s.Hkv, combine_zblocks(s));
  if (dtype == 0)
    hipLaunchKernelGGL(attn_combine_kernel<float>, grid, dim3(kCombineThreads), 0, stream, s, bt, parts,
                       static_cast<float*>(out));
  else
    hipLaunchKernelGGL(attn_combine_kernel<uint16_t>, grid, dim3(kCombineThreads), 0, stream, s, bt, parts,
                       static_cast<uint16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_tree_masks(int B, int N, const int32_t* parent, uint64_t* masks, hipStream_t stream) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(tree_masks_kernel, dim3(B), dim3(kWave), 0, stream, N, parent, masks);
  return hipGetLastError();
}

hipError_t launch_tree_commit(const CommitBatch& cb, int Hkv, int G, int D, int esz, const int32_t* out_node,
                              const int32_t* accept_len, void* k_pool, void* v_pool, hipStream_t stream) {
  if (cb.nreq <= 0) return hipSuccess;
  hipLaunchKernelGGL(tree_commit_kernel, dim3(cb.nreq, Hkv), dim3(kAttnThreads), 0, stream, cb, G, D, esz, out_node,
                     accept_len, static_cast<unsigned char*>(k_pool), static_cast<unsigned char*>(v_pool));
  return hipGetLastError();
}

}  // namespace sdv
