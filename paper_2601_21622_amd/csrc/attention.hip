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
// another.  The host picks the chunk length from the total work so that the
// items fill the GPU about twice over.  Two bf16 kernels:
//   * one 16-row block (multi-head attention: the G queries of one head):
//     each wave loads the next 32-key tile's K fragments and V rows into its
//     other register set while it folds in the current tile; V goes through a
//     wave-private LDS tile so that the transposing read ds_read_b64_tr_b16
//     hands each lane its V^T fragment;
//   * several 16-row blocks (grouped-query attention): K and V tiles go from
//     HBM into wave-private LDS stages by DMA (no registers, completion
//     tracked with explicit vmcnt waits), again one tile ahead.
// Both compute S^T = K Q^T and O^T += V^T P^T on MFMA 16x16x32 bf16 (the Q
// fragments stay in registers, P comes straight from the S^T accumulator
// layout) with the online softmax in the log2 domain, each lane owning one
// query row (for up to two row blocks the reference maximum moves lazily, so
// most tiles skip the rescale of O).  Each item writes one partial (max, sum, O) to the workspace; a
// combine kernel merges the chunks of each request in fixed order and writes
// O in the input dtype.  LDS tiles keep rows whole but rotate their 16-byte
// pieces so that the fragment reads are free of bank conflicts.
#include <hip/hip_ext.h>

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

// Online softmax of one 16-row block over a 32-key tile, in the log2 domain:
// the lane owns row lr of the block and keys k0 + kb*16 + lg*4 + e.  With
// LAZY the reference maximum m of the rows moves lazily: only when some row's
// tile maximum exceeds it by more than kLazyLog2 does the wave move m to the
// new maxima and rescale the sums and O (rows whose maximum did not grow get
// alpha = 1).  Otherwise p = 2^(s*scale - m) stays below 2^kLazyLog2, well
// inside float32 and bfloat16 range, and O and the sum share the same m, so
// the normalised result is unchanged.  Masking (key_visible) applies only
// when `masked` (always without LAZY, which keeps the step one branch-free
// block); a fully masked row gives p = 0.
// Requires scale_log2 > 0 (the row maximum is taken before scaling).
constexpr float kLazyLog2 = 8.f;
// Up to this many row blocks the rescale branch costs nothing; with more, the
// output accumulators no longer fit beside the rest in plain registers and
// the branch makes the compiler move them every tile, so the rescale runs on
// every tile instead (alpha is 1 whenever the maximum did not grow).
constexpr int kLazyMaxBlocks = 2;

__device__ __forceinline__ float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }

// TREE = false promises chain rows, whose test is one comparison with the
// row's last visible key lim (-1: nothing visible); pend and anc are then unused.
template <int DB, bool LAZY, bool TREE>
__device__ __forceinline__ bf16x8 softmax_tile(const f32x4 (&sc)[2], float scale_log2, bool masked, int k0, int pend,
                                               uint64_t anc, int lim, float& m, float& lsum, f32x4 (&o)[DB]) {
  const int lg = (threadIdx.x & 63) >> 4;
  float raw[8];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int e = 0; e < 4; ++e) raw[kb * 4 + e] = sc[kb][e];
  if (!LAZY || masked) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (TREE ? !key_visible(k0 + kb * 16 + lg * 4 + e, pend, anc) : k0 + kb * 16 + lg * 4 + e > lim)
          raw[kb * 4 + e] = -INFINITY;
  }
  float mx = fmaxf(fmaxf(fmaxf(raw[0], raw[1]), fmaxf(raw[2], raw[3])),
                   fmaxf(fmaxf(raw[4], raw[5]), fmaxf(raw[6], raw[7])));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  mx *= scale_log2;
  if (!LAZY || __ballot(mx > m + kLazyLog2) != 0) {
    const float mn = fmaxf(m, mx);
    const float alpha = exp2_raw(m - mn);
    m = mn;
    lsum *= alpha;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] *= alpha;
  }
  const float mneg = -m;
  bf16x8 pf;
  float ps = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 pb = (__bf16)exp2_raw(fmaf(raw[e], scale_log2, mneg));
    pf[e] = pb;
    ps += (float)pb;
  }
  lsum += ps;
  return pf;
}

// K or V tile of one wave in LDS: 32 keys x D, row r (D*2 bytes) holding its
// 16-byte pieces rotated by rot(r) pieces.  K: rot(r) = r*P/16 (mod P), so a
// piece read by 16 consecutive keys hits 16 distinct bank groups.  V:
// rot(r) = 2*(r*P/16) (mod P), so the four rows a 16-lane group touches in one
// transposing read fall on distinct banks.
template <int D, bool IS_V>
struct KVTile {
  static constexpr int kPieces = D / 8;          // 16-byte pieces per row
  static constexpr int kBytes = kTile * D * 2;   // one tile
  static constexpr int kRowsPerDma = 64 / kPieces;
  static constexpr int kDmas = kTile / kRowsPerDma;  // DMA instructions per tile
  __device__ static constexpr int rot(int r) {
    return ((IS_V ? 2 : 1) * ((r * kPieces) >> 4)) % kPieces;
  }
  // Byte offset of element d of row r.
  __device__ static constexpr int at(int r, int d) {
    return r * D * 2 + (((d >> 3) + rot(r)) % kPieces) * 16 + (d & 7) * 2;
  }
  // DMA instruction i of a tile: lane l brings row r = i*kRowsPerDma +
  // l/kPieces, the global piece that belongs in LDS slot l%kPieces.  t0 is
  // key k0's row; rows past the request's last key L - 1 repeat it.  A dead
  // tile (past the item's last, issued only to keep the pipeline shape) has
  // every lane read the same 16 bytes: one cache line per instruction.
  __device__ static void load(const uint16_t* t0, int k0, int L, unsigned char* tile, int lane, bool dead = false) {
#pragma unroll
    for (int i = 0; i < kDmas; ++i) {
      const int r = i * kRowsPerDma + lane / kPieces;
      const int piece = (lane % kPieces - rot(r) + kPieces) % kPieces;
      const int key = min(k0 + r, L - 1);
      const int src = dead ? 0 : (key - k0) * D + piece * 8;
      dma_16B_to_lds_opaque(t0 + src, tile + i * 1024);
    }
  }
};

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

// Fold one staged 32-key tile (keys from k0, K in ksrc, V in vsrc) into the
// running state of a wave's rows: S^T = K Q^T, online softmax, O^T += V^T P^T.
// `masked` says whether some key of the tile may lie past a row's causal
// limit (only then are the limits applied); a tile with live == false
// contributes nothing (all of its keys are masked).
template <int RB, int D, bool TREE>
__device__ __forceinline__ void attn_fold(AttnRows<RB, D>& st, float scale_log2, int k0, bool masked,
                                          const unsigned char* __restrict__ ksrc,
                                          const unsigned char* __restrict__ vsrc, bool live = true) {
  constexpr int DS = D / 32;
  constexpr int DB = D / 16;
  using KT = KVTile<D, false>;
  using VT = KVTile<D, true>;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lg = lane >> 4;

  // K fragments (A operand): lane holds key kb*16 + lr, d = ds*32 + lg*8 .. +8.
  bf16x8 kf[2][DS];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      kf[kb][ds] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(ksrc + KT::at(kb * 16 + lr, ds * 32 + lg * 8)));
  f32x4 sc[RB][2];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) acc = mfma16x16x32(kf[kb][ds], st.qf[rb][ds], acc);
      sc[rb][kb] = acc;
    }

  bf16x8 pf[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
    pf[rb] = softmax_tile<DB, (RB <= kLazyMaxBlocks), TREE>(sc[rb], scale_log2, masked || !live, k0,
                                                            live ? st.pend[rb] : -1, live ? st.anc[rb] : 0ull,
                                                            live ? st.lim[rb] : -1, st.m[rb], st.lsum[rb], st.o[rb]);

  // V^T fragments (A operand of O^T += V^T P^T): lane (lg, lr) needs
  // d = db*16 + lr and keys {lg*4 .. +3} then {16 + lg*4 .. +3}, the
  // P fragment's k-slots.  Lane j of the 16-lane group lg points at row
  // 4*lg + j/4 (+16), d = db*16 + 4*(j%4) .. +3.
  const int jr = 4 * lg + (lr >> 2);
  const int jd = 4 * (lr & 3);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const s16x4 lo = lds_read_tr16(vsrc + VT::at(jr, db * 16 + jd));
    const s16x4 hi = lds_read_tr16(vsrc + VT::at(16 + jr, db * 16 + jd));
    const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) st.o[rb][db] = mfma16x16x32(vf, pf[rb], st.o[rb][db]);
  }
}

// One step of a wave's software pipeline: start the DMAs of the next tile
// (keys from k0_next, rows at kn / vn) into (kdst, vdst), wait until only those are in flight,
// then fold the current tile.  The stage pointers are restrict-qualified, so
// the compiler knows the new DMAs cannot write what this step reads and
// leaves the ordering to the explicit wait.
template <int RB, int D, bool TREE>
__device__ __forceinline__ void attn_step(AttnRows<RB, D>& st, float scale_log2, const uint16_t* kn,
                                          const uint16_t* vn, int L, int k0_next, bool next_dead, int k0,
                                          bool masked, unsigned char* __restrict__ kdst,
                                          unsigned char* __restrict__ vdst, const unsigned char* __restrict__ ksrc,
                                          const unsigned char* __restrict__ vsrc) {
  using KT = KVTile<D, false>;
  using VT = KVTile<D, true>;
  const int lane = threadIdx.x & 63;
  KT::load(kn, k0_next, L, kdst, lane, next_dead);
  VT::load(vn, k0_next, L, vdst, lane, next_dead);
  wait_vmcnt<KT::kDmas + VT::kDmas>();
  attn_fold<RB, D, TREE>(st, scale_log2, k0, masked, ksrc, vsrc);
}

// Item of wave `wave` in workgroup blockIdx.x: (chunk, KV head), KV head
// fastest.  Returns false past the last item.
__device__ __forceinline__ bool attn_item(const AttnShape& s, const AttnBatch& bt, int& c_local, int& g) {
  const int item = blockIdx.x * kAttnWaves + (threadIdx.x >> 6);
  c_local = item / s.Hkv;
  g = item - c_local * s.Hkv;
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
  constexpr int DS = D / 32;  // 32-wide steps of the q.k contraction
  constexpr int DB = D / 16;  // 16-wide blocks of the output
  using KT = KVTile<D, false>;
  using VT = KVTile<D, true>;
  constexpr size_t kStage = (size_t)kAttnWaves * kTile * D * 2;  // one stage of K or V, all waves
  // Two stages of K and V tiles, each its own object.
  __shared__ __align__(16) unsigned char ks0[kStage];
  __shared__ __align__(16) unsigned char ks1[kStage];
  __shared__ __align__(16) unsigned char vs0[kStage];
  __shared__ __align__(16) unsigned char vs1[kStage];

  int c_local, g;
  if (!attn_item(s, bt, c_local, g)) return;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;  // row (or column) within a 16-block
  const int lg = lane >> 4;  // lane group: k-slice of MFMA operands

  const int b = find_request(bt, c_local);
  const int L = bt.kv_len[b];
  const int req = bt.req0 + b;
  const int k_begin = (c_local - bt.chunk_prefix[b]) * s.chunk_keys;
  const int k_end = min(L, k_begin + s.chunk_keys);
  const KVSrc<D, PAGED> src = kv_src<D, PAGED>(s, bt, kp, vp, b, g, L, k_begin);

  AttnRows<RB, D> st;
  init_rows<RB, D>(st, s, bt.anc, q, req, g, L, 0);

  // Tile i of the item starts at key k_begin + 32i; the load past the last
  // tile is dead (one cache line per instruction, never folded in).  Tile i+1 loads while
  // tile i is folded in; the two stages swap after every tile.
  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  unsigned char* k0s = ks0 + wave * KT::kBytes;
  unsigned char* k1s = ks1 + wave * KT::kBytes;
  unsigned char* v0s = vs0 + wave * VT::kBytes;
  unsigned char* v1s = vs1 + wave * VT::kBytes;
  auto key0 = [&](int i) { return k_begin + min(i, ntiles - 1) * kTile; };
  const int64_t t0 = src.tile(key0(0));
  KT::load(src.k + t0, key0(0), L, k0s, lane);
  VT::load(src.v + t0, key0(0), L, v0s, lane);
  for (int i = 0; i < ntiles; ++i) {
    const int64_t tn = src.tile(key0(i + 1));
    attn_step<RB, D, TREE>(st, s.scale_log2, src.k + tn, src.v + tn, L, key0(i + 1), i + 1 >= ntiles, key0(i),
                           key0(i) + kTile - 1 > L - s.G, k1s, v1s, k0s, v0s);
    unsigned char* t = k0s;
    k0s = k1s;
    k1s = t;
    t = v0s;
    v0s = v1s;
    v1s = t;
  }
  wait_vmcnt<0>();
  write_partial<RB, D>(s, bt, parts, c_local, g, st.m, st.lsum, st.o);
}

// Register-staged variant: whole K and V rows go HBM -> registers ->
// wave-private LDS tiles (rotated rows) -> MFMA fragments.  All loads land in
// registers, so the compiler's own vmcnt accounting covers the pipeline, and
// two tiles of each wave are in flight while it folds.  With one 16-row block
// (multi-head attention) two workgroups share a CU.
template <int RB, int D, bool TREE, bool PAGED>
__global__ __launch_bounds__(kAttnThreads, (RB == 1 ? 2 : 1))
void attn_bf16_reg_kernel(const AttnShape s, const AttnBatch bt, const uint16_t* __restrict__ q,
                          const uint16_t* __restrict__ kp, const uint16_t* __restrict__ vp,
                          AttnPartials parts) {
  constexpr int LPR = D / 8;       // lanes per row (16 bytes each)
  constexpr int KPI = 64 / LPR;    // rows per wave-wide load
  constexpr int NV = kTile / KPI;  // loads of K (and of V) per tile
  using VT = KVTile<D, true>;
  using KT = KVTile<D, false>;
  __shared__ __align__(16) unsigned char vsm[kAttnWaves * VT::kBytes];
  __shared__ __align__(16) unsigned char ksm[kAttnWaves * KT::kBytes];

  int c_local, g;
  if (!attn_item(s, bt, c_local, g)) return;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;

  const int b = find_request(bt, c_local);
  const int L = bt.kv_len[b];
  const int req = bt.req0 + b;
  const int k_begin = (c_local - bt.chunk_prefix[b]) * s.chunk_keys;
  const int k_end = min(L, k_begin + s.chunk_keys);
  const KVSrc<D, PAGED> src = kv_src<D, PAGED>(s, bt, kp, vp, b, g, L, k_begin);

  AttnRows<RB, D> st;
  init_rows<RB, D>(st, s, bt.anc, q, req, g, L, 0);

  const int ntiles = (k_end - k_begin + kTile - 1) / kTile;
  unsigned char* vt = vsm + wave * VT::kBytes;
  unsigned char* kt = ksm + wave * KT::kBytes;
  auto key0 = [&](int i) { return k_begin + min(i, ntiles - 1) * kTile; };

  // Whole K and V rows, KPI rows per wave-wide load (full cache lines),
  // streamed with the nontemporal hint: every row is read once.
  u32x4 kr[2][NV], vr[2][NV];
  // A dead tile (past the item's last) has every lane read one cache line.
  auto issue = [&](int set, int i) {
    const int k0 = key0(i);
    const bool dead = i >= ntiles;
    const int64_t t = src.tile(k0);
#pragma unroll
    for (int it = 0; it < NV; ++it) {
      const int row = dead ? 0 : (min(k0 + it * KPI + lane / LPR, L - 1) - k0) * D + (lane % LPR) * 8;
      kr[set][it] = load_u32x4_stream(src.k + t + row);
      vr[set][it] = load_u32x4_stream(src.v + t + row);
    }
  };
  // Fold tile (set, k0) into the running state; live == false masks it.
  auto fold = [&](int set, int k0, bool live) {
#pragma unroll
    for (int it = 0; it < NV; ++it) {
      const int r = it * KPI + lane / LPR, d = (lane % LPR) * 8;
      *reinterpret_cast<u32x4*>(kt + KT::at(r, d)) = kr[set][it];
      *reinterpret_cast<u32x4*>(vt + VT::at(r, d)) = vr[set][it];
    }
    attn_fold<RB, D, TREE>(st, s.scale_log2, k0, k0 + kTile - 1 > L - s.G, kt, vt, live);
  };

  // Tile i+1 loads while tile i is folded in; the body always folds two
  // tiles (the second masked when the count is odd), so no branch separates
  // a load from its use.
  issue(0, 0);
  for (int i = 0; i < ntiles; i += 2) {
    issue(1, i + 1);
    __builtin_amdgcn_sched_barrier(0);  // keep the next tile's loads ahead of this tile's work
    fold(0, key0(i), true);
    issue(0, i + 2);
    __builtin_amdgcn_sched_barrier(0);
    fold(1, key0(i + 1), i + 1 < ntiles);
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
  const int items = nchunks * s.Hkv;
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
    case 6: return launch_bf16<6, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 7: return launch_bf16<7, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    case 8: return launch_bf16<8, D, TREE, PAGED>(s, bt, nchunks, q, k, v, parts, stream, e0, e1);
    default: return hipErrorInvalidValue;
  }
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

int attn_chunk_keys(int dtype, int rows, int Hkv, const int32_t* kv_len, int B) {
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
  const int rb = (s.rows + 15) / 16;
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
