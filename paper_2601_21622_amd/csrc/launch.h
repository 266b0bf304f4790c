// Host-side launchers of the verification kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sdv {

// Requests handled by one attention / acceptance launch.  Their per-request
// table travels in the kernel arguments, so no host-to-device copy is needed.
constexpr int kMaxReqPerLaunch = 64;

struct AttnBatch {
  int32_t nreq;                                  // requests in this launch
  int32_t req0;                                  // global index of the first one
  int32_t chunk_base;                            // global chunk index of this launch's first chunk
  int32_t chunk_prefix[kMaxReqPerLaunch + 1];    // local chunk index where each request starts
  int32_t kv_len[kMaxReqPerLaunch];
  int64_t kv_off[kMaxReqPerLaunch];
  const uint64_t* anc;  // tree verification: [B][G] ancestor masks (bit a: tail position a visible), or null
  // Paged cache (kv_off unused): K and V pools [num_pages][Hkv][2^page_shift][D],
  // block table [B][max_pages] of page ids (clamped into [0, num_pages)), or null.
  const int32_t* pages;
  int32_t page_shift, max_pages, num_pages;
};

// Tree verification: ancestor masks [B][N + 1] from parents [B][N] (node i's
// parent in [-1, i), -1 the root; anything else is taken as the root).
hipError_t launch_tree_masks(int B, int N, const int32_t* parent, uint64_t* masks, hipStream_t stream);
// Tree commit: in each request's cache move the accepted nodes' K/V rows next
// to the root.
struct CommitBatch {
  int32_t nreq, req0;
  int32_t kv_len[kMaxReqPerLaunch];
  int64_t kv_off[kMaxReqPerLaunch];
};
hipError_t launch_tree_commit(const CommitBatch& cb, int Hkv, int G, int D, int esz, const int32_t* out_node,
                              const int32_t* accept_len, void* k_pool, void* v_pool, hipStream_t stream);

struct AttnShape {
  int G;            // query positions per request
  int Hq, Hkv, D;
  int group;        // Hq / Hkv
  int rows;         // G * group query rows per KV head
  int row_groups;   // waves that share a (chunk, KV head), each taking 16*RB consecutive rows
  int chunk_keys;   // keys per partial (one work item)
  float scale_log2; // softmax scale * log2(e)
};

// Partial results of one (chunk, KV head): running max m (log2 domain),
// sum l = sum exp2(s - m), unnormalised o = sum exp2(s - m) v.
struct AttnPartials {
  float* m;  // [slots][rows]
  float* l;  // [slots][rows]
  float* o;  // [slots][rows][D]
};

// Keys per work item (chunk), from the total number of keys over the batch;
// attn_max_chunks bounds the chunk count for any lengths up to max_kv_len.
int attn_chunk_keys(int dtype, int rows, int row_groups, int Hkv, const int32_t* kv_len, int B);
// Row groups of one (chunk, KV head): a wave holds at most kMaxRowBlocks
// 16-row blocks of O at head dimension 128 (more would spill registers).
int attn_row_groups(int dtype, int rows, int D);
int64_t attn_max_chunks(int dtype, int Hkv, int B, int64_t max_kv_len);
size_t attn_partial_bytes(int64_t total_chunks, int Hkv, int rows, int D);
AttnPartials attn_carve(void* ws, int64_t total_chunks, int Hkv, int rows, int D);

hipError_t launch_attention(int dtype, const AttnShape& s, const AttnBatch& batch, int nchunks,
                            const void* q, const void* k_pool, const void* v_pool,
                            AttnPartials parts, hipStream_t stream, hipEvent_t ev_start,
                            hipEvent_t ev_stop);
hipError_t launch_attention_combine(int dtype, const AttnShape& s, const AttnBatch& batch,
                                    AttnPartials parts, void* out, hipStream_t stream);

// Vocabulary projection.
struct VocabPlan {
  int M, K, V;
  int tile_n;      // vocabulary columns per workgroup
  int ntiles;      // ceil(V / tile_n)
  int mtiles;      // workgroups along the hidden rows
  int mblocks;     // bf16 row blocks per M-tile: of 16 rows (shallow), of 32 (deep)
  int nbw;         // 16-entry vocabulary blocks per wave (bf16)
  int waves;       // waves per workgroup
  bool deep;       // bf16 deep-pipelined 32x32 schedule (more than 64 rows)
  bool packed;     // W in the fragment-order layout of launch_pack_vocab
};
VocabPlan vocab_plan(int dtype, int M, int K, int V, bool packed);
size_t vocab_packed_bytes(int K, int V);
hipError_t launch_pack_vocab(int K, int V, const void* w, void* out, hipStream_t stream);
// Workspace of launch_vocab: the per-(row, tile) softmax statistics
// (float2[M][ntiles]) at its start, then, for the deep schedule, the hidden
// rows repacked into MFMA fragments.
size_t vocab_workspace_bytes(const VocabPlan& p);
// `clear` (nclear ints, may be null) is set to zero by the launch: the
// acceptance's arrival counters, for a fused acceptance launch that follows.
hipError_t launch_vocab(int dtype, const VocabPlan& p, const void* hidden, const void* w,
                        float* logits, void* workspace, hipStream_t stream, hipEvent_t ev_start,
                        hipEvent_t ev_stop, int* clear = nullptr, int nclear = 0);
hipError_t launch_lse_combine(const VocabPlan& p, const float2* partials, float* row_lse,
                              hipStream_t stream);

// Warped target rows for sampled verification: p'(v) = exp(logit(v) * inv_t
// - lse) where order_key(logit(v)) >= theta, else 0; greedy rows (argmax >= 0)
// are one-hot on argmax and have theta = 0xffffffff.
struct WarpRow {
  float inv_t;
  uint32_t theta;
  float lse;
  int32_t argmax;
};
// temperature 0 selects greedy; top_k 0 or >= V and top_p >= 1 switch the cuts off.
// Also writes each row's normaliser and smallest kept logit (-inf: no cut,
// +inf: greedy) to row_lse / row_min_logit.  ev_start (may be null) is
// recorded as the kernel starts.
hipError_t launch_warp(int M, int V, const float* logits, float temperature, int top_k, float top_p, WarpRow* out,
                       float* row_lse, float* row_min_logit, hipStream_t stream, hipEvent_t ev_start);

// Acceptance and resampling.
struct AcceptBatch {
  int32_t nreq;
  int32_t req0;
  int32_t has_kv_len;
  int32_t kv_len[kMaxReqPerLaunch];
};
size_t accept_workspace_bytes(int B, int V);
// The per-request arrival counters of the fused launch inside an acceptance
// workspace of accept_workspace_bytes(B, V) (B ints, global request index).
int* accept_arrivals(void* ws, int B, int V);
// x: logits with row_lse, or probabilities when row_lse is null.  With
// `partials` (the vocabulary kernel's per-tile statistics, ntiles per row) the
// row log-sum-exp is folded first and written to row_lse.  ws holds
// accept_workspace_bytes(B, V).  ev_start/ev_stop (may be null) time the
// segment-sum kernel.
// With `warp` (one WarpRow per row, from launch_warp) x holds logits and the
// test and correction use the warped p'; row_lse and partials are then unused.
// With `combine`, the pick launch also carries that attention merge.
// With `fused`, the sums and the pick run as one launch, which needs the
// arrival counters (accept_arrivals) of every request of the batch cleared by
// an earlier launch on the stream.
struct CombineJob;
hipError_t launch_accept(int gamma, int V, int B, const AcceptBatch& batch, const float* x,
                         const float* row_lse, const float2* partials, int ntiles,
                         const float* q_draft, const int32_t* draft_tok, const float* u, void* ws,
                         int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                         hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop,
                         const WarpRow* warp = nullptr, const CombineJob* combine = nullptr, bool fused = false);

// Tree verification (N = gamma nodes, position 0 the root, position i + 1 node
// i): walk the candidate tree, then draw the final token.  ws holds
// accept_tree_workspace_bytes(B, V).  out_node [B][N + 1]: the accepted nodes,
// then -1.  With `partials` (ntiles per row) the walk launch first folds the
// row log-sum-exps and writes them to row_lse; `fused` as for launch_accept.
size_t accept_tree_workspace_bytes(int B, int V);
hipError_t launch_accept_tree(int N, int V, int B, const AcceptBatch& batch, const float* x, const float* row_lse,
                              const int32_t* tokens, const int32_t* parent, const float* u, void* ws,
                              int32_t* accept_len, int32_t* out_tok, int32_t* out_node, int32_t* new_kv_len,
                              hipStream_t stream, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr,
                              const CombineJob* combine = nullptr, const float2* partials = nullptr, int ntiles = 0,
                              bool fused = false);

// Acceptance rate of every draft position: beta[b * gamma + i] = sum_v
// min(p(v), q_draft[b][i][v]), p from row b * (gamma + 1) + i of x (logits
// with row_lse, probabilities without), float64.  ws holds
// rate_workspace_bytes(B, gamma, V).  ev_start/ev_stop (may be null) bracket
// both launches.
size_t rate_workspace_bytes(int B, int gamma, int V);
hipError_t launch_rate(int gamma, int V, int B, const float* x, const float* row_lse, const float* q_draft, void* ws,
                       double* beta, hipStream_t stream, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// Draft-side layer expansion: children first_child + f*k + j (j < k, rank
// order) of frontier node frontier0 + f (-1: the root) of each of B requests,
// from the draft logits [B][F][V]; tokens, parent, q_child are [B][N].
constexpr int kExpandMaxK = 16;
struct ExpandArgs {
  int32_t B, F, V, k, frontier0, first_child, N;
};
hipError_t launch_expand(const ExpandArgs& e, const float* logits, int32_t* tokens, int32_t* parent, float* q_child,
                         hipStream_t stream, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

}  // namespace sdv
