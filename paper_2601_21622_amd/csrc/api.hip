// C-ABI of the verification library: argument checks, workspace layout and
// the launch sequence of each entry point.  Every check runs on the host
// before anything is enqueued.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>

#include <vector>

#include "sdverify.h"
#include "combine.h"
#include "launch.h"

#include <mutex>

// Scratch of sd_verify_step_static, for callers that cannot allocate: one
// copy per device, kept until the process ends.  Host code never uses this
// name as an address; it uses the device address hipGetSymbolAddress returns
// for the current device (static_scratch below).
static __device__ __align__(256) unsigned char scratch[SD_STATIC_SCRATCH_BYTES];

namespace {

using namespace sdv;

constexpr int kMaxRows = 128;       // G * (Hq / Hkv) handled by one attention workgroup
constexpr int kMaxRowsF32 = 64;
constexpr int kMaxVocab = 2097152;
constexpr int kMaxGamma = 63;
constexpr int64_t kMaxKvLen = int64_t(1) << 30;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t elem_size(int dtype) { return dtype == SD_DTYPE_BF16 ? 2 : 4; }

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

int check_dims(const sd_dims_t* d) {
  if (d == nullptr) return SD_ERR_INVALID_ARGUMENT;
  if (d->batch < 1 || d->gamma < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->hidden < 1 ||
      d->vocab < 1 || d->head_dim < 1)
    return SD_ERR_INVALID_ARGUMENT;
  if (d->dtype != SD_DTYPE_F32 && d->dtype != SD_DTYPE_BF16) return SD_ERR_INVALID_ARGUMENT;
  if (d->n_q_heads % d->n_kv_heads != 0) return SD_ERR_INVALID_ARGUMENT;
  if (d->head_dim != 64 && d->head_dim != 128) return SD_ERR_UNSUPPORTED;
  if (d->hidden % 32 != 0) return SD_ERR_UNSUPPORTED;
  if (d->vocab > kMaxVocab) return SD_ERR_UNSUPPORTED;
  if (d->gamma > kMaxGamma) return SD_ERR_UNSUPPORTED;
  const int64_t rows = int64_t(d->gamma + 1) * (d->n_q_heads / d->n_kv_heads);
  if (rows > (d->dtype == SD_DTYPE_F32 ? kMaxRowsF32 : kMaxRows)) return SD_ERR_UNSUPPORTED;
  if (int64_t(d->batch) * (d->gamma + 1) > (int64_t(1) << 24)) return SD_ERR_UNSUPPORTED;
  if ((d->flags & ~SD_FLAG_PACKED_VOCAB) != 0) return SD_ERR_INVALID_ARGUMENT;
  if ((d->flags & SD_FLAG_PACKED_VOCAB) && d->dtype != SD_DTYPE_BF16) return SD_ERR_UNSUPPORTED;
  return SD_OK;
}

// page_size > 0 (paged caches): chunks are whole pages, so each work item's
// page ids fit one register (a chunk is at most 4096 keys, a page at least 64).
AttnShape attn_shape(const sd_dims_t* d, float scale, const int32_t* kv_len = nullptr, int page_size = 0) {
  AttnShape s;
  s.G = d->gamma + 1;
  s.Hq = d->n_q_heads;
  s.Hkv = d->n_kv_heads;
  s.D = d->head_dim;
  s.group = d->n_q_heads / d->n_kv_heads;
  s.rows = s.G * s.group;
  s.row_groups = attn_row_groups(d->dtype, s.rows, s.D);
  s.chunk_keys = attn_chunk_keys(d->dtype, s.rows, s.row_groups, s.Hkv, kv_len, d->batch);
  if (page_size > 0) s.chunk_keys = (s.chunk_keys + page_size - 1) / page_size * page_size;
  s.scale_log2 = scale * 1.4426950408889634f;
  return s;
}

int64_t total_chunks(const int32_t* kv_len, int B, int chunk) {
  int64_t n = 0;
  for (int b = 0; b < B; ++b) n += (kv_len[b] + chunk - 1) / chunk;
  return n;
}

size_t attention_ws(const sd_dims_t* d, int64_t chunks) {
  const AttnShape s = attn_shape(d, 1.f);
  return align_up(attn_partial_bytes(chunks, s.Hkv, s.rows, s.D));
}

// Tree verification: the ancestor masks, at the start of the workspace.
size_t tree_ws(const sd_dims_t* d) { return align_up(sizeof(uint64_t) * static_cast<size_t>(d->batch) * (d->gamma + 1)); }

size_t logits_ws(const sd_dims_t* d) {
  const VocabPlan p = vocab_plan(d->dtype, d->batch * (d->gamma + 1), d->hidden, d->vocab, (d->flags & SD_FLAG_PACKED_VOCAB) != 0);
  return align_up(vocab_workspace_bytes(p));
}

int log2_exact(int v) {
  int k = 0;
  while ((1 << k) < v) ++k;
  return (1 << k) == v ? k : -1;
}

// A paged cache (bf16 only): table present and aligned, page size a power of
// two in [64, 4096], every request's keys within its table row.
int check_pages(const sd_dims_t* d, const sd_kv_pages_t* pg, const int32_t* kv_len) {
  if (pg == nullptr || kv_len == nullptr || pg->block_table == nullptr || !aligned(pg->block_table, 4))
    return SD_ERR_INVALID_ARGUMENT;
  if (d->dtype != SD_DTYPE_BF16) return SD_ERR_UNSUPPORTED;
  const int shift = log2_exact(pg->page_size);
  if (pg->page_size < 64 || pg->page_size > 4096 || shift < 0) return SD_ERR_INVALID_ARGUMENT;
  if (pg->num_pages < 1 || pg->max_pages < 1) return SD_ERR_INVALID_ARGUMENT;
  const int G = d->gamma + 1;
  for (int b = 0; b < d->batch; ++b) {
    if (kv_len[b] < G || kv_len[b] > kMaxKvLen) return SD_ERR_INVALID_ARGUMENT;
    if (int64_t(kv_len[b]) > int64_t(pg->max_pages) * pg->page_size) return SD_ERR_INVALID_ARGUMENT;
  }
  return SD_OK;
}

int check_kv(const sd_dims_t* d, const int64_t* kv_off, const int32_t* kv_len) {
  if (kv_off == nullptr || kv_len == nullptr) return SD_ERR_INVALID_ARGUMENT;
  const int G = d->gamma + 1;
  const size_t es = elem_size(d->dtype);
  for (int b = 0; b < d->batch; ++b) {
    if (kv_len[b] < G || kv_len[b] > kMaxKvLen) return SD_ERR_INVALID_ARGUMENT;
    if (kv_off[b] < 0 || (uint64_t(kv_off[b]) * es) % 16 != 0) return SD_ERR_INVALID_ARGUMENT;
  }
  return SD_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? SD_OK : SD_ERR_HIP; }

// Enqueue attention (partials + combine) for all requests, in launches of at
// most kMaxReqPerLaunch requests whose tables ride in the kernel arguments.
// With `deferred`, the merges are not launched: one CombineJob per launch is
// appended there instead, for a later launch to carry.
int run_attention(const sd_dims_t* d, const void* q, const void* k, const void* v, const int64_t* kv_off,
                  const int32_t* kv_len, float scale, void* out, void* ws, hipStream_t stream,
                  hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr, const uint64_t* anc = nullptr,
                  const sd_kv_pages_t* pages = nullptr, std::vector<CombineJob>* deferred = nullptr) {
  const AttnShape s = attn_shape(d, scale, kv_len, pages != nullptr ? pages->page_size : 0);
  const int64_t chunks = total_chunks(kv_len, d->batch, s.chunk_keys);
  const AttnPartials parts = attn_carve(ws, chunks, s.Hkv, s.rows, s.D);
  int64_t chunk_base = 0;
  for (int r0 = 0; r0 < d->batch; r0 += kMaxReqPerLaunch) {
    AttnBatch bt;
    memset(&bt, 0, sizeof(bt));
    bt.nreq = std::min(kMaxReqPerLaunch, d->batch - r0);
    bt.req0 = r0;
    bt.chunk_base = static_cast<int32_t>(chunk_base);
    bt.anc = anc;
    if (pages != nullptr) {
      bt.pages = pages->block_table;
      bt.page_shift = log2_exact(pages->page_size);
      bt.max_pages = pages->max_pages;
      bt.num_pages = pages->num_pages;
    }
    int32_t acc = 0;
    for (int i = 0; i < bt.nreq; ++i) {
      bt.chunk_prefix[i] = acc;
      bt.kv_len[i] = kv_len[r0 + i];
      bt.kv_off[i] = kv_off != nullptr ? kv_off[r0 + i] : 0;
      acc += (kv_len[r0 + i] + s.chunk_keys - 1) / s.chunk_keys;
    }
    bt.chunk_prefix[bt.nreq] = acc;
    const bool first = r0 == 0, last = r0 + kMaxReqPerLaunch >= d->batch;
    hipError_t e = launch_attention(d->dtype, s, bt, acc, q, k, v, parts, stream, first ? ev_start : nullptr,
                                    last ? ev_stop : nullptr);
    if (e != hipSuccess) return SD_ERR_HIP;
    if (deferred != nullptr) {
      CombineJob cj;
      memset(&cj, 0, sizeof(cj));
      cj.s = s;
      cj.bt = bt;
      cj.parts = parts;
      cj.out = out;
      cj.bf16 = d->dtype == SD_DTYPE_BF16;
      cj.nblocks = bt.nreq * s.Hkv * combine_zblocks(s);
      deferred->push_back(cj);
    } else if (launch_attention_combine(d->dtype, s, bt, parts, out, stream) != hipSuccess) {
      return SD_ERR_HIP;
    }
    chunk_base += acc;
  }
  return SD_OK;
}

int run_logits(const sd_dims_t* d, const void* hidden, const void* w, float* logits, float* row_lse, void* ws,
               hipStream_t stream, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr) {
  const VocabPlan p = vocab_plan(d->dtype, d->batch * (d->gamma + 1), d->hidden, d->vocab, (d->flags & SD_FLAG_PACKED_VOCAB) != 0);
  float2* partials = static_cast<float2*>(ws);
  hipError_t e = launch_vocab(d->dtype, p, hidden, w, logits, ws, stream, ev_start, ev_stop);
  if (e == hipSuccess) e = launch_lse_combine(p, partials, row_lse, stream);
  return hip_status(e);
}

// x holds logits with row_lse, or probabilities when row_lse is null.
// With `partials`, row_lse is an output: the log-sum-exp fold runs inside the
// acceptance stage.
int run_accept(const sd_dims_t* d, const float* x, const float* row_lse, const float2* partials, int ntiles,
               const float* q_draft, const int32_t* draft_tok, const float* u, const int32_t* kv_len,
               int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len, void* ws, hipStream_t stream,
               hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr, const WarpRow* warp = nullptr,
               const std::vector<CombineJob>* merges = nullptr, bool fused = false) {
  for (int r0 = 0; r0 < d->batch; r0 += kMaxReqPerLaunch) {
    AcceptBatch bt;
    memset(&bt, 0, sizeof(bt));
    bt.nreq = std::min(kMaxReqPerLaunch, d->batch - r0);
    bt.req0 = r0;
    bt.has_kv_len = kv_len != nullptr;
    if (kv_len != nullptr)
      for (int i = 0; i < bt.nreq; ++i) bt.kv_len[i] = kv_len[r0 + i];
    const bool first = r0 == 0, last = r0 + kMaxReqPerLaunch >= d->batch;
    // Both stages split the batch into the same launches of kMaxReqPerLaunch requests.
    const CombineJob* cj = merges != nullptr ? &(*merges)[r0 / kMaxReqPerLaunch] : nullptr;
    hipError_t e = launch_accept(d->gamma, d->vocab, d->batch, bt, x, row_lse, partials, ntiles, q_draft, draft_tok,
                                 u, ws, accept_len, out_tok, new_kv_len, stream, first ? ev_start : nullptr,
                                 last ? ev_stop : nullptr, warp, cj, fused);
    if (e != hipSuccess) return SD_ERR_HIP;
  }
  return SD_OK;
}

size_t accept_ws(const sd_dims_t* d) { return align_up(accept_workspace_bytes(d->batch, d->vocab)); }

// Warped target rows of sampled verification, after the acceptance sums.
size_t warp_ws(const sd_dims_t* d) { return align_up(sizeof(WarpRow) * static_cast<size_t>(d->batch) * (d->gamma + 1)); }

size_t accept_tree_ws(const sd_dims_t* d) { return align_up(accept_tree_workspace_bytes(d->batch, d->vocab)); }

// Workspace of the acceptance stage, whichever variant runs.
size_t accept_stage_ws(const sd_dims_t* d) { return std::max(accept_ws(d) + warp_ws(d), accept_tree_ws(d)); }

int run_accept_tree(const sd_dims_t* d, const float* x, const float* row_lse, const int32_t* tokens,
                    const int32_t* parent, const float* u, const int32_t* kv_len, int32_t* accept_len,
                    int32_t* out_tok, int32_t* out_node, int32_t* new_kv_len, void* ws, hipStream_t stream,
                    hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr,
                    const std::vector<CombineJob>* merges = nullptr, const float2* partials = nullptr, int ntiles = 0,
                    bool fused = false) {
  for (int r0 = 0; r0 < d->batch; r0 += kMaxReqPerLaunch) {
    AcceptBatch bt;
    memset(&bt, 0, sizeof(bt));
    bt.nreq = std::min(kMaxReqPerLaunch, d->batch - r0);
    bt.req0 = r0;
    bt.has_kv_len = kv_len != nullptr;
    if (kv_len != nullptr)
      for (int i = 0; i < bt.nreq; ++i) bt.kv_len[i] = kv_len[r0 + i];
    const bool first = r0 == 0, last = r0 + kMaxReqPerLaunch >= d->batch;
    const CombineJob* cj = merges != nullptr ? &(*merges)[r0 / kMaxReqPerLaunch] : nullptr;
    hipError_t e = launch_accept_tree(d->gamma, d->vocab, d->batch, bt, x, row_lse, tokens, parent, u, ws, accept_len,
                                      out_tok, out_node, new_kv_len, stream, first ? ev_start : nullptr,
                                      last ? ev_stop : nullptr, cj, partials, ntiles, fused);
    if (e != hipSuccess) return SD_ERR_HIP;
  }
  return SD_OK;
}

int check_sampling(const sd_sampling_t* sp) {
  if (sp == nullptr) return SD_ERR_INVALID_ARGUMENT;
  if (!std::isfinite(sp->temperature) || sp->temperature < 0.f) return SD_ERR_INVALID_ARGUMENT;
  if (sp->top_k < 0) return SD_ERR_INVALID_ARGUMENT;
  if (!(sp->top_p > 0.f && sp->top_p <= 1.f)) return SD_ERR_INVALID_ARGUMENT;
  return SD_OK;
}

size_t rate_ws(const sd_dims_t* d) { return align_up(rate_workspace_bytes(d->batch, d->gamma, d->vocab)); }

int check_accept_args(const float* x, const float* row_lse, const float* q_draft, const int32_t* draft_tok,
                      const float* u, const int32_t* kv_len, const int32_t* accept_len, const int32_t* out_tok,
                      const int32_t* new_kv_len) {
  if (!x || !q_draft || !draft_tok || !u || !accept_len || !out_tok) return SD_ERR_INVALID_ARGUMENT;
  if (new_kv_len != nullptr && kv_len == nullptr) return SD_ERR_INVALID_ARGUMENT;
  const void* p4[] = {x, row_lse, q_draft, draft_tok, u, accept_len, out_tok, new_kv_len};
  for (const void* p : p4)
    if (p != nullptr && !aligned(p, 4)) return SD_ERR_INVALID_ARGUMENT;
  return SD_OK;
}

int verify_step(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool, const int64_t* kv_off,
                const sd_kv_pages_t* pages, const int32_t* kv_len, float scale, const void* hidden,
                const void* w_vocab, const float* q_draft, const int32_t* draft_tok, const float* u,
                void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                int32_t* new_kv_len, void* workspace, size_t workspace_bytes, sd_stream_t stream,
                void* const* kernel_events);

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SD_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SD_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SD_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SD_OK;
}

// Workspace of one step's attention partials for these lengths.
size_t step_attention_ws(const sd_dims_t* dims, const int32_t* kv_len, float scale, const sd_kv_pages_t* pages) {
  const AttnShape s = attn_shape(dims, scale, kv_len, pages != nullptr ? pages->page_size : 0);
  return attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys));
}

// Workspace one step needs (arguments already checked).  With the caller's
// hidden rows the projection does not read the attention output, so the
// attention merge rides in the acceptance's last launch and its partials
// keep their own region: [partials][projection][acceptance].  Otherwise the
// stages reuse one region in stream order.
size_t step_ws(const sd_dims_t* dims, const int32_t* kv_len, float scale, const void* hidden,
               const sd_kv_pages_t* pages) {
  const size_t attn_bytes = step_attention_ws(dims, kv_len, scale, pages);
  return hidden != nullptr ? attn_bytes + logits_ws(dims) + accept_stage_ws(dims)
                           : std::max(attn_bytes, logits_ws(dims) + accept_stage_ws(dims));
}

}  // namespace

extern "C" {

size_t sd_workspace_bytes(const sd_dims_t* dims, int32_t max_kv_len) {
  if (check_dims(dims) != SD_OK || max_kv_len < dims->gamma + 1) return 0;
  const int64_t chunks = attn_max_chunks(dims->dtype, dims->n_kv_heads, dims->batch, max_kv_len);
  return std::max({tree_ws(dims) + attention_ws(dims, chunks) + logits_ws(dims) + accept_stage_ws(dims),
                   rate_ws(dims)});
}

int sd_verify_attention(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                        const int64_t* kv_off, const int32_t* kv_len, float scale, void* out, void* workspace,
                        size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!q || !k_pool || !v_pool || !out || !workspace) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(out, 16) ||
      !aligned(workspace, 16))
    return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const AttnShape s = attn_shape(dims, scale, kv_len);
  if (workspace_bytes < attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys)))
    return SD_ERR_WORKSPACE;
  return run_attention(dims, q, k_pool, v_pool, kv_off, kv_len, scale, out, workspace,
                       static_cast<hipStream_t>(stream));
}

int sd_verify_attention_tree(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                             const int64_t* kv_off, const int32_t* kv_len, const int32_t* parent, float scale,
                             void* out, void* workspace, size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!q || !k_pool || !v_pool || !out || !workspace || !parent) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(out, 16) ||
      !aligned(workspace, 16) || !aligned(parent, 4))
    return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const AttnShape s = attn_shape(dims, scale, kv_len);
  if (workspace_bytes < tree_ws(dims) + attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys)))
    return SD_ERR_WORKSPACE;
  hipStream_t stm = static_cast<hipStream_t>(stream);
  uint64_t* masks = static_cast<uint64_t*>(workspace);
  if (launch_tree_masks(dims->batch, dims->gamma, parent, masks, stm) != hipSuccess) return SD_ERR_HIP;
  return run_attention(dims, q, k_pool, v_pool, kv_off, kv_len, scale, out,
                       static_cast<char*>(workspace) + tree_ws(dims), stm, nullptr, nullptr, masks);
}

int sd_verify_logits(const sd_dims_t* dims, const void* hidden, const void* w_vocab, float* logits,
                     float* row_lse, void* workspace, size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!hidden || !w_vocab || !logits || !row_lse || !workspace) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(hidden, 16) || !aligned(w_vocab, 16) || !aligned(logits, 16) || !aligned(row_lse, 4) ||
      !aligned(workspace, 16))
    return SD_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < logits_ws(dims)) return SD_ERR_WORKSPACE;
  return run_logits(dims, hidden, w_vocab, logits, row_lse, workspace, static_cast<hipStream_t>(stream));
}

int sd_accept_resample(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse,
                       const float* q_draft, const int32_t* draft_tok, const float* u, const int32_t* kv_len,
                       int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len, void* workspace,
                       size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  st = check_accept_args(logits_or_probs, row_lse, q_draft, draft_tok, u, kv_len, accept_len, out_tok,
                         new_kv_len);
  if (st != SD_OK) return st;
  if (workspace == nullptr || !aligned(workspace, 16)) return SD_ERR_INVALID_ARGUMENT;
  if (kv_len != nullptr)
    for (int b = 0; b < dims->batch; ++b)
      if (kv_len[b] < dims->gamma + 1 || kv_len[b] > kMaxKvLen) return SD_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < accept_ws(dims)) return SD_ERR_WORKSPACE;
  return run_accept(dims, logits_or_probs, row_lse, nullptr, 0, q_draft, draft_tok, u, kv_len, accept_len, out_tok,
                    new_kv_len, workspace, static_cast<hipStream_t>(stream));
}

int sd_verify_step(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                   const int64_t* kv_off, const int32_t* kv_len, float scale, const void* hidden,
                   const void* w_vocab, const float* q_draft, const int32_t* draft_tok, const float* u,
                   void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                   int32_t* new_kv_len, void* workspace, size_t workspace_bytes, sd_stream_t stream,
                   void* const* kernel_events) {
  return verify_step(dims, q, k_pool, v_pool, kv_off, nullptr, kv_len, scale, hidden, w_vocab, q_draft, draft_tok, u,
                     attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace, workspace_bytes, stream,
                     kernel_events);
}

int sd_verify_step_paged(const sd_dims_t* dims, const void* q, const void* k_pages, const void* v_pages,
                         const sd_kv_pages_t* pages, const int32_t* kv_len, float scale, const void* hidden,
                         const void* w_vocab, const float* q_draft, const int32_t* draft_tok, const float* u,
                         void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                         int32_t* new_kv_len, void* workspace, size_t workspace_bytes, sd_stream_t stream,
                         void* const* kernel_events) {
  if (pages == nullptr) return SD_ERR_INVALID_ARGUMENT;
  return verify_step(dims, q, k_pages, v_pages, nullptr, pages, kv_len, scale, hidden, w_vocab, q_draft, draft_tok,
                     u, attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, workspace, workspace_bytes,
                     stream, kernel_events);
}

int sd_verify_attention_paged(const sd_dims_t* dims, const void* q, const void* k_pages, const void* v_pages,
                              const sd_kv_pages_t* pages, const int32_t* kv_len, float scale, void* out,
                              void* workspace, size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!q || !k_pages || !v_pages || !out || !workspace) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pages, 16) || !aligned(v_pages, 16) || !aligned(out, 16) ||
      !aligned(workspace, 16))
    return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_pages(dims, pages, kv_len);
  if (st != SD_OK) return st;
  const AttnShape s = attn_shape(dims, scale, kv_len, pages->page_size);
  if (workspace_bytes < attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys)))
    return SD_ERR_WORKSPACE;
  return run_attention(dims, q, k_pages, v_pages, nullptr, kv_len, scale, out, workspace,
                       static_cast<hipStream_t>(stream), nullptr, nullptr, nullptr, pages);
}

}  // extern "C"

namespace {

// One whole step; the cache is segments (kv_off) or pages (pages).
int verify_step(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool, const int64_t* kv_off,
                const sd_kv_pages_t* pages, const int32_t* kv_len, float scale, const void* hidden,
                const void* w_vocab, const float* q_draft, const int32_t* draft_tok, const float* u,
                void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                int32_t* new_kv_len, void* workspace, size_t workspace_bytes, sd_stream_t stream,
                void* const* kernel_events) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!q || !k_pool || !v_pool || !attn_out || !w_vocab || !logits || !row_lse || !workspace)
    return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(attn_out, 16) ||
      !aligned(w_vocab, 16) || !aligned(logits, 16) || !aligned(row_lse, 4) || !aligned(workspace, 16) ||
      (hidden != nullptr && !aligned(hidden, 16)))
    return SD_ERR_INVALID_ARGUMENT;
  if (hidden == nullptr && dims->hidden != dims->n_q_heads * dims->head_dim) return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_accept_args(logits, row_lse, q_draft, draft_tok, u, kv_len, accept_len, out_tok, new_kv_len);
  if (st != SD_OK) return st;
  st = pages != nullptr ? check_pages(dims, pages, kv_len) : check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const bool defer = hidden != nullptr;
  const size_t base = defer ? step_attention_ws(dims, kv_len, scale, pages) : 0;
  if (workspace_bytes < step_ws(dims, kv_len, scale, hidden, pages)) return SD_ERR_WORKSPACE;

  hipEvent_t ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  if (kernel_events != nullptr)
    for (int i = 0; i < 6; ++i) ev[i] = static_cast<hipEvent_t>(kernel_events[i]);
  hipStream_t stm = static_cast<hipStream_t>(stream);
  std::vector<CombineJob> merges;
  st = run_attention(dims, q, k_pool, v_pool, kv_off, kv_len, scale, attn_out, workspace, stm, ev[0], ev[1],
                     nullptr, pages, defer ? &merges : nullptr);
  if (st != SD_OK) return st;
  // The vocabulary statistics come first in their region and the acceptance
  // sums after them, since the fold reads the former while the segment kernel
  // writes the latter.
  void* vws = static_cast<char*>(workspace) + base;
  const VocabPlan vp = vocab_plan(dims->dtype, dims->batch * (dims->gamma + 1), dims->hidden, dims->vocab, (dims->flags & SD_FLAG_PACKED_VOCAB) != 0);
  float2* partials = static_cast<float2*>(vws);
  // The projection launch clears the acceptance's arrival counters, so the
  // acceptance runs as one launch.
  void* acc_ws = static_cast<char*>(vws) + logits_ws(dims);
  if (launch_vocab(dims->dtype, vp, hidden != nullptr ? hidden : attn_out, w_vocab, logits, vws, stm, ev[2], ev[3],
                   accept_arrivals(acc_ws, dims->batch, dims->vocab), dims->batch) != hipSuccess)
    return SD_ERR_HIP;
  return run_accept(dims, logits, row_lse, partials, vp.ntiles, q_draft, draft_tok, u, kv_len, accept_len, out_tok,
                    new_kv_len, acc_ws, stm, ev[4], ev[5], nullptr, defer ? &merges : nullptr, true);
}

}  // namespace

extern "C" {

int sd_accept_resample_sampled(const sd_dims_t* dims, const sd_sampling_t* sampling, const float* logits,
                               const float* q_draft, const int32_t* draft_tok, const float* u, const int32_t* kv_len,
                               float* row_lse, float* row_min_logit, int32_t* accept_len, int32_t* out_tok,
                               int32_t* new_kv_len, void* workspace, size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  st = check_sampling(sampling);
  if (st != SD_OK) return st;
  st = check_accept_args(logits, row_lse, q_draft, draft_tok, u, kv_len, accept_len, out_tok, new_kv_len);
  if (st != SD_OK) return st;
  if (!row_lse || !row_min_logit || !aligned(row_min_logit, 4)) return SD_ERR_INVALID_ARGUMENT;
  if (workspace == nullptr || !aligned(workspace, 16)) return SD_ERR_INVALID_ARGUMENT;
  if (kv_len != nullptr)
    for (int b = 0; b < dims->batch; ++b)
      if (kv_len[b] < dims->gamma + 1 || kv_len[b] > kMaxKvLen) return SD_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < accept_ws(dims) + warp_ws(dims)) return SD_ERR_WORKSPACE;
  hipStream_t stm = static_cast<hipStream_t>(stream);
  WarpRow* warp = reinterpret_cast<WarpRow*>(static_cast<char*>(workspace) + accept_ws(dims));
  if (launch_warp(dims->batch * (dims->gamma + 1), dims->vocab, logits, sampling->temperature, sampling->top_k,
                  sampling->top_p, warp, row_lse, row_min_logit, stm, nullptr) != hipSuccess)
    return SD_ERR_HIP;
  return run_accept(dims, logits, nullptr, nullptr, 0, q_draft, draft_tok, u, kv_len, accept_len, out_tok,
                    new_kv_len, workspace, stm, nullptr, nullptr, warp);
}

int sd_verify_step_sampled(const sd_dims_t* dims, const sd_sampling_t* sampling, const void* q, const void* k_pool,
                           const void* v_pool, const int64_t* kv_off, const int32_t* kv_len, float scale,
                           const void* hidden, const void* w_vocab, const float* q_draft, const int32_t* draft_tok,
                           const float* u, void* attn_out, float* logits, float* row_lse, float* row_min_logit,
                           int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len, void* workspace,
                           size_t workspace_bytes, sd_stream_t stream, void* const* kernel_events) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  st = check_sampling(sampling);
  if (st != SD_OK) return st;
  if (!q || !k_pool || !v_pool || !attn_out || !w_vocab || !logits || !row_lse || !row_min_logit || !workspace)
    return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(attn_out, 16) ||
      !aligned(w_vocab, 16) || !aligned(logits, 16) || !aligned(row_lse, 4) || !aligned(row_min_logit, 4) ||
      !aligned(workspace, 16) || (hidden != nullptr && !aligned(hidden, 16)))
    return SD_ERR_INVALID_ARGUMENT;
  if (hidden == nullptr && dims->hidden != dims->n_q_heads * dims->head_dim) return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_accept_args(logits, row_lse, q_draft, draft_tok, u, kv_len, accept_len, out_tok, new_kv_len);
  if (st != SD_OK) return st;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const AttnShape s = attn_shape(dims, scale, kv_len);
  const size_t need = std::max(attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys)),
                               logits_ws(dims) + accept_stage_ws(dims));
  if (workspace_bytes < need) return SD_ERR_WORKSPACE;

  hipEvent_t ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  if (kernel_events != nullptr)
    for (int i = 0; i < 6; ++i) ev[i] = static_cast<hipEvent_t>(kernel_events[i]);
  hipStream_t stm = static_cast<hipStream_t>(stream);
  st = run_attention(dims, q, k_pool, v_pool, kv_off, kv_len, scale, attn_out, workspace, stm, ev[0], ev[1]);
  if (st != SD_OK) return st;
  const VocabPlan vp = vocab_plan(dims->dtype, dims->batch * (dims->gamma + 1), dims->hidden, dims->vocab,
                                  (dims->flags & SD_FLAG_PACKED_VOCAB) != 0);
  // The projection launch clears the acceptance's arrival counters, so the
  // acceptance runs as one launch.
  void* acc_ws = static_cast<char*>(workspace) + logits_ws(dims);
  if (launch_vocab(dims->dtype, vp, hidden != nullptr ? hidden : attn_out, w_vocab, logits, workspace, stm, ev[2],
                   ev[3], accept_arrivals(acc_ws, dims->batch, dims->vocab), dims->batch) != hipSuccess)
    return SD_ERR_HIP;
  WarpRow* warp = reinterpret_cast<WarpRow*>(static_cast<char*>(acc_ws) + accept_ws(dims));
  if (launch_warp(dims->batch * (dims->gamma + 1), dims->vocab, logits, sampling->temperature, sampling->top_k,
                  sampling->top_p, warp, row_lse, row_min_logit, stm, ev[4]) != hipSuccess)
    return SD_ERR_HIP;
  return run_accept(dims, logits, nullptr, nullptr, 0, q_draft, draft_tok, u, kv_len, accept_len, out_tok,
                    new_kv_len, acc_ws, stm, nullptr, ev[5], warp, nullptr, true);
}

int sd_accept_tree(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse, const int32_t* tokens,
                   const int32_t* parent, const float* u, const int32_t* kv_len, int32_t* accept_len,
                   int32_t* out_tok, int32_t* out_node, int32_t* new_kv_len, void* workspace,
                   size_t workspace_bytes, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!logits_or_probs || !tokens || !parent || !u || !accept_len || !out_tok || !out_node || !workspace)
    return SD_ERR_INVALID_ARGUMENT;
  if (new_kv_len != nullptr && kv_len == nullptr) return SD_ERR_INVALID_ARGUMENT;
  const void* p4[] = {logits_or_probs, row_lse, tokens, parent, u, accept_len, out_tok, out_node, new_kv_len};
  for (const void* p : p4)
    if (p != nullptr && !aligned(p, 4)) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(workspace, 16)) return SD_ERR_INVALID_ARGUMENT;
  if (kv_len != nullptr)
    for (int b = 0; b < dims->batch; ++b)
      if (kv_len[b] < dims->gamma + 1 || kv_len[b] > kMaxKvLen) return SD_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < accept_tree_ws(dims)) return SD_ERR_WORKSPACE;
  return run_accept_tree(dims, logits_or_probs, row_lse, tokens, parent, u, kv_len, accept_len, out_tok, out_node,
                         new_kv_len, workspace, static_cast<hipStream_t>(stream));
}

int sd_verify_step_tree(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                        const int64_t* kv_off, const int32_t* kv_len, const int32_t* parent, float scale,
                        const void* hidden, const void* w_vocab, const int32_t* tokens, const float* u,
                        void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                        int32_t* out_node, int32_t* new_kv_len, void* workspace, size_t workspace_bytes,
                        sd_stream_t stream, void* const* kernel_events) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!q || !k_pool || !v_pool || !attn_out || !w_vocab || !logits || !row_lse || !workspace || !parent || !tokens ||
      !u || !accept_len || !out_tok || !out_node)
    return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(attn_out, 16) ||
      !aligned(w_vocab, 16) || !aligned(logits, 16) || !aligned(row_lse, 4) || !aligned(workspace, 16) ||
      !aligned(parent, 4) || !aligned(tokens, 4) || !aligned(u, 4) || !aligned(accept_len, 4) ||
      !aligned(out_tok, 4) || !aligned(out_node, 4) || (new_kv_len != nullptr && !aligned(new_kv_len, 4)) ||
      (hidden != nullptr && !aligned(hidden, 16)))
    return SD_ERR_INVALID_ARGUMENT;
  if (hidden == nullptr && dims->hidden != dims->n_q_heads * dims->head_dim) return SD_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const AttnShape s = attn_shape(dims, scale, kv_len);
  const size_t attn_bytes = tree_ws(dims) + attention_ws(dims, total_chunks(kv_len, dims->batch, s.chunk_keys));
  // As in the chain step: with the caller's hidden rows the attention merge
  // rides in the acceptance's last launch, and the masks and partials keep
  // their region: [masks][partials][projection][acceptance].
  const bool defer = hidden != nullptr;
  const size_t base = defer ? attn_bytes : 0;
  const size_t need = defer ? attn_bytes + logits_ws(dims) + accept_stage_ws(dims)
                            : std::max(attn_bytes, logits_ws(dims) + accept_stage_ws(dims));
  if (workspace_bytes < need) return SD_ERR_WORKSPACE;

  hipEvent_t ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  if (kernel_events != nullptr)
    for (int i = 0; i < 6; ++i) ev[i] = static_cast<hipEvent_t>(kernel_events[i]);
  hipStream_t stm = static_cast<hipStream_t>(stream);
  uint64_t* masks = static_cast<uint64_t*>(workspace);
  if (launch_tree_masks(dims->batch, dims->gamma, parent, masks, stm) != hipSuccess) return SD_ERR_HIP;
  std::vector<CombineJob> merges;
  st = run_attention(dims, q, k_pool, v_pool, kv_off, kv_len, scale, attn_out,
                     static_cast<char*>(workspace) + tree_ws(dims), stm, ev[0], ev[1], masks, nullptr,
                     defer ? &merges : nullptr);
  if (st != SD_OK) return st;
  void* vws = static_cast<char*>(workspace) + base;
  // The projection launch clears the acceptance's arrival counters; the walk
  // launch folds the row log-sum-exps from the projection's statistics, and
  // the final draw runs as one launch.
  const VocabPlan vp = vocab_plan(dims->dtype, dims->batch * (dims->gamma + 1), dims->hidden, dims->vocab,
                                  (dims->flags & SD_FLAG_PACKED_VOCAB) != 0);
  void* acc_ws = static_cast<char*>(vws) + logits_ws(dims);
  if (launch_vocab(dims->dtype, vp, hidden != nullptr ? hidden : attn_out, w_vocab, logits, vws, stm, ev[2], ev[3],
                   accept_arrivals(acc_ws, dims->batch, dims->vocab), dims->batch) != hipSuccess)
    return SD_ERR_HIP;
  return run_accept_tree(dims, logits, row_lse, tokens, parent, u, kv_len, accept_len, out_tok, out_node,
                         new_kv_len, acc_ws, stm, ev[4], ev[5], defer ? &merges : nullptr,
                         static_cast<const float2*>(vws), vp.ntiles, true);
}

int sd_tree_commit_kv(const sd_dims_t* dims, void* k_pool, void* v_pool, const int64_t* kv_off,
                      const int32_t* kv_len, const int32_t* out_node, const int32_t* accept_len, sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!k_pool || !v_pool || !out_node || !accept_len) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(out_node, 4) || !aligned(accept_len, 4))
    return SD_ERR_INVALID_ARGUMENT;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  const int G = dims->gamma + 1;
  for (int r0 = 0; r0 < dims->batch; r0 += kMaxReqPerLaunch) {
    CommitBatch cb;
    memset(&cb, 0, sizeof(cb));
    cb.nreq = std::min(kMaxReqPerLaunch, dims->batch - r0);
    cb.req0 = r0;
    for (int i = 0; i < cb.nreq; ++i) {
      cb.kv_len[i] = kv_len[r0 + i];
      cb.kv_off[i] = kv_off[r0 + i];
    }
    if (launch_tree_commit(cb, dims->n_kv_heads, G, dims->head_dim, static_cast<int>(elem_size(dims->dtype)),
                           out_node, accept_len, k_pool, v_pool, static_cast<hipStream_t>(stream)) != hipSuccess)
      return SD_ERR_HIP;
  }
  return SD_OK;
}

int sd_acceptance_rate(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse,
                       const float* q_draft, double* beta, void* workspace, size_t workspace_bytes,
                       sd_stream_t stream) {
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (!logits_or_probs || !q_draft || !beta || !workspace) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(logits_or_probs, 4) || (row_lse != nullptr && !aligned(row_lse, 4)) || !aligned(q_draft, 4) ||
      !aligned(beta, 8) || !aligned(workspace, 16))
    return SD_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < rate_ws(dims)) return SD_ERR_WORKSPACE;
  return hip_status(launch_rate(dims->gamma, dims->vocab, dims->batch, logits_or_probs, row_lse, q_draft, workspace,
                                beta, static_cast<hipStream_t>(stream)));
}

int sd_expand_layer(const sd_expand_t* e, const float* draft_logits, int32_t* tokens, int32_t* parent,
                    float* q_child, sd_stream_t stream) {
  if (e == nullptr || !draft_logits || !tokens || !parent || !q_child) return SD_ERR_INVALID_ARGUMENT;
  if (!aligned(draft_logits, 4) || !aligned(tokens, 4) || !aligned(parent, 4) || !aligned(q_child, 4))
    return SD_ERR_INVALID_ARGUMENT;
  if (e->batch < 1 || e->frontier < 1 || e->vocab < 1 || e->top_k < 1 || e->nodes < 1 || e->first_child < 0 ||
      e->frontier0 < -1)
    return SD_ERR_INVALID_ARGUMENT;
  if (e->top_k > e->vocab) return SD_ERR_INVALID_ARGUMENT;
  if (e->top_k > kExpandMaxK || e->vocab > kMaxVocab) return SD_ERR_UNSUPPORTED;
  if (int64_t(e->first_child) + int64_t(e->frontier) * e->top_k > e->nodes) return SD_ERR_INVALID_ARGUMENT;
  if (e->frontier0 >= 0 && int64_t(e->frontier0) + e->frontier > e->first_child) return SD_ERR_INVALID_ARGUMENT;
  if (int64_t(e->batch) * e->frontier > 0x7fffffff) return SD_ERR_UNSUPPORTED;
  const ExpandArgs a{e->batch, e->frontier, e->vocab, e->top_k, e->frontier0, e->first_child, e->nodes};
  return hip_status(launch_expand(a, draft_logits, tokens, parent, q_child, static_cast<hipStream_t>(stream)));
}

size_t sd_vocab_packed_bytes(const sd_dims_t* dims) {
  if (check_dims(dims) != SD_OK || dims->dtype != SD_DTYPE_BF16) return 0;
  return vocab_packed_bytes(dims->hidden, dims->vocab);
}

int sd_pack_vocab(const sd_dims_t* dims, const void* w_vocab, void* w_packed, sd_stream_t stream) {
  const int st = check_dims(dims);
  if (st != SD_OK) return st;
  if (dims->dtype != SD_DTYPE_BF16) return SD_ERR_UNSUPPORTED;
  if (!w_vocab || !w_packed || !aligned(w_vocab, 16) || !aligned(w_packed, 16)) return SD_ERR_INVALID_ARGUMENT;
  const char* a = static_cast<const char*>(w_vocab);
  const char* b = static_cast<const char*>(w_packed);
  const size_t na = sizeof(uint16_t) * static_cast<size_t>(dims->vocab) * dims->hidden;
  const size_t nb = vocab_packed_bytes(dims->hidden, dims->vocab);
  if (a < b + nb && b < a + na) return SD_ERR_INVALID_ARGUMENT;  // overlapping buffers
  return hip_status(launch_pack_vocab(dims->hidden, dims->vocab, w_vocab, w_packed, static_cast<hipStream_t>(stream)));
}

int sd_verify_step_static(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                          const int64_t* kv_off, const int32_t* kv_len, float scale, const void* hidden,
                          const void* w_vocab, const float* q_draft, const int32_t* draft_tok, const float* u,
                          void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                          int32_t* new_kv_len, sd_stream_t stream) {
  // The checks the step's size depends on, then the size against the static
  // maximum, on the host before anything touches a device.
  int st = check_dims(dims);
  if (st != SD_OK) return st;
  st = check_kv(dims, kv_off, kv_len);
  if (st != SD_OK) return st;
  if (!(scale > 0.f) || !std::isfinite(scale)) return SD_ERR_INVALID_ARGUMENT;
  if (step_ws(dims, kv_len, scale, hidden, nullptr) > SD_STATIC_SCRATCH_BYTES) return SD_ERR_WORKSPACE;
  void* ws = nullptr;
  st = static_scratch(&ws);
  if (st != SD_OK) return st;
  return verify_step(dims, q, k_pool, v_pool, kv_off, nullptr, kv_len, scale, hidden, w_vocab, q_draft, draft_tok, u,
                     attn_out, logits, row_lse, accept_len, out_tok, new_kv_len, ws, SD_STATIC_SCRATCH_BYTES, stream,
                     nullptr);
}

const char* sd_vocab_kernel_name(const sd_dims_t* dims) {
  if (check_dims(dims) != SD_OK) return nullptr;
  const VocabPlan p = vocab_plan(dims->dtype, dims->batch * (dims->gamma + 1), dims->hidden, dims->vocab,
                                 (dims->flags & SD_FLAG_PACKED_VOCAB) != 0);
  if (dims->dtype == SD_DTYPE_F32) return "vocab_f32_kernel";
  if (!p.deep) return "vocab_bf16_kernel";
  // The wide schedule is the deep shape with four 32-entry blocks per wave
  // on four waves (16-entry blocks per wave: 8).
  return (p.nbw == 8 && p.waves == 4) ? "vocab_bf16_wide_kernel" : "vocab_bf16_deep_kernel";
}

const char* sd_status_string(int status) {
  switch (status) {
    case SD_OK: return "SD_OK: success";
    case SD_ERR_INVALID_ARGUMENT: return "SD_ERR_INVALID_ARGUMENT: null or misaligned pointer, bad size or inconsistent shape";
    case SD_ERR_UNSUPPORTED: return "SD_ERR_UNSUPPORTED: shape outside what the kernels implement";
    case SD_ERR_WORKSPACE: return "SD_ERR_WORKSPACE: workspace smaller than sd_workspace_bytes requires";
    case SD_ERR_HIP: return "SD_ERR_HIP: a HIP launch or runtime call failed";
    case SD_ERR_CAPACITY: return "SD_ERR_CAPACITY: the KV page pool has too few free pages";
    default: return "unknown status";
  }
}

const char* sd_version(void) { return "0.1.0"; }

}  // extern "C"
