/*
 * sdverify.h -- batched, lossless speculative verification on one MI355X (gfx950).
 *
 * The verification step of StarSD's one-for-many speculative decoding: one
 * verifier scores a pooled batch of B requests, each carrying gamma draft
 * tokens x_1..x_gamma, the draft distributions q_1..q_gamma they were drawn
 * from, its own KV cache and uniform draws, and returns for every request the
 * accepted prefix plus one corrected (or bonus) token.
 *   - Algorithm 2 (EAGLE speculative decoding), verification of a path: the
 *     target model runs along the gamma + 1 prefixes in parallel, giving
 *     p_1..p_{gamma+1}; a stochastic test gives the accept length l; a
 *     correction is sampled from norm(max(0, p_{l+1} - q_{l+1})).
 *   - Sec. 2 (Preliminary): the per-request primitive and the Leviathan et al.
 *     formulation whose ratio test u < p_i(x_i)/q_i(x_i) is used here.
 *   - Sec. 3.2, Eq. (1): the acceptance probability sum_x min(p, q) that test has.
 *   - Algorithm 1 and its design properties: requests from many targets are
 *     pooled, each isolated to its own state; here each request owns its own
 *     KV segment and all share one vocabulary projection.
 *
 * Conventions shared by every call
 *   - G = gamma + 1 query positions per request: position 0 is the root (last
 *     verified token), position i >= 1 is draft x_i.  M = B * G.
 *   - All pointers are DEVICE pointers unless marked (host).  Device buffers
 *     are read or written only by work enqueued on `stream`; they must stay
 *     alive until that work completes.  The library allocates no device memory,
 *     keeps no pointer after returning, enqueues work only (never synchronises)
 *     and is re-entrant.  Scratch space comes from the caller's `workspace`;
 *     its size is given by sd_workspace_bytes.  Its contents on entry do not
 *     matter: what a call needs at zero (the per-request arrival counters of a
 *     step's one-launch acceptance) it clears itself, on the same stream.
 *   - Device pointers to Q/K/V/hidden/W/workspace must be 16-byte aligned;
 *     float/int32 arrays 4-byte aligned.
 *   - Return value: SD_OK or a negative status (see sd_status_string).  All
 *     argument checks run on the host before anything is enqueued; on an
 *     error nothing is enqueued.  The library never aborts or exits.
 *   - Device-array preconditions that are not checked (documented only):
 *     draft tokens lie in [0, vocab) (a token outside it is treated as
 *     rejected, never read out of bounds); q rows are distributions.
 *   - Results are deterministic: no floating-point atomics, fixed reduction order
 *     (the one integer atomic only counts workgroups in; which one comes last
 *     does not change any result).
 */
#ifndef SDVERIFY_H
#define SDVERIFY_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define SD_API __attribute__((visibility("default")))
#else
#define SD_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* A hipStream_t passed as an opaque pointer (NULL = the null stream). */
typedef void* sd_stream_t;

typedef enum {
  SD_DTYPE_F32 = 0,  /* float32 Q/K/V/hidden/W; attention output float32 */
  SD_DTYPE_BF16 = 1  /* bfloat16 Q/K/V/hidden/W; attention output bfloat16 */
} sd_dtype_t;

enum {
  SD_OK = 0,
  SD_ERR_INVALID_ARGUMENT = -1, /* null/misaligned pointer, bad size, inconsistent shape */
  SD_ERR_UNSUPPORTED = -2,      /* valid but outside what the kernels implement */
  SD_ERR_WORKSPACE = -3,        /* workspace smaller than sd_workspace_bytes requires */
  SD_ERR_HIP = -4,              /* a HIP launch or runtime call failed */
  SD_ERR_CAPACITY = -5          /* a KV page pool has too few free pages */
};

/* Flags of sd_dims_t.flags. */
enum {
  /* w_vocab arguments point to weights repacked by sd_pack_vocab (bf16 only). */
  SD_FLAG_PACKED_VOCAB = 1
};

/* Problem shape.  Accumulation is always float32 (float64 for the sampling sums). */
typedef struct {
  int32_t batch;      /* B >= 1 pooled requests (one per target session) */
  int32_t gamma;      /* draft tokens per request, >= 1 (the paper's depth d, branching 1) */
  int32_t n_q_heads;  /* query heads, a multiple of n_kv_heads */
  int32_t n_kv_heads; /* KV heads; query head h reads KV head h / (n_q_heads / n_kv_heads) */
  int32_t head_dim;   /* 64 or 128 */
  int32_t hidden;     /* width of the vocabulary projection's input, a multiple of 32 */
  int32_t vocab;      /* V, 1 .. 2,097,152 */
  int32_t dtype;      /* sd_dtype_t */
  int32_t flags;      /* bitwise OR of SD_FLAG_*, 0 by default */
} sd_dims_t;

/*
 * Workspace bytes needed by any call below for `dims` with every kv_len <=
 * max_kv_len.  Returns 0 for an invalid shape.
 */
SD_API size_t sd_workspace_bytes(const sd_dims_t* dims, int32_t max_kv_len);

/*
 * Causal multi-query verification attention (Algorithm 2: the target model
 * along the gamma + 1 prefixes of a path, evaluated in parallel).
 *   q        [B][G][Hq][D]          query vectors, already position-encoded
 *   k_pool   request b: [Hkv][kv_len[b]][D] starting at element kv_off[b]
 *   v_pool   same layout as k_pool
 *   kv_off   (host) [B] element offsets; kv_off[b] * sizeof(dtype) % 16 == 0
 *   kv_len   (host) [B] cached length L_b INCLUDING this step's G positions,
 *            G <= L_b <= 2^30; query j attends to keys 0 .. L_b - G + j
 *   scale    softmax scale, finite and > 0 (SD_ERR_INVALID_ARGUMENT otherwise);
 *            1/sqrt(head_dim) for the usual definition
 *   out      [B][G][Hq][D] in dtype: softmax(q k^T * scale) v per (request, head, query)
 * Requires G * (n_q_heads / n_kv_heads) <= 128 (SD_ERR_UNSUPPORTED otherwise).
 */
SD_API int sd_verify_attention(const sd_dims_t* dims, const void* q, const void* k_pool,
                        const void* v_pool, const int64_t* kv_off, const int32_t* kv_len,
                        float scale, void* out, void* workspace, size_t workspace_bytes,
                        sd_stream_t stream);

/*
 * Tree verification: attention of the G = gamma + 1 positions of a candidate
 * tree (Algorithm 2's proposal tree, scored in one pass).  Here gamma is the
 * number of tree nodes N; position 0 is the root (the last verified token)
 * and position i + 1 is node i.  Arguments as in sd_verify_attention, plus
 *   parent   [B][N] int32 (device): parent[b][i] in [-1, i) is node i's parent
 *            node (-1: the root); parents precede their children.  A value
 *            outside that range is taken as -1.
 * The last G entries of each request's cache are the root and the nodes in
 * position order.  Position g attends to every key before them and to tail
 * position a iff a is g, the root or an ancestor of g.  A chain (parent[i] =
 * i - 1) gives sd_verify_attention's result.
 */
SD_API int sd_verify_attention_tree(const sd_dims_t* dims, const void* q, const void* k_pool,
                                    const void* v_pool, const int64_t* kv_off, const int32_t* kv_len,
                                    const int32_t* parent, float scale, void* out, void* workspace,
                                    size_t workspace_bytes, sd_stream_t stream);

/*
 * Repacked vocabulary weights.  The projection streams W once per step; in
 * the [V][hidden] layout every MFMA operand load touches 16 rows 2*hidden
 * bytes apart.  sd_pack_vocab rewrites W once (at weight-load time) into
 * fragment order, [hidden/32][ceil(V/16)][64 lanes][8 bf16]: fragment (s, n)
 * holds, for lane l, W[16n + l%16][32s + 8(l/16) .. +8], rows past V zero.
 * Each operand load is then 1 KB contiguous, and at every k-step the whole
 * grid reads one contiguous slab.  A w_vocab in this layout is passed with
 * SD_FLAG_PACKED_VOCAB set in dims->flags.  bf16 only.
 *   sd_vocab_packed_bytes  bytes of the packed buffer (0 for an invalid or fp32 shape)
 *   sd_pack_vocab          w_vocab [V][hidden] bf16 (device) -> w_packed (device,
 *                          sd_vocab_packed_bytes bytes, 16-byte aligned, not
 *                          overlapping w_vocab); enqueued on `stream`.
 */
SD_API size_t sd_vocab_packed_bytes(const sd_dims_t* dims);
SD_API int sd_pack_vocab(const sd_dims_t* dims, const void* w_vocab, void* w_packed, sd_stream_t stream);

/*
 * Vocabulary projection and row log-sum-exp: the target distributions
 * p_1..p_{gamma+1} of Algorithm 2 (temperature 1).
 *   hidden   [M][hidden] in dtype; row b*G + j feeds p_{j+1} of request b
 *   w_vocab  [V][hidden] in dtype (one row per vocabulary entry), or the
 *            sd_pack_vocab layout when dims->flags has SD_FLAG_PACKED_VOCAB
 *   logits   [M][V] float32 output: logits[m][v] = sum_k hidden[m][k] * w_vocab[v][k]
 *   row_lse  [M] float32 output: log sum_v exp(logits[m][v])
 * so that p_{j+1}(v) = exp(logits[b*G+j][v] - row_lse[b*G+j]).
 */
SD_API int sd_verify_logits(const sd_dims_t* dims, const void* hidden, const void* w_vocab,
                     float* logits, float* row_lse, void* workspace, size_t workspace_bytes,
                     sd_stream_t stream);

/*
 * Acceptance test, first rejection, residual resampling and output assembly
 * (Algorithm 2, stochastic test and correction; Leviathan ratio rule).
 *   logits_or_probs [M][V] float32: logits if row_lse != NULL, else probabilities
 *   row_lse         [M] float32 or NULL
 *   q_draft         [B][gamma][V] float32: q_draft[b][i] is the distribution x_{i+1} was drawn from
 *   draft_tok       [B][gamma] int32: x_1..x_gamma
 *   u               [B][G] float32 in [0,1): u[b][i] tests x_{i+1}; u[b][gamma] drives the final sample
 *   kv_len          (host) [B] as for sd_verify_attention; required iff new_kv_len != NULL
 *   accept_len      [B] int32 output: l_b in [0, gamma]
 *   out_tok         [B][G] int32 output: x_1..x_l, then the sampled token, then -1 padding
 *   new_kv_len      [B] int32 output or NULL: kv_len[b] - gamma + l_b (cache entries to keep)
 *   workspace       at least sd_workspace_bytes(dims, ...) bytes (per-segment partial sums)
 * Rules (per request, p_i = row b*G + i - 1):
 *   ratio_i = p_i(x_i) / q_i(x_i), with ratio = 0 if p_i(x_i) = 0 and +inf if
 *   q_i(x_i) = 0 < p_i(x_i); x_i passes iff u[b][i-1] < ratio_i; l = number of
 *   leading passes.  The final token is drawn from r = max(0, p_{l+1} - q_{l+1})
 *   if l < gamma, else r = p_{gamma+1} (the bonus), by inverse CDF in ascending
 *   token id: t = min{k : C_k > u[b][gamma] * Z}, C the float64 inclusive prefix
 *   sums of r and Z = C_{V-1}; if no k qualifies, t is the largest k with
 *   r(k) > 0; if Z is not positive, r falls back to p_{l+1}.  p(v) is evaluated
 *   from logits as exp(logit - lse) with the difference kept exact; the ratio test
 *   runs in float64.
 */
SD_API int sd_accept_resample(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse,
                       const float* q_draft, const int32_t* draft_tok, const float* u,
                       const int32_t* kv_len, int32_t* accept_len, int32_t* out_tok,
                       int32_t* new_kv_len, void* workspace, size_t workspace_bytes,
                       sd_stream_t stream);

/*
 * One whole verification step: sd_verify_attention, then sd_verify_logits on
 * `hidden` (or, when hidden == NULL, on the attention output viewed as
 * [M][n_q_heads * head_dim], which then must equal dims->hidden), then
 * sd_accept_resample on the logits and row_lse it produced.  Arguments as in
 * the three calls; attn_out, logits, row_lse are outputs the caller owns.
 *   kernel_events  (host) NULL, or 6 hipEvent_t handles (created with timing
 *                  enabled): start/stop of the attention kernel (without its
 *                  combine), of the vocabulary projection kernel (for more
 *                  than 64 rows the hidden repacking launch before it is
 *                  outside the pair) and
 *                  of the acceptance (one launch in a step: the segment sums,
 *                  then the draw by the last workgroup of each request).
 *                  They are recorded by the kernel
 *                  launches themselves (no extra work on the stream), so the
 *                  elapsed time of each pair is that span's execution time.
 */
SD_API int sd_verify_step(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                   const int64_t* kv_off, const int32_t* kv_len, float scale,
                   const void* hidden, const void* w_vocab, const float* q_draft,
                   const int32_t* draft_tok, const float* u, void* attn_out, float* logits,
                   float* row_lse, int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                   void* workspace, size_t workspace_bytes, sd_stream_t stream,
                   void* const* kernel_events);

/*
 * sd_verify_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The step's scratch is a static device
 * array of SD_STATIC_SCRATCH_BYTES per device, which the library holds on
 * every device it runs on until the process ends; the call itself allocates
 * nothing.  Arguments, layout and results are those of sd_verify_step (no
 * kernel events).  A problem whose step needs more scratch than
 * SD_STATIC_SCRATCH_BYTES (sd_workspace_bytes gives an upper bound) returns
 * SD_ERR_WORKSPACE before any device work.  Every call on one device shares
 * that device's array: calls that overlap on one device (other streams,
 * other host threads) race and must not be issued; calls in stream order are
 * fine, and no part of the array needs clearing between them.
 */
#define SD_STATIC_SCRATCH_BYTES ((size_t)96 << 20)
SD_API int sd_verify_step_static(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                                 const int64_t* kv_off, const int32_t* kv_len, float scale,
                                 const void* hidden, const void* w_vocab, const float* q_draft,
                                 const int32_t* draft_tok, const float* u, void* attn_out, float* logits,
                                 float* row_lse, int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                                 sd_stream_t stream);

/*
 * Sampled verification.  The test and correction of sd_accept_resample run on
 * a warped target p' instead of p (the Leviathan test of Sec. 2 is lossless
 * with respect to whichever target it is given).  q_draft must then hold the
 * distributions the drafts were actually drawn from, i.e. the draft model's
 * distributions warped the same way.  Warps of one row of target logits, in
 * this order:
 *   temperature T > 0     z = logit / T (T = 0 selects greedy, below);
 *   top_k >= 1 (0: off)   keep every token whose logit is >= the k-th largest
 *                         logit (ties of the k-th all kept; k >= V: off);
 *   top_p in (0, 1)       of the kept tokens, keep the smallest set
 *   (1: off)              {logit >= c} whose mass sum exp(z) reaches top_p
 *                         times the kept total;
 *   p'(v) = exp(z(v) - row_lse) on the kept set, 0 elsewhere.
 * Greedy (T = 0): p' is one-hot on the first (smallest id) largest logit, so
 * a draft is accepted iff it equals its row's argmax and the emitted token is
 * the argmax of row l + 1; u and q do not change the result.
 * "Order" is the order of float32 values with -0 below +0.  Logits must be
 * finite.  Masses are evaluated in float32 and summed as 64-bit fixed point
 * (2^(62 - ceil(log2 V)) per unit), so the cut is deterministic; it may differ
 * from a float64 evaluation only when top_p lies within about 1e-6 of a
 * cumulative mass.
 */
typedef struct {
  float temperature;  /* >= 0, finite */
  int32_t top_k;      /* >= 0 */
  float top_p;        /* in (0, 1] */
} sd_sampling_t;

/*
 * sd_accept_resample with a warped target.  Arguments as there, except:
 *   logits         [M][V] float32 target logits (never probabilities)
 *   row_lse        [M] float32 output: log sum over the kept set of exp(logit / T)
 *                  (greedy rows: 0)
 *   row_min_logit  [M] float32 output: the smallest kept logit; -inf when no cut
 *                  applies, +inf for greedy rows.  Together with row_lse it
 *                  defines p' exactly (see above).
 *   workspace      sd_workspace_bytes(dims, ...) bytes suffice.
 * The drafts' tests use p'(x_i) in float64 from the row's float32 cut and
 * normaliser; the correction uses the float32 p' with float64 sums, as in
 * sd_accept_resample.
 */
SD_API int sd_accept_resample_sampled(const sd_dims_t* dims, const sd_sampling_t* sampling, const float* logits,
                                      const float* q_draft, const int32_t* draft_tok, const float* u,
                                      const int32_t* kv_len, float* row_lse, float* row_min_logit,
                                      int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                                      void* workspace, size_t workspace_bytes, sd_stream_t stream);

/*
 * sd_verify_step with a warped target: attention, projection, then
 * sd_accept_resample_sampled on the logits it produced.  Arguments as in
 * sd_verify_step and sd_accept_resample_sampled; kernel_events' last pair
 * spans the warp kernel through the pick kernel.
 */
SD_API int sd_verify_step_sampled(const sd_dims_t* dims, const sd_sampling_t* sampling, const void* q,
                                  const void* k_pool, const void* v_pool, const int64_t* kv_off,
                                  const int32_t* kv_len, float scale, const void* hidden, const void* w_vocab,
                                  const float* q_draft, const int32_t* draft_tok, const float* u, void* attn_out,
                                  float* logits, float* row_lse, float* row_min_logit, int32_t* accept_len,
                                  int32_t* out_tok, int32_t* new_kv_len, void* workspace, size_t workspace_bytes,
                                  sd_stream_t stream, void* const* kernel_events);

/*
 * Tree verification: lossless acceptance of a candidate tree (Algorithm 2's
 * top-k proposal tree, whose longest-path rule as printed does not preserve
 * the target distribution).  dims->gamma is the number of nodes N; rows and
 * draws follow the positions of sd_verify_attention_tree (position 0 the
 * root, position i + 1 node i).
 *   logits_or_probs [B*(N+1)][V] float32, row_lse [B*(N+1)] or NULL: as in
 *                   sd_accept_resample (row g: the target after position g)
 *   tokens   [B][N] int32: node i's token (a token outside [0, V) never passes)
 *   parent   [B][N] int32: as in sd_verify_attention_tree
 *   u        [B][N+1] float32 in [0,1): u[b][i] tests node i, u[b][N] drives
 *            the final sample
 *   accept_len [B] int32 output: accepted nodes (the depth reached)
 *   out_tok  [B][N+1] int32 output: the accepted nodes' tokens, the final
 *            token, then -1
 *   out_node [B][N+1] int32 output: the accepted nodes in order, then -1
 *   new_kv_len [B] int32 output or NULL: kv_len[b] - N + accept_len[b] (the
 *            caller keeps the prefix, the root and the accepted nodes, moved
 *            into consecutive positions)
 *   workspace sd_workspace_bytes(dims, ...) bytes suffice.
 * Rule: candidates are point-mass proposals of the Leviathan test (Sec. 2).
 * At the current position (starting at the root) its children are tested in
 * node order: child c passes iff u[c] < p(token_c) / (1 - R), R the target
 * mass of the candidates rejected before it at this position (a token already
 * rejected there has mass 0); the first child that passes is accepted and the
 * walk moves to it.  When none passes (or there are none), the final token is
 * drawn by inverse CDF in ascending token id, with u[N], from that position's
 * p with the rejected candidates removed (float64 prefix sums; falls back to
 * p itself when rounding leaves no mass).  Every emitted token then follows
 * the target's next-token distribution; the draft distributions do not enter.
 */
SD_API int sd_accept_tree(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse,
                          const int32_t* tokens, const int32_t* parent, const float* u, const int32_t* kv_len,
                          int32_t* accept_len, int32_t* out_tok, int32_t* out_node, int32_t* new_kv_len,
                          void* workspace, size_t workspace_bytes, sd_stream_t stream);

/*
 * One whole tree verification step: sd_verify_attention_tree, sd_verify_logits
 * (row_lse is an output), then sd_accept_tree.  Arguments as in those calls
 * and sd_verify_step; kernel_events' last pair spans the tree walk (which
 * also folds the row log-sum-exps) through the final draw.
 */
SD_API int sd_verify_step_tree(const sd_dims_t* dims, const void* q, const void* k_pool, const void* v_pool,
                               const int64_t* kv_off, const int32_t* kv_len, const int32_t* parent, float scale,
                               const void* hidden, const void* w_vocab, const int32_t* tokens, const float* u,
                               void* attn_out, float* logits, float* row_lse, int32_t* accept_len, int32_t* out_tok,
                               int32_t* out_node, int32_t* new_kv_len, void* workspace, size_t workspace_bytes,
                               sd_stream_t stream, void* const* kernel_events);

/*
 * After a tree verification step: in every request's cache, move the K and V
 * rows of the accepted nodes (out_node[b][0..accept_len[b]) from
 * sd_accept_tree) into consecutive positions right after the root, in place,
 * so that the first new_kv_len[b] = kv_len[b] - N + accept_len[b] entries are
 * the verified sequence.  k_pool, v_pool, kv_off, kv_len as in
 * sd_verify_attention_tree; out_node [B][N+1], accept_len [B] (device).
 * Accept lengths or node numbers out of range end that request's move early.
 */
SD_API int sd_tree_commit_kv(const sd_dims_t* dims, void* k_pool, void* v_pool, const int64_t* kv_off,
                             const int32_t* kv_len, const int32_t* out_node, const int32_t* accept_len,
                             sd_stream_t stream);

/*
 * Acceptance rate of every draft position (Sec. 3, eq. beta_cond): the sum
 * over the vocabulary of min(p(v), q(v)), i.e. one minus the total-variation
 * distance of the target and draft distributions, which is the probability
 * that the ratio test accepts a draft drawn from q.  Its mean over positions
 * is the beta of the expected accept length beta (1 - beta^d) / (1 - beta)
 * (eq. El_closed) that the performance model of Sec. 3 builds on.
 *   logits_or_probs [B*G][V] float32 (device): logits if row_lse != NULL, else
 *                   probabilities; row b*G + i is the target distribution p
 *                   that tests draft position i (i < gamma)
 *   row_lse         [B*G] float32 (device) or NULL: p(v) = exp(logit - lse),
 *                   the difference kept exact, as in sd_accept_resample
 *   q_draft         [B][gamma][V] float32 (device): the draft distributions
 *   beta            [B][gamma] float64 (device) output
 *   workspace       at least sd_workspace_bytes(dims, ...) bytes, 16-byte aligned
 * min(p, q) is summed in float64 in an order fixed by the shapes, so repeated
 * calls give identical results.  Two kernel launches on `stream`.
 */
SD_API int sd_acceptance_rate(const sd_dims_t* dims, const float* logits_or_probs, const float* row_lse,
                              const float* q_draft, double* beta, void* workspace, size_t workspace_bytes,
                              sd_stream_t stream);

/*
 * Paged KV caches: per-session (per-tag) state in one shared pool
 * (Algorithm 1: each target's KV cache is isolated and indexed by its tag;
 * the session's cache is created with the session, grows by the gamma + 1
 * positions of every step, is cut back to the accepted prefix after it, and
 * is released at the end).  K and V each live in a pool of num_pages pages of
 * page_size keys, laid out [num_pages][n_kv_heads][page_size][head_dim]
 * (bf16).  Request b's key k is row k % page_size of page
 * block_table[b][k / page_size].  page_size is a power of two in [64, 4096],
 * so a 32-key attention tile never crosses a page.
 */
typedef struct {
  const int32_t* block_table; /* device [B][max_pages] int32 page ids; an id outside
                                 [0, num_pages) is clamped into it (never read out of bounds) */
  int32_t max_pages;          /* entries per request in block_table; kv_len[b] <= max_pages * page_size */
  int32_t page_size;          /* keys per page: a power of two in [64, 4096] */
  int32_t num_pages;          /* pages in each of the K and V pools */
} sd_kv_pages_t;

/*
 * sd_verify_attention over a paged cache: identical results to the segment
 * layout holding the same rows (same kernels; only the row addresses differ,
 * and the split of each request's keys into chunks is rounded to whole
 * pages).  k_pages, v_pages: the pools (16-byte aligned).  kv_len (host) as
 * for sd_verify_attention; the last G keys of request b are this step's
 * positions.  bf16 only (SD_ERR_UNSUPPORTED for fp32).
 */
SD_API int sd_verify_attention_paged(const sd_dims_t* dims, const void* q, const void* k_pages, const void* v_pages,
                                     const sd_kv_pages_t* pages, const int32_t* kv_len, float scale, void* out,
                                     void* workspace, size_t workspace_bytes, sd_stream_t stream);

/* sd_verify_step with the attention reading a paged cache; other arguments as there. */
SD_API int sd_verify_step_paged(const sd_dims_t* dims, const void* q, const void* k_pages, const void* v_pages,
                                const sd_kv_pages_t* pages, const int32_t* kv_len, float scale,
                                const void* hidden, const void* w_vocab, const float* q_draft,
                                const int32_t* draft_tok, const float* u, void* attn_out, float* logits,
                                float* row_lse, int32_t* accept_len, int32_t* out_tok, int32_t* new_kv_len,
                                void* workspace, size_t workspace_bytes, sd_stream_t stream,
                                void* const* kernel_events);

/*
 * Host-side page allocator of a paged pool (host memory only; no device
 * work; not thread-safe: one caller at a time per pool).  Sessions are
 * non-negative int32 tags.  Pages are handed out from a free list, lowest id
 * first when the pool is fresh, and a freed page is the next one handed out.
 *   sd_kv_pool_create      NULL if num_pages < 1 or page_size is not a power of two in [64, 4096]
 *   sd_kv_pool_reserve     grow `tag`'s pages to hold `length` keys (a new tag starts empty);
 *                          SD_ERR_CAPACITY, with nothing changed, if the free pages do not suffice
 *   sd_kv_pool_truncate    keep the pages holding keys [0, length), free the rest
 *                          (the roll-back to new_kv_len after a step)
 *   sd_kv_pool_release     free all of `tag`'s pages and forget it
 *   sd_kv_pool_free_pages  free pages in the pool
 *   sd_kv_pool_tag_pages   pages `tag` holds (0 for an unknown tag)
 *   sd_kv_pool_block_table (host) table [n][max_pages]: row i lists tags[i]'s pages in key
 *                          order, then -1; SD_ERR_INVALID_ARGUMENT if a tag holds more than max_pages
 * Negative tags or lengths give SD_ERR_INVALID_ARGUMENT.
 */
typedef struct sd_kv_pool sd_kv_pool_t;
SD_API sd_kv_pool_t* sd_kv_pool_create(int32_t num_pages, int32_t page_size);
SD_API void sd_kv_pool_destroy(sd_kv_pool_t* pool);
SD_API int sd_kv_pool_reserve(sd_kv_pool_t* pool, int32_t tag, int32_t length);
SD_API int sd_kv_pool_truncate(sd_kv_pool_t* pool, int32_t tag, int32_t length);
SD_API int sd_kv_pool_release(sd_kv_pool_t* pool, int32_t tag);
SD_API int32_t sd_kv_pool_free_pages(const sd_kv_pool_t* pool);
SD_API int32_t sd_kv_pool_tag_pages(const sd_kv_pool_t* pool, int32_t tag);
SD_API int sd_kv_pool_block_table(const sd_kv_pool_t* pool, const int32_t* tags, int32_t n, int32_t max_pages,
                                  int32_t* table);

/*
 * Draft-side tree expansion, batched over pooled requests (Algorithm 2,
 * ExpandLayer: the draft model grows its proposal tree one layer at a time,
 * every frontier node taking the top-k tokens of the draft's next-token
 * distribution there as children, and keeps their draft probabilities for
 * the correction step).  The draft model's forward pass is the caller's; this
 * call turns its logits at the frontier into the next layer of the tree
 * arrays that sd_verify_step_tree consumes.
 *   draft_logits  [B][F][V] float32 (device): row (b, f) holds the draft's logits
 *                 at frontier node frontier0 + f of request b (finite or -inf,
 *                 at least one finite per row)
 *   tokens, parent [B][N] int32 (device), q_child [B][N] float32 (device):
 *                 entries first_child + f*k + j, j < k, are written: the j-th
 *                 ranked token of row (b, f), its parent frontier0 + f (-1 when
 *                 frontier0 = -1, i.e. the frontier is the root), and its draft
 *                 probability exp(logit - logsumexp(row)); nothing else is written
 * Rank: larger float32 logit first (-0 below +0), equal logits by increasing
 * token id.  Requires 1 <= k <= min(V, 16), first_child + F*k <= N and, for
 * frontier0 >= 0, frontier0 + F <= first_child (parents precede children).
 * For a full k-ary tree numbered layer by layer: layer 1 (frontier0 = -1,
 * first_child = 0, F = 1), layer t + 1 (frontier0 = first_child of layer t,
 * F = k^t, first_child = that plus k^t).
 */
typedef struct {
  int32_t batch;        /* B requests */
  int32_t frontier;     /* F frontier nodes per request */
  int32_t vocab;        /* V */
  int32_t top_k;        /* k children per frontier node */
  int32_t frontier0;    /* tree index of frontier node 0, -1 for the root */
  int32_t first_child;  /* tree index of the first new node */
  int32_t nodes;        /* N: entries per request in tokens, parent and q_child */
} sd_expand_t;
SD_API int sd_expand_layer(const sd_expand_t* e, const float* draft_logits, int32_t* tokens, int32_t* parent,
                           float* q_child, sd_stream_t stream);

/*
 * Name of the vocabulary-projection kernel that sd_verify_logits and the
 * verification steps launch for `dims`, as a kernel trace lists it without
 * template arguments ("vocab_bf16_kernel", "vocab_bf16_deep_kernel",
 * "vocab_bf16_wide_kernel" or "vocab_f32_kernel"): for tools that match
 * measurements to kernels.  Host only; a static string, or NULL for an
 * invalid shape.
 */
SD_API const char* sd_vocab_kernel_name(const sd_dims_t* dims);

/* Static description of a status code. */
SD_API const char* sd_status_string(int status);

/* Library version, "major.minor.patch". */
SD_API const char* sd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SDVERIFY_H */
