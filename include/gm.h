/*
 * gm.h -- C ABI of the batched speculative-decoding step (MI355X / gfx950).
 *
 * One step of speculative rollout generation for a batch of B sequences
 * (GrowMTP, Sec. 2.2): the target verifies a block of k+1 positions per
 * sequence in one forward (gm_verify_forward, gm_verify_attention), accepts a
 * prefix of the k drafts and draws one more token (gm_spec_accept), commits
 * the accepted KV entries and rolls back the rest (gm_kv_commit), and the MTP
 * draft head proposes the next block (gm_mtp_draft).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers unless a comment says "host".  Every buffer
 *   is owned by the caller; no call keeps a pointer after it returns and no
 *   call allocates or frees device memory.  Scratch memory is passed in as a
 *   workspace whose size gm_workspace_size() reports.
 * - Every call enqueues its kernels on `stream` (a hipStream_t; NULL is the
 *   null stream) and returns without waiting for them.
 * - Shapes and arguments are validated on the host before anything is
 *   launched; a failed check returns a negative gm_status, launches nothing
 *   and leaves a message for gm_last_error().  Faults that only the device
 *   can see (a token id outside the vocabulary, a block-table entry outside
 *   the page pool) are reported through the optional `dev_err` word: the
 *   kernel ORs a GM_DEVERR_* bit into it and skips the offending access.
 * - Outputs are bit-deterministic for fixed inputs (no reduction depends on
 *   the order of atomics).
 * - Token ids are int32.  Logits, uniforms and hidden states are float32.
 *   Weights and KV entries use the model dtype: GM_F32 (float) or GM_BF16
 *   (bfloat16 stored as uint16).  Norm weights use the model dtype too.
 * - Block layout: block position i of sequence b (0 <= i <= k) is absolute
 *   position m_b + i, where m_b = seq_lens[b] is the committed length; the
 *   block is [t_m, d_1 .. d_k]: the pending token (drawn by the last cycle,
 *   not yet in the cache) followed by the k drafts.
 */
#ifndef GM_H
#define GM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GM_OK = 0,
  GM_ERR_INVALID_ARG = -1,   /* null pointer, bad size or shape */
  GM_ERR_UNSUPPORTED = -2,   /* a valid configuration this build does not implement */
  GM_ERR_CAPACITY = -3,      /* the KV page table cannot hold the positions the call writes */
  GM_ERR_WORKSPACE = -4,     /* workspace missing or smaller than gm_workspace_size() */
  GM_ERR_DEVICE = -5         /* a HIP runtime call failed */
} gm_status;

enum { GM_DEVERR_TOKEN = 1, GM_DEVERR_PAGE = 2 };

typedef enum { GM_F32 = 0, GM_BF16 = 1 } gm_dtype;
typedef enum { GM_GREEDY = 0, GM_SAMPLE = 1 } gm_accept_mode;
typedef enum {
  GM_OP_VERIFY_FORWARD = 0,
  GM_OP_VERIFY_ATTENTION = 1,
  GM_OP_SPEC_ACCEPT = 2,
  GM_OP_MTP_DRAFT = 3,
  GM_OP_DCA_LOSS = 4,    /* B = cycles N, k = draft length K, cfg->vocab = V */
  GM_OP_MTP_RECONSTRUCT = 5   /* B = cycles R, k = depth K, max_ctx = the cache's max_ctx */
} gm_op;

/* Decoder shape: pre-norm RMSNorm / RoPE (rotate-half, angle pos * base^(-2i/d))
 * / grouped-query attention / SwiGLU, the layer of the paper's backbones
 * (App. "Models and Draft Heads").  Limits of this build: head_dim 128 for
 * GM_BF16 (64 or 128 for GM_F32), n_heads a multiple of n_kv_heads with
 * (n_heads / n_kv_heads) * (k + 1) <= 64, hidden and ffn multiples of 64,
 * hidden and (n_heads + 2 n_kv_heads) * head_dim at most 16384, vocab at
 * most 524288 (also the limit of gm_spec_accept's V);
 * GM_BF16 needs vocab a multiple of 128 and hidden, ffn and
 * n_heads * head_dim multiples of 256. */
typedef struct {
  int n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  float rope_base;       /* 10000 */
  float rms_eps;         /* 1e-6 */
  int dtype;             /* gm_dtype */
  int qk_norm;           /* 1: per-head RMSNorm of q and k before RoPE (Qwen3) */
  int tie_embed;         /* informational: lm_head may alias embed */
} gm_model_config;

/* One decoder layer.  A linear weight W[out][in] (y = W x) is stored
 *  - GM_F32: row-major;
 *  - GM_BF16: tiled, in tiles of 16 rows x 32 columns (out a multiple of 128):
 *    element (n, c) at
 *      (((n / 128) * (in / 32) + c / 32) * 8 + (n / 16) % 8) * 512
 *        + ((c % 32) / 8) * 128 + (n % 16) * 8 + c % 8,
 *    so that each 1 KiB tile is read by one 16-byte-per-lane load of a
 *    64-lane wave in the operand order of the matrix cores, and the tiles of
 *    8 consecutive 16-row strips at one 32-column step are consecutive (the
 *    strips streamed together are one contiguous run per step).  (Row-major W
 *    converts to this layout by viewing it as [out/128][8][16][in/32][4][8]
 *    and permuting to [out/128][in/32][8][4][16][8].)
 * The tiled layout applies to w_qkv, w_o, w_gate_up, w_down, the MTP w_proj
 * and lm_head; embeddings and norm weights are plain vectors / row-major. */
typedef struct {
  const void *attn_norm;  /* [H] */
  const void *w_qkv;      /* [(n_heads + 2 n_kv_heads) head_dim, H]: the rows of W_q, then W_k, then W_v */
  const void *q_norm;     /* [head_dim], or NULL when qk_norm == 0 */
  const void *k_norm;     /* [head_dim], or NULL when qk_norm == 0 */
  const void *w_o;        /* [H, n_heads head_dim] */
  const void *ffn_norm;   /* [H] */
  const void *w_gate_up;  /* [2 ffn, H]: the rows of W_gate, then W_up */
  const void *w_down;     /* [H, ffn] */
} gm_layer_weights;

typedef struct {
  const void *embed;                /* [vocab, H] */
  const void *final_norm;           /* [H] */
  const void *lm_head;              /* [vocab, H] */
  const gm_layer_weights *layers;   /* host array [n_layers] */
} gm_model_weights;

/* The recurrent MTP draft head (App. "Models and Draft Heads"): RMSNorm_h of
 * the conditioning hidden and RMSNorm_e of the token embedding, concatenated
 * hidden first, a bias-free projection 2H -> H, one decoder layer with a KV
 * cache of its own, a final RMSNorm and the backbone's LM head. */
typedef struct {
  const void *norm_h;      /* [H] */
  const void *norm_e;      /* [H] */
  const void *w_proj;      /* [H, 2H]: columns 0..H-1 act on RMSNorm_h(h), H..2H-1 on RMSNorm_e(E[t]) */
  const void *final_norm;  /* [H] */
  gm_layer_weights layer;
} gm_mtp_weights;

/* Paged KV cache.  Each layer owns two page pools, K and V, each
 * [num_pages][n_kv_heads][page_size * head_dim] elements of the model dtype.
 * Position t of sequence b lives in page block_table[b][t / page_size] at
 * offset t % page_size.  Inside the block of one (page, kv head) the tokens
 * come in tiles of 16 (tile j holds offsets 16j .. 16j+15) of 16 * head_dim
 * elements, and inside a tile (token s = 0..15, channel c = 0..head_dim-1):
 *   K element at  (c / 32) * 512 + ((c % 32) / 8) * 128 + s * 8 + c % 8
 *   V element at  (c / 32) * 512 + (s / 4) * 128 + (c % 16) * 8 + ((c / 16) % 2) * 4 + s % 4
 * so that one 64-lane load of 16 bytes per lane reads 1 KiB of the tile in
 * the order the matrix-core operands take it.  page_size is a multiple of 16. */
typedef struct {
  void *const *k_pages;        /* host array [n_layers] of device bases */
  void *const *v_pages;        /* host array [n_layers] of device bases */
  int n_layers;
  int page_size;
  int num_pages;
  int max_pages_per_seq;
  const int32_t *block_table;  /* [B][max_pages_per_seq] */
  int32_t *seq_lens;           /* [B] committed lengths m_b */
  int max_ctx;                 /* host: an upper bound on every seq_lens[b] */
} gm_kv_cache;

/* Softmax statistics of one logits row z at temperature T: the max of z / T,
 * the lowest id attaining it, and sum over ids of exp(z / T - max).
 * gm_mtp_draft can emit them for its draft logits; gm_spec_accept can take them
 * in place of its own pass over those rows (q's normaliser, Sec. 2.2). */
typedef struct {
  float max;
  int32_t argmax;
  double sum;
} gm_row_stats;

/* Top-p: the nucleus of one logits row (see gm_spec_accept's top_p): the kept ids are
 * those whose logit's order key exceeds `key`, and those with that key up to id
 * `last_id`; `mass` is sum over them of exp(z / T - m).  (The order key of a float32
 * x: its bits with the sign bit set if x >= 0, all bits inverted if x < 0; -0 as +0.)
 * gm_mtp_draft can emit them for its draft rows under top-p; gm_spec_accept can take
 * them in place of its own passes over those rows. */
typedef struct {
  double m;
  double mass;
  uint32_t key;
  int32_t last_id;
} gm_nucleus;

/* The cycle record's verification distributions (App. "Implementing Draft-Path
 * Reconstruction in verl", recording in rollout): for every sequence b and draft
 * position i < k, the `topk` largest entries of p_i = softmax(target_logits[b][i] / T),
 * as log p_i (normalised over the whole vocabulary, not over the kept entries)
 * rounded to bf16, and their ids; in decreasing probability, equal probabilities
 * in increasing id.  (The record's other items -- the drafts, the accepted
 * length, the start position and the hidden at the cycle's start -- are inputs
 * or outputs of the step already.) */
typedef struct {
  int topk;           /* 1..64, at most V */
  uint16_t *logp;     /* [B][k][topk] bf16 */
  int32_t *ids;       /* [B][k][topk] */
} gm_record;

/* Bytes of workspace the given call needs (0 on invalid arguments).
 * `max_ctx` is the bound that the call's gm_kv_cache carries. */
size_t gm_workspace_size(int op, const gm_model_config *cfg, int B, int k, int max_ctx);

/* Verification forward (Sec. 3.1, Eq. verification-context; App.
 * "Draft-Path Reconstruction": one target forward over the draft path).
 * tokens [B][k+1] is the block [t_m, d_1..d_k].  Writes the K/V entries of
 * the block at positions m_b .. m_b+k of every layer (seq_lens is not
 * changed: gm_kv_commit decides what stays), logits [B][k+1][vocab] float32
 * (row i is the target's distribution for the token after block position i)
 * and hidden [B][k+1][H] float32, the last layer's output before the final
 * RMSNorm (the feature the MTP head consumes).
 * target_stats [B][k+1] (may be NULL): also the softmax statistics of every
 * logits row at `temperature` (gm_row_stats), taken in the LM head's epilogue;
 * gm_spec_accept takes them for the same rows and temperature in place of its
 * pass over the target rows (Sec. 2.2, Eq. accept-rule: p's normaliser and
 * arg-max).  temperature is read only when target_stats is given (> 0).
 * Errors: GM_ERR_CAPACITY if max_ctx + k + 1 > max_pages_per_seq * page_size;
 * GM_ERR_INVALID_ARG for target_stats with temperature <= 0. */
gm_status gm_verify_forward(const gm_model_config *cfg, const gm_model_weights *w,
                            const gm_kv_cache *cache, int B, int k, const int32_t *tokens,
                            float *logits, float *hidden, float temperature, gm_row_stats *target_stats,
                            void *ws, size_t ws_bytes, int32_t *dev_err, void *stream);

/* Verify attention of one layer: the query at block position i of sequence b
 * attends causally to cache positions 0 .. m_b + i (the committed prefix and
 * block positions 0..i, which must already be in the cache), scale
 * 1/sqrt(head_dim), query head h reading KV head h / (n_heads / n_kv_heads).
 * q and out are [B][k+1][n_heads][head_dim] in the model dtype; q is after
 * RoPE. */
gm_status gm_verify_attention(const gm_model_config *cfg, const gm_kv_cache *cache, int layer,
                              int B, int k, const void *q, void *out, void *ws, size_t ws_bytes,
                              int32_t *dev_err, void *stream);

/* Accept rule (Sec. 2.2, Eq. accept-rule).  p_i = softmax(target_logits[b][i] / T),
 * q_i = softmax(draft_logits[b][i] / T).
 * GM_SAMPLE: scanning i = 0..k-1, draft d_i is accepted iff u_accept[b][i] <
 *   p_i(d_i) / q_i(d_i) (ratio rounded to float32); the scan stops at the
 *   first rejection.  With n accepted, the final token is an inverse-CDF draw
 *   with u_final[b] (smallest id x with sum_{y<=x} w(y) > u * sum w) from
 *   w = max(0, p_n - q_n) if n < k (from p_n if that mass is 0), or from
 *   w = p_k (bonus token) if n = k.
 * GM_GREEDY: d_i is accepted iff it is the argmax of target_logits[b][i]
 *   (lowest id on ties); the final token is the argmax of row n.
 *   draft_logits, draft_stats, u_accept and u_final may be NULL.
 * top_p in (0, 1] (GM_SAMPLE; the evaluation setting of App. "Evaluation
 *   Configuration" decodes at T = 1, top-p 0.7): below 1, every p_i and q_i is
 *   replaced by its nucleus before the rule -- the ids ranked by logit (larger
 *   first, the lower id first among equal logits) up to the first at which the
 *   running probability reaches top_p, renormalised -- so the drafts must be
 *   samples of the head's nucleus (gm_mtp_draft with the same top_p).  The
 *   running masses are exact sums of float64 exponentials rounded to 2^-44 of
 *   the row maximum's term.  GM_GREEDY ignores top_p; 1 keeps every id.
 *   GM_ERR_INVALID_ARG outside (0, 1].
 * draft_nucleus [B][k] (may be NULL; read in GM_SAMPLE mode with top_p < 1 only): the
 *   nuclei of the draft_logits rows at this T and top_p, as gm_mtp_draft writes them.
 *   Given, they stand in for the passes over the draft rows (their statistics and
 *   their nucleus); the caller guarantees that they describe these draft_logits.
 * draft_stats [B][k] (may be NULL; read in GM_SAMPLE mode only): the statistics
 *   of softmax(draft_logits[b][i] / T) at this temperature, as gm_mtp_draft
 *   writes them.  Given, they stand in for a pass over the draft rows; the
 *   caller guarantees that they describe these draft_logits.
 * target_stats [B][k+1] (may be NULL): the statistics of softmax(target_logits[b][i] / T)
 *   at this temperature, as gm_verify_forward writes them.  Given, they stand in for
 *   the pass over the target rows (that pass still runs when a record is requested,
 *   whose selection needs it); the caller guarantees that they describe these
 *   target_logits.
 * Outputs: n_accept [B] in [0, k]; out_tokens [B][k+1] = d_0..d_{n-1}, final, -1 pad.
 * record (host struct, may be NULL): also writes the cycle record's top-k
 *   log-probabilities of the target rows 0..k-1 (see gm_record), taken in the same
 *   pass over the target logits.  GM_ERR_INVALID_ARG if topk is outside 1..min(64, V)
 *   or a record buffer is NULL.
 * The logits rows are read in place; no probability matrix is written. */
gm_status gm_spec_accept(int B, int k, int V, int mode, float temperature, float top_p,
                         const float *target_logits, const float *draft_logits,
                         const gm_row_stats *target_stats, const gm_row_stats *draft_stats,
                         const gm_nucleus *draft_nucleus,
                         const int32_t *draft_tokens, const float *u_accept, const float *u_final,
                         int32_t *n_accept, int32_t *out_tokens, const gm_record *record, void *ws,
                         size_t ws_bytes, void *stream);

/* gm_spec_accept for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same arguments and
 * results, without the workspace.  Its scratch is a fixed 16 MiB device array that
 * each GPU the library runs on holds until the process ends; the call allocates and
 * frees nothing.  Limit: calls whose gm_workspace_size(GM_OP_SPEC_ACCEPT, ...) exceeds
 * 16 MiB return GM_ERR_CAPACITY before touching the device (B = 256 sequences at
 * k = 7, V = 151936 fit, top-p included).  Every call on one GPU shares that GPU's
 * scratch: calls that overlap in time on one GPU (other streams, other threads) race
 * and must be serialised by the caller.  GM_ERR_DEVICE if the scratch's device
 * address cannot be obtained on the current device. */
gm_status gm_spec_accept_noalloc(int B, int k, int V, int mode, float temperature, float top_p,
                                 const float *target_logits, const float *draft_logits,
                                 const gm_row_stats *target_stats, const gm_row_stats *draft_stats,
                                 const gm_nucleus *draft_nucleus, const int32_t *draft_tokens,
                                 const float *u_accept, const float *u_final, int32_t *n_accept,
                                 int32_t *out_tokens, const gm_record *record, void *stream);

/* Commit / rollback (Sec. 2.2; App. "Train--Inference Inconsistency under
 * Teacher Forcing", Eq. tf-restart-kv): block positions 0..n_b stay, the rest
 * are rolled back by index only (no KV bytes move): seq_lens[b] += n_b + 1.
 * committed_slots [B][k+1] (may be NULL) receives the physical slot
 * (page * page_size + offset) of each committed block position, -1 for rolled
 * back ones. */
gm_status gm_kv_commit(const gm_kv_cache *cache, int B, int k, const int32_t *n_accept,
                       int32_t *committed_slots, void *stream);

/* MTP draft of the next block (Sec. 2.2; App. "Models and Draft Heads";
 * Eqs. tf-restart, tf-restart-kv).  mtp_cache is a one-layer cache whose
 * seq_lens hold the head's committed length, equal to the target's committed
 * length before the last verification.  Slot s of the head's cache holds the
 * entry of the pair (h_s, x_{s+1}) rotated at position s+1, where h_s is the
 * target hidden at position s.  Extend: the n_b+1 rows (verify_hidden[b][i],
 * out_tokens[b][i]), i = 0..n_b, are written at slots m_b..m_b+n_b and the
 * head's length becomes m_b+n_b+1 (the entries behind the boundary come from
 * target features).  The output of row n_b gives q_1; chain step j feeds
 * (layer output of step j-1, draft j-1) at slot m_b+n_b+j; those entries lie
 * past the committed length and are overwritten by the next extend.
 * Drafts are argmax (GM_GREEDY) or inverse-CDF draws with u_draft[b][j]
 * (GM_SAMPLE) from softmax(z / T).  Outputs: drafts [B][k],
 * draft_logits [B][k][vocab] float32, and (if draft_stats is not NULL)
 * draft_stats [B][k], the softmax statistics of each draft_logits row at T
 * (the draw's own; gm_spec_accept takes them for the same rows and T).
 * top_p in (0, 1] (GM_SAMPLE): below 1, each draft is the inverse-CDF draw with
 * u_draft[b][j] from the nucleus of softmax(z / T) (as in gm_spec_accept);
 * draft_stats must then be NULL (GM_ERR_UNSUPPORTED otherwise); draft_nucleus [B][k]
 * (may be NULL) receives the nucleus of every draft_logits row (gm_spec_accept takes
 * them for the same rows, T and top_p).  With top_p = 1 or GM_GREEDY it is not written.
 * Errors: GM_ERR_CAPACITY if max_ctx + 2k + 1 > max_pages_per_seq * page_size
 * of the head's cache; GM_ERR_INVALID_ARG for top_p outside (0, 1]. */
gm_status gm_mtp_draft(const gm_model_config *cfg, const gm_mtp_weights *mtp,
                       const gm_model_weights *shared, const gm_kv_cache *mtp_cache, int B, int k,
                       int mode, float temperature, float top_p, const float *verify_hidden,
                       const int32_t *n_accept, const int32_t *out_tokens, const float *u_draft,
                       int32_t *drafts, float *draft_logits, gm_row_stats *draft_stats,
                       gm_nucleus *draft_nucleus, void *ws,
                       size_t ws_bytes, int32_t *dev_err, void *stream);

/* Draft-path reconstruction (App. "Draft-Path Reconstruction"; App. "Parallelizing
 * GrowMTP Training"): the head's chain of each of R recorded cycles re-run under the
 * current head weights with the recorded drafts as inputs and nothing sampled, as K
 * batched single-row steps (one per depth, all cycles together).  mtp_cache is a
 * one-layer cache with one block table row per cycle; seq_lens[r] = s_r, the number of
 * committed head entries the cycle sees (slot s holds the pair (h_s, x_{s+1}) rotated
 * at position s+1, as gm_mtp_draft writes them).  Depth 1 feeds (start_hidden[r],
 * start_tokens[r]) -- the boundary hidden and the last committed token the cycle
 * started from -- at slot s_r; depth j >= 2 feeds (its layer output at depth j-1,
 * drafts[r][j-2]) at slot s_r + j - 1.  Depth j attends to slots 0 .. s_r + j - 1 of the
 * cycle's own table: causal over the committed prefix, its own chain's entries (the
 * diagonal mask of the batched form).  The entries at slots s_r .. s_r + K - 1 are
 * written, so those pages must be the cycle's own (cycles may share the pages of their
 * prefix).  seq_lens is not changed.
 * start_hidden [R][H] float32; start_tokens [R]; drafts [R][K] (d_1..d_{K-1} are read;
 * may be NULL when K = 1); head_logits [R][K][vocab] float32: row j is the head's
 * logits at depth j+1 (q_{r,j+1} = softmax of it), the input of gm_dca_loss.
 * Errors: GM_ERR_CAPACITY if max_ctx + K > max_pages_per_seq * page_size. */
gm_status gm_mtp_reconstruct(const gm_model_config *cfg, const gm_mtp_weights *mtp,
                             const gm_model_weights *shared, const gm_kv_cache *mtp_cache, int R, int K,
                             const float *start_hidden, const int32_t *start_tokens, const int32_t *drafts,
                             float *head_logits, void *ws, size_t ws_bytes, int32_t *dev_err, void *stream);

/* Depth-coupled acceptance loss with verify-gated masking, and its gradient in
 * the head logits (Sec. "The Depth-Coupled Acceptance Loss" and "Learning up to
 * the First Rejection", Eqs. alpha, chain, dca, vgm; App. "DCA"), over the cycle
 * record's sparse support (App. "Implementing Draft-Path Reconstruction in
 * verl").  For cycle n and draft position k: q = softmax(head_logits[n][k]) over
 * the whole vocabulary, gathered at the record's ids S; p = exp(rec_logp); one
 * residual bin holds the mass outside S, p_R = max(0, 1 - sum_S p), q_R = 1 - sum_S q.
 *   alpha[n][k] = sum_S min(p, q) + min(p_R, q_R)
 *   loss[n]     = -log sum_{l=1}^{L} prod_{i<=l} alpha[n][i],
 *                 L = min(n_accept[n] + 1, K) if vgm, else K
 * grad (may be NULL) [N][K][V]: d loss[n] / d head_logits[n][k][x] (positions past
 * L get 0; the subgradient of min is 0 where its arguments are equal).
 * head_logits [N][K][V] float32; rec_logp [N][K][topk] bf16; rec_ids [N][K][topk]
 * (distinct ids in 0..V-1; an id outside gets q = 0 and is never read); n_accept [N] in 0..K.
 * loss [N] and alpha [N][K] are float32 (computed in float64); grad is float32.
 * Limits: 1 <= K <= 15, 1 <= topk <= min(64, V), V <= 524288. */
gm_status gm_dca_loss(int N, int K, int V, int topk, const float *head_logits, const uint16_t *rec_logp,
                      const int32_t *rec_ids, const int32_t *n_accept, int vgm, float *loss, float *alpha,
                      float *grad, void *ws, size_t ws_bytes, void *stream);

/* Thread-local message describing the last non-OK status of this thread. */
const char *gm_last_error(void);

/* Kernel timing.  While tracing is on, every kernel the library launches
 * whose name matches `filter` (all kernels when NULL) is bracketed by a pair
 * of HIP events on its stream.  gm_trace_stop() waits for the recorded events
 * and sums their durations per kernel name.  The events record timestamps
 * only (no system-scope fence); each still leaves the stream idle for a few
 * microseconds.  gm_trace_every(n) (n >= 1, else GM_ERR_INVALID_ARG; default
 * 1) brackets only every n-th matching launch, counted from gm_trace_start, so
 * that a timing sample perturbs fewer launches. */
gm_status gm_trace_every(int n);
gm_status gm_trace_start(const char *filter);
gm_status gm_trace_stop(void);
int gm_trace_count(void);
gm_status gm_trace_get(int i, const char **name, int *launches, double *total_ms);

#ifdef __cplusplus
}
#endif
#endif /* GM_H */
