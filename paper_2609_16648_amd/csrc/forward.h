// Internal interfaces of the verify forward, verify attention and MTP draft.
#pragma once

#include "../../include/gm.h"
#include "launch.h"

namespace gm {

constexpr int kMaxRowFloats = 16384;   // float32 row that the row kernels stage in LDS (64 KiB)
constexpr int kAttnMaxRows = 64;   // (n_heads / n_kv_heads) * block rows per KV head
constexpr int kAttnMaxSplitTokens = 4096;                           // tokens of one workgroup's range
constexpr int kAttnMaxSplitPages = kAttnMaxSplitTokens / 16 + 8;    // pages one range can touch

struct Carve {
  size_t off = 0;
  size_t take(size_t n) {
    size_t o = off;
    off += (n + 255) & ~size_t(255);
    return o;
  }
};

// ---------------------------------------------------------------- attention
struct AttnPlan {
  int parts;           // ranges the tiles of all sequences are cut into (workgroups per head group)
  int rows_pad;        // 16-row tiles * 16
  size_t part_o, part_ml, cum, total;
};
AttnPlan plan_attention(const gm_model_config &cfg, int B, int R, int max_ctx);

struct AttnArgs {
  int dtype, B, R, n_heads, n_kv, head_dim;
  int page_size, max_pages, num_pages;
  const void *k_pages, *v_pages;
  const int32_t *block_table;
  const int32_t *base_lens;   // block start of sequence b: base_lens[b] + base_off
  int base_off;
  const int32_t *blk_len;     // rows of the block that are valid (< R), or null: all R
  int blk_len_add;            // valid rows = blk_len[b] + blk_len_add
  const void *q;              // [B][R][n_heads][head_dim] model dtype, after RoPE
  void *out;                  // [B][R][n_heads][head_dim] model dtype
  int32_t *dev_err;
  float scale;                // 1 / sqrt(head_dim)
  const char *trace, *trace_combine;   // kernel names for gm_trace
};
AttnArgs attn_args(const gm_model_config &cfg, const gm_kv_cache &c, int layer, int B, int R,
                   const int32_t *base_lens, int base_off, const int32_t *blk_len);
void run_attention(const AttnArgs &a, const AttnPlan &p, char *ws, hipStream_t s);

// ---------------------------------------------------------------- GEMM  Y[M,N] = X[M,K] W[N,K]^T
enum GemmEpi {
  EPI_STORE_F32 = 0,   // Y (float) = acc
  EPI_ADD_F32 = 1,     // Y (float) += acc
  EPI_STORE_ACT = 2,   // Y (model dtype) = acc
  EPI_SWIGLU = 3,      // W = [W_gate; W_up] (2N rows); Y (model dtype)[m][n] = silu(gate) * up
  EPI_STATS = 4        // Y (float) = acc, plus softmax statistics of Y / T per 128-column tile
};
struct GemmPlan {
  int shape, Nw, n_tiles, m_tiles, k_iters, splits;
  int cw;              // compute waves per workgroup (4, 5, 7: 128-, 160-, 224-column tiles)
  size_t part_bytes;   // float32 K-split partials
};
GemmPlan plan_gemm(int dtype, int epi, int M, int N, int K);
// bf16: W pre-tiled (gm.h), X row-major [M][ldx]; `part` must hold plan_gemm().part_bytes.
// Returns the K splits; with defer_reduce and more than one split, no reduce runs and
// the partials stay in `part` ([splits][M][Nw] float32) for the consumer to sum.
int launch_gemm(const char *name, int dtype, int epi, int M, int N, int K, const void *X, int ldx,
                const void *W, void *Y, long ldy, float *part, hipStream_t s,
                RowStat *tile_stats = nullptr, float inv_t = 1.f, bool defer_reduce = false);
// tile geometry of the softmax statistics an EPI_STATS launch at M rows emits (the draw reads it);
// *strips_kernel: whether the persistent strip-range kernel runs
TileGeom plan_lm_head(int dtype, int M, int V, int K, bool *strips_kernel = nullptr);
// Y[M][N] (+)= sum of `splits` partials, then out = RMSNorm(Y) * norm_w (epi: STORE_F32 or ADD_F32)
void launch_reduce_norm(int dtype, int epi, int M, int N, int splits, const float *part, float *Y,
                        const void *norm_w, float eps, void *out, hipStream_t s);

// ---------------------------------------------------------------- row kernels
void launch_embed(int dtype, int M, int H, int V, const int32_t *tokens, const void *E, float *x,
                  int32_t *dev_err, hipStream_t s);
void launch_rmsnorm(int dtype, int M, int H, float eps, const float *x, const void *w, void *out,
                    hipStream_t s);
// x = E[tokens] (float32) and out = RMSNorm(x) * norm_w (model dtype)
void launch_embed_norm(int dtype, int M, int H, int V, const int32_t *tokens, const void *E, float *x,
                       const void *norm_w, float eps, void *out, int32_t *dev_err, hipStream_t s);
struct RopeArgs {
  int dtype, M, R, n_heads, n_kv, head_dim;
  const float *qkv;            // [M][(n_heads + 2 n_kv) head_dim], or, with splits > 1,
  const float *part;           // the projection's K-split partials [splits][M][...] to sum
  int splits;
  void *q_out;                 // [M][n_heads][head_dim]
  void *k_pages, *v_pages;
  const int32_t *block_table;
  int page_size, max_pages, num_pages;
  const int32_t *base_lens;
  int base_off;
  const int32_t *blk_len;
  int blk_len_add;
  int pos_off;                 // rotary position = slot + pos_off
  float rope_base, eps;
  const void *q_norm, *k_norm; // or null
  int32_t *dev_err;
};
void launch_rope_append(const RopeArgs &a, hipStream_t s);

// DCA loss with verify-gated masking over the cycle record (dca.hip)
size_t dca_workspace(int N, int K, int V);
void run_dca_loss(int N, int K, int V, int topk, const float *head_logits, const uint16_t *rec_logp,
                  const int32_t *rec_ids, const int32_t *n_accept, int vgm, float *loss, float *alpha, float *grad,
                  char *ws, hipStream_t s);
void launch_mtp_input(int dtype, int M, int H, int V, float eps, const float *h, const int32_t *tok,
                      int tok_stride, const void *E, const void *norm_h, const void *norm_e, void *out,
                      int32_t *dev_err, hipStream_t s);
// per sequence b: row sel[b] (clamped to 0..R-1) of src_a [B][R][Ca] and of src_b [B][R][Cb]
// into dst_a [B][Ca] and dst_b [B][Cb], and lens[b] += sel[b] + 1 (clamped alike)
void launch_gather_commit(int B, int R, int Ca, size_t elem_a, const void *src_a, void *dst_a, int Cb, size_t elem_b,
                          const void *src_b, void *dst_b, const int32_t *sel, int32_t *lens, hipStream_t s);

// ---------------------------------------------------------------- accept (api.cpp)
// the accept with a given workspace (validation included); shared by the entry points
gm_status spec_accept_impl(int B, int k, int V, int mode, float temperature, float top_p, const float *target_logits,
                           const float *draft_logits, const gm_row_stats *target_stats, const gm_row_stats *draft_stats,
                           const gm_nucleus *draft_nucleus, const int32_t *draft_tokens, const float *u_accept,
                           const float *u_final, int32_t *n_accept, int32_t *out_tokens, const gm_record *record,
                           void *ws, size_t ws_bytes, void *stream);
size_t accept_workspace_bytes(int B, int k, int V);
// sets the thread's gm_last_error() message and returns st
gm_status set_error(gm_status st, const char *fmt, ...);

// ---------------------------------------------------------------- orchestration
struct ForwardPlan {
  size_t nbuf, act, qkv, q, attn, attn_ws, part, tiles, total;
  AttnPlan attn_plan;
};
ForwardPlan plan_forward(const gm_model_config &cfg, int B, int k, int max_ctx);
// target_stats (may be null): one RowStat per logits row at 1 / inv_t, from the LM head's epilogue
void run_verify_forward(const gm_model_config &cfg, const gm_model_weights &w, const gm_kv_cache &c, int B, int k,
                        const int32_t *tokens, float *logits, float *hidden, float inv_t, RowStat *target_stats,
                        const ForwardPlan &p, char *ws, int32_t *dev_err, hipStream_t s);

struct MtpPlan {
  size_t u, x, xg, nbuf, act, qkv, q, attn, attn_g, attn_ws, stat, nuc, sel, wsum, psum, nucpart, part, total;
  AttnPlan attn_ext, attn_chain;
};
MtpPlan plan_mtp(const gm_model_config &cfg, int B, int k, int max_ctx);
// draft-path reconstruction of R recorded cycles over K depths (workspace: plan_mtp(cfg, R, K, max_ctx))
void run_mtp_reconstruct(const gm_model_config &cfg, const gm_mtp_weights &mtp, const gm_model_weights &shared,
                         const gm_kv_cache &c, int R, int K, const float *start_hidden, const int32_t *start_tokens,
                         const int32_t *drafts, float *head_logits, const MtpPlan &p, char *ws, int32_t *dev_err,
                         hipStream_t s);
// top_p < 1 (sample mode): each draft is drawn from the nucleus of its row (inv_td = 1 / T in float64)
void run_mtp_draft(const gm_model_config &cfg, const gm_mtp_weights &mtp, const gm_model_weights &shared,
                   const gm_kv_cache &c, int B, int k, int mode, float inv_t, double top_p, double inv_td,
                   const float *verify_hidden,
                   const int32_t *n_accept, const int32_t *out_tokens, const float *u_draft, int32_t *drafts,
                   float *draft_logits, RowStat *draft_stats, NucRow *draft_nucleus, const MtpPlan &p, char *ws,
                   int32_t *dev_err,
                   hipStream_t s);

}  // namespace gm
