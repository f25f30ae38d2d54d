// Orchestration of the verify forward (Sec. 3.1, Eq. verification-context)
// and of the MTP draft (App. "Models and Draft Heads"; Eqs. tf-restart,
// tf-restart-kv) as sequences of kernel launches on one stream.
#include "forward.h"

namespace gm {

namespace {
size_t esize(int dtype) { return dtype == GM_BF16 ? 2 : 4; }
int qkv_width(const gm_model_config &c) { return (c.n_heads + 2 * c.n_kv_heads) * c.head_dim; }

// largest K-split partial buffer over the layer GEMMs at M rows (plus the LM head)
size_t part_bytes(const gm_model_config &c, int M, bool with_proj) {
  const int H = c.hidden, qd = c.n_heads * c.head_dim;
  size_t b = 0;
  auto upd = [&](int epi, int N, int K) {
    const size_t x = plan_gemm(c.dtype, epi, M, N, K).part_bytes;
    if (x > b) b = x;
  };
  upd(EPI_STORE_F32, qkv_width(c), H);
  upd(EPI_ADD_F32, H, qd);
  upd(EPI_SWIGLU, c.ffn, H);
  upd(EPI_ADD_F32, H, c.ffn);
  upd(EPI_STORE_F32, c.vocab, H);
  if (with_proj) upd(EPI_STORE_F32, H, 2 * H);
  return b;
}

// GEMM into the float32 residual rows Y [M][N] followed by the RMSNorm of those
// rows into nbuf: with a K split the reduce and the norm run as one kernel.
void gemm_norm(const char *name, int dt, int epi, int M, int N, int K, const void *X, int ldx, const void *W,
               float *Y, float *part, const void *norm_w, float eps, void *nbuf, hipStream_t s) {
  const int sp = launch_gemm(name, dt, epi, M, N, K, X, ldx, W, Y, N, part, s, nullptr, 1.f, true);
  if (sp > 1) launch_reduce_norm(dt, epi, M, N, sp, part, Y, norm_w, eps, nbuf, s);
  else launch_rmsnorm(dt, M, N, eps, Y, norm_w, nbuf, s);
}

// qkv projection: `splits` > 1 leaves the partials in `part` for the RoPE kernel to sum
RopeArgs rope_args(const gm_model_config &cfg, const gm_kv_cache &c, int layer, int M, int R, const float *qkv,
                   const float *part, int splits, void *q_out, const int32_t *base, int base_off,
                   const int32_t *blk_len, int pos_off, const gm_layer_weights &L, int32_t *dev_err) {
  RopeArgs a{};
  a.dtype = cfg.dtype;
  a.M = M;
  a.R = R;
  a.n_heads = cfg.n_heads;
  a.n_kv = cfg.n_kv_heads;
  a.head_dim = cfg.head_dim;
  a.qkv = qkv;
  a.part = part;
  a.splits = splits;
  a.q_out = q_out;
  a.k_pages = c.k_pages[layer];
  a.v_pages = c.v_pages[layer];
  a.block_table = c.block_table;
  a.page_size = c.page_size;
  a.max_pages = c.max_pages_per_seq;
  a.num_pages = c.num_pages;
  a.base_lens = base;
  a.base_off = base_off;
  a.blk_len = blk_len;
  a.blk_len_add = blk_len ? 1 : 0;
  a.pos_off = pos_off;
  a.rope_base = cfg.rope_base;
  a.eps = cfg.rms_eps;
  a.q_norm = cfg.qk_norm ? L.q_norm : nullptr;
  a.k_norm = cfg.qk_norm ? L.k_norm : nullptr;
  a.dev_err = dev_err;
  return a;
}
}  // namespace

// ---------------------------------------------------------------- verify forward
ForwardPlan plan_forward(const gm_model_config &cfg, int B, int k, int max_ctx) {
  ForwardPlan p{};
  const size_t M = (size_t)B * (k + 1), e = esize(cfg.dtype);
  const size_t qd = (size_t)cfg.n_heads * cfg.head_dim;
  Carve c;
  p.nbuf = c.take(M * cfg.hidden * e);
  p.act = c.take(M * cfg.ffn * e);
  p.qkv = c.take(M * qkv_width(cfg) * sizeof(float));
  p.q = c.take(M * qd * e);
  p.attn = c.take(M * qd * e);
  p.attn_plan = plan_attention(cfg, B, k + 1, max_ctx);
  p.attn_ws = c.take(p.attn_plan.total);
  p.part = c.take(part_bytes(cfg, (int)M, false));
  // the LM head's tile statistics when the caller wants the rows' softmax statistics
  p.tiles = c.take(sizeof(RowStat) * M * plan_lm_head(cfg.dtype, (int)M, cfg.vocab, cfg.hidden).tiles);
  p.total = c.off;
  return p;
}

// One target forward over the block of every sequence.  The residual stream
// lives in `hidden` (float32); it is the last layer's output at the end.
void run_verify_forward(const gm_model_config &cfg, const gm_model_weights &w, const gm_kv_cache &c, int B, int k,
                        const int32_t *tokens, float *logits, float *hidden, float inv_t, RowStat *target_stats,
                        const ForwardPlan &p, char *ws, int32_t *dev_err, hipStream_t s) {
  const int R = k + 1, M = B * R, H = cfg.hidden, F = cfg.ffn, V = cfg.vocab, dt = cfg.dtype;
  const int qd = cfg.n_heads * cfg.head_dim;
  void *nbuf = ws + p.nbuf, *act = ws + p.act, *q = ws + p.q, *attn = ws + p.attn;
  float *qkv = (float *)(ws + p.qkv);
  float *x = hidden, *part = (float *)(ws + p.part);
  const float eps = cfg.rms_eps;
  // the RMSNorm that opens a layer (or the final one) runs fused into the kernel before it
  auto next_norm = [&](int l) { return l < cfg.n_layers ? w.layers[l].attn_norm : w.final_norm; };
  launch_embed_norm(dt, M, H, V, tokens, w.embed, x, next_norm(0), eps, nbuf, dev_err, s);
  for (int l = 0; l < cfg.n_layers; ++l) {
    const gm_layer_weights &L = w.layers[l];
    const int sq = launch_gemm("gemm_qkv", dt, EPI_STORE_F32, M, qkv_width(cfg), H, nbuf, H, L.w_qkv, qkv,
                               qkv_width(cfg), part, s, nullptr, 1.f, true);
    launch_rope_append(rope_args(cfg, c, l, M, R, qkv, part, sq, q, c.seq_lens, 0, nullptr, 0, L, dev_err), s);
    AttnArgs a = attn_args(cfg, c, l, B, R, c.seq_lens, 0, nullptr);
    a.trace = "attn_verify";
    a.trace_combine = "attn_verify_combine";
    a.q = q;
    a.out = attn;
    a.dev_err = dev_err;
    run_attention(a, p.attn_plan, ws + p.attn_ws, s);
    gemm_norm("gemm_o", dt, EPI_ADD_F32, M, H, qd, attn, qd, L.w_o, x, part, L.ffn_norm, eps, nbuf, s);
    launch_gemm("gemm_gate_up", dt, EPI_SWIGLU, M, F, H, nbuf, H, L.w_gate_up, act, F, part, s);
    gemm_norm("gemm_down", dt, EPI_ADD_F32, M, H, F, act, F, L.w_down, x, part, next_norm(l + 1), eps, nbuf, s);
  }
  if (target_stats) {
    // the rows' softmax statistics in the LM head's epilogue (per tile of ids), then one per row
    RowStat *tiles = (RowStat *)(ws + p.tiles);
    launch_gemm("gemm_lm_head", dt, EPI_STATS, M, V, H, nbuf, H, w.lm_head, logits, V, part, s, tiles, inv_t);
    launch_tile_combine(M, plan_lm_head(dt, M, V, H).tiles, tiles, target_stats, 1, s);
  } else {
    launch_gemm("gemm_lm_head", dt, EPI_STORE_F32, M, V, H, nbuf, H, w.lm_head, logits, V, part, s);
  }
}

// ---------------------------------------------------------------- MTP draft
MtpPlan plan_mtp(const gm_model_config &cfg, int B, int k, int max_ctx) {
  MtpPlan p{};
  const size_t R = k + 1, Me = (size_t)B * R, e = esize(cfg.dtype), H = cfg.hidden;
  const size_t qd = (size_t)cfg.n_heads * cfg.head_dim;
  Carve c;
  p.u = c.take(Me * 2 * H * e);
  p.x = c.take(Me * H * sizeof(float));
  p.xg = c.take((size_t)B * H * sizeof(float));
  p.nbuf = c.take(Me * H * e);
  p.act = c.take((size_t)B * cfg.ffn * e);
  p.qkv = c.take(Me * qkv_width(cfg) * sizeof(float));
  p.q = c.take(Me * qd * e);
  p.attn = c.take(Me * qd * e);
  p.attn_g = c.take((size_t)B * qd * e);
  p.attn_ext = plan_attention(cfg, B, (int)R, max_ctx);
  p.attn_chain = plan_attention(cfg, B, 1, max_ctx + 2 * k);
  p.attn_ws = c.take(p.attn_ext.total > p.attn_chain.total ? p.attn_ext.total : p.attn_chain.total);
  const int V = cfg.vocab;
  p.stat = c.take(sizeof(RowStat) * (size_t)B * plan_lm_head(cfg.dtype, B, V, cfg.hidden).tiles);
  p.nuc = c.take(sizeof(NucRow) * (size_t)B);        // top-p draws: nuclei, draws, chunk masses
  p.sel = c.take(sizeof(RowSel) * (size_t)B);
  p.wsum = c.take(sizeof(double) * (size_t)B * scan_chunks(V));
  p.psum = c.take(sizeof(double) * (size_t)B * scan_chunks(V));
  p.nucpart = c.take(kNucPartBytes);
  const size_t pe = part_bytes(cfg, (int)Me, true), pb = part_bytes(cfg, B, true);
  p.part = c.take(pe > pb ? pe : pb);
  p.total = c.off;
  return p;
}

// Extend the head's cache with the n_b + 1 rows of target features behind the
// new boundary, then run the chain of k drafts.  Only the K/V projection of
// the first n_b extend rows is needed; the rest of the layer runs on the last
// row of each sequence (and on the single row of every chain step).
void run_mtp_draft(const gm_model_config &cfg, const gm_mtp_weights &mtp, const gm_model_weights &shared,
                   const gm_kv_cache &c, int B, int k, int mode, float inv_t, double top_p, double inv_td,
                   const float *verify_hidden,
                   const int32_t *n_accept, const int32_t *out_tokens, const float *u_draft, int32_t *drafts,
                   float *draft_logits, RowStat *draft_stats, NucRow *draft_nucleus, const MtpPlan &p, char *ws,
                   int32_t *dev_err,
                   hipStream_t s) {
  const int R = k + 1, Me = B * R, H = cfg.hidden, F = cfg.ffn, V = cfg.vocab, dt = cfg.dtype;
  const int qd = cfg.n_heads * cfg.head_dim, qw = qkv_width(cfg);
  const size_t e = esize(dt);
  const gm_layer_weights &L = mtp.layer;
  void *u = ws + p.u, *nbuf = ws + p.nbuf, *act = ws + p.act, *q = ws + p.q, *attn = ws + p.attn,
       *attn_g = ws + p.attn_g;
  float *x = (float *)(ws + p.x), *xg = (float *)(ws + p.xg), *qkv = (float *)(ws + p.qkv);
  RowStat *tiles = (RowStat *)(ws + p.stat);
  float *part = (float *)(ws + p.part);
  int32_t *lens = c.seq_lens;

  // the layer tail on one row per sequence (x1 [B][H] float32 in place), then the
  // shared LM head into draft_logits[:, j, :] and the draw of drafts[:, j]
  const float eps = cfg.rms_eps;
  auto tail_and_draw = [&](float *x1, int j) {
    gemm_norm("mtp_gemm_o", dt, EPI_ADD_F32, B, H, qd, attn_g, qd, L.w_o, x1, part, L.ffn_norm, eps, nbuf, s);
    launch_gemm("mtp_gemm_gate_up", dt, EPI_SWIGLU, B, F, H, nbuf, H, L.w_gate_up, act, F, part, s);
    gemm_norm("mtp_gemm_down", dt, EPI_ADD_F32, B, H, F, act, F, L.w_down, x1, part, mtp.final_norm, eps, nbuf, s);
    float *zl = draft_logits + (long)j * V;
    // the LM head emits the logits and their softmax statistics per tile of ids; the draw
    // then reads only the tile statistics and one tile of logits per sequence
    launch_gemm("mtp_gemm_lm_head", dt, EPI_STATS, B, V, H, nbuf, H, shared.lm_head, zl, (long)k * V, part, s, tiles,
                inv_t);
    const TileGeom geo = plan_lm_head(dt, B, V, H);
    if (top_p < 1.0) {   // top-p: a draw from each row's nucleus (a selection, then an inverse-CDF scan)
      // the nuclei go to the caller's draft_nucleus[:, j] when given (the accept's handoff)
      NucRow *nuc = draft_nucleus ? draft_nucleus + j : (NucRow *)(ws + p.nuc);
      const int ns = draft_nucleus ? k : 1;
      RowSel *sel = (RowSel *)(ws + p.sel);
      launch_nucleus("draft_nucleus", B, V, inv_td, top_p, zl, (long)k * V, tiles, geo.tiles, nuc, ns,
                     (unsigned long long *)(ws + p.nucpart), s);
      launch_nucleus_select(B, zl, (long)k * V, nuc, ns, u_draft + j, k, drafts + j, k, sel, s);
      launch_residual_draw("draft_nucleus_chunk", "draft_nucleus_scan", B, V, inv_t, sel, (double *)(ws + p.wsum),
                           (double *)(ws + p.psum), true, s);
    } else {
      // below the last depth the draw also builds the next chain step's input row (the
      // drawn id with the layer output x1), in place of a separate input launch
      const DrawNextInput next{dt, H, cfg.rms_eps, x1, shared.embed, mtp.norm_h, mtp.norm_e, u, dev_err};
      launch_tile_draw(B, V, mode, inv_t, zl, (long)k * V, geo, tiles, u_draft ? u_draft + j : nullptr, k, drafts + j,
                       k, draft_stats ? draft_stats + j : nullptr, k, s, j + 1 < k ? &next : nullptr);
    }
  };

  // ---- extend: rows (h_{m+i}, x_{m+i+1}), i = 0..n_b, at slots m_b + i
  launch_mtp_input(dt, Me, H, V, cfg.rms_eps, verify_hidden, out_tokens, 1, shared.embed, mtp.norm_h, mtp.norm_e, u,
                   dev_err, s);
  gemm_norm("mtp_gemm_proj", dt, EPI_STORE_F32, Me, H, 2 * H, u, 2 * H, mtp.w_proj, x, part, L.attn_norm, eps, nbuf,
            s);
  int sq = launch_gemm("mtp_gemm_qkv", dt, EPI_STORE_F32, Me, qw, H, nbuf, H, L.w_qkv, qkv, qw, part, s, nullptr, 1.f,
                       true);
  launch_rope_append(rope_args(cfg, c, 0, Me, R, qkv, part, sq, q, lens, 0, n_accept, 1, L, dev_err), s);
  {
    AttnArgs a = attn_args(cfg, c, 0, B, R, lens, 0, n_accept);
    a.blk_len_add = 1;
    a.trace = "attn_mtp";
    a.trace_combine = "attn_mtp_combine";
    a.q = q;
    a.out = attn;
    a.dev_err = dev_err;
    run_attention(a, p.attn_ext, ws + p.attn_ws, s);
  }
  // the boundary rows of the attention output and the residual stream, and the head's
  // committed length moved to the new boundary m_b + n_b + 1, in one launch
  launch_gather_commit(B, R, qd, e, attn, attn_g, H, sizeof(float), x, xg, n_accept, lens, s);
  tail_and_draw(xg, 0);

  // ---- chain: step j feeds (g_{j-1}, d_{j-1}) at slot boundary + j - 1
  for (int j = 1; j < k; ++j) {
    if (top_p < 1.0)   // (at top-p 1 the draw of depth j - 1 has built this input)
      launch_mtp_input(dt, B, H, V, cfg.rms_eps, xg, drafts + (j - 1), k, shared.embed, mtp.norm_h, mtp.norm_e, u,
                       dev_err, s);
    gemm_norm("mtp_gemm_proj", dt, EPI_STORE_F32, B, H, 2 * H, u, 2 * H, mtp.w_proj, xg, part, L.attn_norm, eps, nbuf,
              s);
    sq = launch_gemm("mtp_gemm_qkv", dt, EPI_STORE_F32, B, qw, H, nbuf, H, L.w_qkv, qkv, qw, part, s, nullptr, 1.f,
                     true);
    launch_rope_append(rope_args(cfg, c, 0, B, 1, qkv, part, sq, q, lens, j - 1, nullptr, 1, L, dev_err), s);
    AttnArgs a = attn_args(cfg, c, 0, B, 1, lens, j - 1, nullptr);
    a.trace = "attn_mtp";
    a.trace_combine = "attn_mtp_combine";
    a.q = q;
    a.out = attn_g;
    a.dev_err = dev_err;
    run_attention(a, p.attn_chain, ws + p.attn_ws, s);
    tail_and_draw(xg, j);
  }
}

// Draft-path reconstruction: K batched single-row steps of the head, one row per
// recorded cycle.  Depth j + 1 feeds the recorded start pair (j = 0) or
// (g_j, d_j) at slot start + j, rotated at slot + 1, and attends to slots
// 0 .. start + j of its own block table: the committed prefix and its own chain.
// Nothing is drawn; the head logits of depth j + 1 go to head_logits[:, j, :].
void run_mtp_reconstruct(const gm_model_config &cfg, const gm_mtp_weights &mtp, const gm_model_weights &shared,
                         const gm_kv_cache &c, int R, int K, const float *start_hidden, const int32_t *start_tokens,
                         const int32_t *drafts, float *head_logits, const MtpPlan &p, char *ws, int32_t *dev_err,
                         hipStream_t s) {
  const int H = cfg.hidden, F = cfg.ffn, V = cfg.vocab, dt = cfg.dtype;
  const int qd = cfg.n_heads * cfg.head_dim, qw = qkv_width(cfg);
  const gm_layer_weights &L = mtp.layer;
  void *u = ws + p.u, *nbuf = ws + p.nbuf, *act = ws + p.act, *q = ws + p.q, *attn_g = ws + p.attn_g;
  float *xg = (float *)(ws + p.xg), *qkv = (float *)(ws + p.qkv);
  float *part = (float *)(ws + p.part);
  int32_t *lens = c.seq_lens;
  const float eps = cfg.rms_eps;
  for (int j = 0; j < K; ++j) {
    if (j == 0)
      launch_mtp_input(dt, R, H, V, eps, start_hidden, start_tokens, 1, shared.embed, mtp.norm_h, mtp.norm_e, u,
                       dev_err, s);
    else
      launch_mtp_input(dt, R, H, V, eps, xg, drafts + (j - 1), K, shared.embed, mtp.norm_h, mtp.norm_e, u, dev_err,
                       s);
    gemm_norm("recon_gemm_proj", dt, EPI_STORE_F32, R, H, 2 * H, u, 2 * H, mtp.w_proj, xg, part, L.attn_norm, eps,
              nbuf, s);
    const int sq = launch_gemm("recon_gemm_qkv", dt, EPI_STORE_F32, R, qw, H, nbuf, H, L.w_qkv, qkv, qw, part, s,
                               nullptr, 1.f, true);
    launch_rope_append(rope_args(cfg, c, 0, R, 1, qkv, part, sq, q, lens, j, nullptr, 1, L, dev_err), s);
    AttnArgs a = attn_args(cfg, c, 0, R, 1, lens, j, nullptr);
    a.trace = "attn_recon";
    a.trace_combine = "attn_recon_combine";
    a.q = q;
    a.out = attn_g;
    a.dev_err = dev_err;
    run_attention(a, p.attn_chain, ws + p.attn_ws, s);
    gemm_norm("recon_gemm_o", dt, EPI_ADD_F32, R, H, qd, attn_g, qd, L.w_o, xg, part, L.ffn_norm, eps, nbuf, s);
    launch_gemm("recon_gemm_gate_up", dt, EPI_SWIGLU, R, F, H, nbuf, H, L.w_gate_up, act, F, part, s);
    gemm_norm("recon_gemm_down", dt, EPI_ADD_F32, R, H, F, act, F, L.w_down, xg, part, mtp.final_norm, eps, nbuf, s);
    launch_gemm("recon_gemm_lm_head", dt, EPI_STORE_F32, R, V, H, nbuf, H, shared.lm_head, head_logits + (long)j * V,
                (long)K * V, part, s);
  }
}

}  // namespace gm
