// C ABI of libgm: argument validation, workspace carving and kernel launches.
// Every entry point validates on the host, then enqueues on the caller's
// stream and returns without synchronising.
#include <stdarg.h>
#include <stddef.h>
#include <stdio.h>

#include <string>

#include "forward.h"
#include "launch.h"

using namespace gm;

namespace {
thread_local std::string g_err;

gm_status vfail(gm_status st, const char *fmt, va_list ap) {
  char buf[512];
  vsnprintf(buf, sizeof(buf), fmt, ap);
  g_err = buf;
  return st;
}

gm_status fail(gm_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  const gm_status r = vfail(st, fmt, ap);
  va_end(ap);
  return r;
}

gm_status check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GM_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
  return GM_OK;
}

constexpr int kMaxK = 15;

// ---------------------------------------------------------------- workspace plans
struct AcceptPlan {
  size_t tstat, dstat, sel, wsum, psum, submax, tnuc, dnuc, nucpart, total;
};
AcceptPlan plan_accept(int B, int k, int V) {
  Carve c;
  AcceptPlan p;
  const int nch = stat_chunks(V), nsc = scan_chunks(V);
  p.tstat = c.take(sizeof(RowStat) * (size_t)B * (k + 1) * nch);
  p.dstat = c.take(sizeof(RowStat) * (size_t)B * (k > 0 ? k : 1) * nch);
  p.sel = c.take(sizeof(RowSel) * (size_t)B);
  p.wsum = c.take(sizeof(double) * (size_t)B * nsc);
  p.psum = c.take(sizeof(double) * (size_t)B * nsc);
  p.submax = c.take(sizeof(float) * (size_t)B * (k + 1) * nch * 64);   // run maxima of the record's selection
  p.tnuc = c.take(sizeof(NucRow) * (size_t)B * (k + 1));                // top-p nuclei of the target rows
  p.dnuc = c.take(sizeof(NucRow) * (size_t)B * (k > 0 ? k : 1));        // and of the draft rows
  p.nucpart = c.take(kNucPartBytes);                                    // their split first pass
  p.total = c.off;
  return p;
}

gm_status check_config(const gm_model_config *cfg, int B, int k) {
  if (!cfg) return fail(GM_ERR_INVALID_ARG, "null model config");
  if (B < 0) return fail(GM_ERR_INVALID_ARG, "B = %d < 0", B);
  if (k < 0 || k > kMaxK) return fail(GM_ERR_UNSUPPORTED, "draft length k = %d outside [0, %d]", k, kMaxK);
  if (cfg->n_layers < 1 || cfg->hidden < 1 || cfg->n_heads < 1 || cfg->n_kv_heads < 1 || cfg->head_dim < 1 ||
      cfg->ffn < 1 || cfg->vocab < 1)
    return fail(GM_ERR_INVALID_ARG, "non-positive model dimension");
  if (cfg->n_heads % cfg->n_kv_heads) return fail(GM_ERR_INVALID_ARG, "n_heads %% n_kv_heads != 0");
  if (cfg->dtype != GM_F32 && cfg->dtype != GM_BF16) return fail(GM_ERR_INVALID_ARG, "unknown dtype %d", cfg->dtype);
  const int G = cfg->n_heads / cfg->n_kv_heads;
  if (G * (k + 1) > kAttnMaxRows)
    return fail(GM_ERR_UNSUPPORTED, "(n_heads / n_kv_heads) * (k + 1) = %d exceeds %d", G * (k + 1), kAttnMaxRows);
  if (cfg->hidden % 64 || cfg->ffn % 64) return fail(GM_ERR_UNSUPPORTED, "hidden and ffn must be multiples of 64");
  if (cfg->vocab > kMaxVocab) return fail(GM_ERR_UNSUPPORTED, "vocab %d exceeds %d", cfg->vocab, kMaxVocab);
  // row kernels stage one hidden row or one projected q/k/v row in 64 KiB of LDS
  if (cfg->hidden > kMaxRowFloats || (cfg->n_heads + 2 * cfg->n_kv_heads) * cfg->head_dim > kMaxRowFloats)
    return fail(GM_ERR_UNSUPPORTED, "hidden and (n_heads + 2 n_kv_heads) * head_dim must be at most %d", kMaxRowFloats);
  if (!(cfg->rms_eps >= 0.f) || !(cfg->rope_base > 0.f)) return fail(GM_ERR_INVALID_ARG, "bad rms_eps or rope_base");
  if (cfg->dtype == GM_BF16) {
    if (cfg->head_dim != 128) return fail(GM_ERR_UNSUPPORTED, "bf16 path needs head_dim 128, got %d", cfg->head_dim);
    if (cfg->vocab % 128 || cfg->hidden % 256 || cfg->ffn % 256 || (cfg->n_heads * cfg->head_dim) % 256)
      return fail(GM_ERR_UNSUPPORTED,
                  "bf16 path needs vocab a multiple of 128 and hidden, ffn, n_heads*head_dim multiples of 256");
  } else {
    if (cfg->head_dim != 64 && cfg->head_dim != 128)
      return fail(GM_ERR_UNSUPPORTED, "f32 path needs head_dim 64 or 128, got %d", cfg->head_dim);
  }
  return GM_OK;
}

gm_status check_layer(const gm_model_config *cfg, const gm_layer_weights *L, const char *what) {
  if (!L->attn_norm || !L->w_qkv || !L->w_o || !L->ffn_norm || !L->w_gate_up || !L->w_down)
    return fail(GM_ERR_INVALID_ARG, "%s: null layer weight", what);
  if (cfg->qk_norm && (!L->q_norm || !L->k_norm)) return fail(GM_ERR_INVALID_ARG, "%s: qk_norm set but q_norm/k_norm null", what);
  return GM_OK;
}

gm_status check_cache(const gm_model_config *cfg, const gm_kv_cache *c, int n_layers, int k_extra,
                      const char *what) {
  if (!c) return fail(GM_ERR_INVALID_ARG, "%s: null cache", what);
  if (c->n_layers != n_layers) return fail(GM_ERR_INVALID_ARG, "%s: cache has %d layers, need %d", what, c->n_layers, n_layers);
  if (!c->k_pages || !c->v_pages || !c->block_table || !c->seq_lens)
    return fail(GM_ERR_INVALID_ARG, "%s: null cache pointer", what);
  for (int l = 0; l < n_layers; ++l)
    if (!c->k_pages[l] || !c->v_pages[l]) return fail(GM_ERR_INVALID_ARG, "%s: null page pool of layer %d", what, l);
  if (c->page_size < 16 || c->page_size % 16) return fail(GM_ERR_UNSUPPORTED, "%s: page_size %d is not a multiple of 16", what, c->page_size);
  if (c->num_pages < 1 || c->max_pages_per_seq < 1) return fail(GM_ERR_INVALID_ARG, "%s: empty page pool", what);
  if (c->max_ctx < 0) return fail(GM_ERR_INVALID_ARG, "%s: max_ctx < 0", what);
  if ((long)c->max_ctx + k_extra > (long)c->max_pages_per_seq * c->page_size)
    return fail(GM_ERR_CAPACITY, "%s: max_ctx %d + %d positions exceed %d pages of %d", what, c->max_ctx, k_extra,
                c->max_pages_per_seq, c->page_size);
  (void)cfg;
  return GM_OK;
}

gm_status check_ws(void *ws, size_t have, size_t need) {
  if (need > have) return fail(GM_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", have, need);
  if (need && !ws) return fail(GM_ERR_WORKSPACE, "null workspace");
  if (((uintptr_t)ws) & 255) return fail(GM_ERR_WORKSPACE, "workspace not 256-byte aligned");
  return GM_OK;
}
}  // namespace

extern "C" const char *gm_last_error(void) { return g_err.c_str(); }

extern "C" size_t gm_workspace_size(int op, const gm_model_config *cfg, int B, int k, int max_ctx) {
  if (B < 0 || k < 0 || k > kMaxK || max_ctx < 0) return 0;
  switch (op) {
    case GM_OP_SPEC_ACCEPT:
      if (!cfg || cfg->vocab < 1) return 0;
      return plan_accept(B, k, cfg->vocab).total;
    case GM_OP_VERIFY_FORWARD:
      if (check_config(cfg, B, k) != GM_OK) return 0;
      return plan_forward(*cfg, B, k, max_ctx).total;
    case GM_OP_VERIFY_ATTENTION:
      if (check_config(cfg, B, k) != GM_OK) return 0;
      return plan_attention(*cfg, B, k + 1, max_ctx).total;
    case GM_OP_MTP_DRAFT:
      if (check_config(cfg, B, k) != GM_OK) return 0;
      return plan_mtp(*cfg, B, k, max_ctx).total;
    case GM_OP_MTP_RECONSTRUCT:
      if (k < 1 || check_config(cfg, B, k) != GM_OK) return 0;
      return plan_mtp(*cfg, B, k, max_ctx).total;
    case GM_OP_DCA_LOSS:
      if (!cfg || k < 1 || cfg->vocab < 1 || cfg->vocab > kMaxVocab) return 0;
      return dca_workspace(B, k, cfg->vocab);
    default:
      return 0;
  }
}

// ---------------------------------------------------------------- gm_spec_accept
static_assert(sizeof(gm_row_stats) == sizeof(RowStat) && offsetof(gm_row_stats, max) == offsetof(RowStat, max) &&
                  offsetof(gm_row_stats, argmax) == offsetof(RowStat, argmax) &&
                  offsetof(gm_row_stats, sum) == offsetof(RowStat, sum),
              "gm_row_stats is the device's RowStat");
static_assert(sizeof(gm_nucleus) == sizeof(NucRow) && offsetof(gm_nucleus, m) == offsetof(NucRow, m) &&
                  offsetof(gm_nucleus, mass) == offsetof(NucRow, s) && offsetof(gm_nucleus, key) == offsetof(NucRow, key) &&
                  offsetof(gm_nucleus, last_id) == offsetof(NucRow, idt),
              "gm_nucleus is the device's NucRow");

namespace gm {
gm_status set_error(gm_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  const gm_status r = vfail(st, fmt, ap);
  va_end(ap);
  return r;
}

size_t accept_workspace_bytes(int B, int k, int V) { return plan_accept(B, k, V).total; }

gm_status spec_accept_impl(int B, int k, int V, int mode, float temperature, float top_p, const float *target_logits,
                           const float *draft_logits, const gm_row_stats *target_stats, const gm_row_stats *draft_stats,
                           const gm_nucleus *draft_nucleus, const int32_t *draft_tokens, const float *u_accept,
                           const float *u_final, int32_t *n_accept, int32_t *out_tokens, const gm_record *record,
                           void *ws, size_t ws_bytes, void *stream) {
  if (B < 0 || k < 0 || k > kMaxK || V < 1) return fail(GM_ERR_INVALID_ARG, "bad B=%d k=%d V=%d", B, k, V);
  if (V > kMaxVocab) return fail(GM_ERR_UNSUPPORTED, "vocab %d exceeds %d", V, kMaxVocab);
  if (mode != GM_GREEDY && mode != GM_SAMPLE) return fail(GM_ERR_INVALID_ARG, "unknown accept mode %d", mode);
  if (!(temperature > 0.f)) return fail(GM_ERR_INVALID_ARG, "temperature must be > 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(GM_ERR_INVALID_ARG, "top_p must be in (0, 1]");
  if (B == 0) return GM_OK;
  if (!target_logits || !n_accept || !out_tokens) return fail(GM_ERR_INVALID_ARG, "null target_logits / outputs");
  if (k > 0 && !draft_tokens) return fail(GM_ERR_INVALID_ARG, "null draft_tokens");
  if (mode == GM_SAMPLE) {
    if (!u_final) return fail(GM_ERR_INVALID_ARG, "sample mode needs u_final");
    if (k > 0 && (!draft_logits || !u_accept)) return fail(GM_ERR_INVALID_ARG, "sample mode needs draft_logits and u_accept");
  }
  if (record && k > 0) {
    if (record->topk < 1 || record->topk > kRecMaxTopk || record->topk > V)
      return fail(GM_ERR_INVALID_ARG, "record topk %d outside 1..min(%d, V)", record->topk, kRecMaxTopk);
    if (!record->logp || !record->ids) return fail(GM_ERR_INVALID_ARG, "null record buffers");
  }
  const AcceptPlan p = plan_accept(B, k, V);
  gm_status st = check_ws(ws, ws_bytes, p.total);
  if (st != GM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  char *w = (char *)ws;
  RowStat *tstat = (RowStat *)(w + p.tstat), *dstat = (RowStat *)(w + p.dstat);
  RowSel *sel = (RowSel *)(w + p.sel);
  const float inv_t = 1.0f / temperature;
  const bool rec = record && k > 0;
  float *submax = rec ? (float *)(w + p.submax) : nullptr;
  // p's statistics: the verify forward's own (one per row) when the caller has them and no record
  // needs the pass's run maxima, else a pass over the target rows
  int nch_t = stat_chunks(V);
  if (target_stats && !rec) {
    tstat = (RowStat *)target_stats;
    nch_t = 1;
  } else {
    launch_row_stats("accept_row_stats", target_logits, V, B * (k + 1), V, inv_t, tstat, s, submax);
  }
  // q's statistics: the draft head's own (one per row) when the caller has them, else a pass over the rows
  int nch_d = stat_chunks(V);
  const bool top_p_on = mode == GM_SAMPLE && top_p < 1.f;
  if (mode == GM_SAMPLE && k > 0) {
    if (top_p_on && draft_nucleus) {
      nch_d = 0;                      // the draft rows' nuclei carry their reference and mass
    } else if (draft_stats) {
      dstat = (RowStat *)draft_stats;
      nch_d = 1;
    } else {
      launch_row_stats("accept_row_stats", draft_logits, V, B * k, V, inv_t, dstat, s);
    }
  }
  // top-p (sample mode): the nuclei of every target and draft row
  const double inv_td = 1.0 / (double)temperature;
  NucRow *tnuc = nullptr, *dnuc = nullptr;
  if (top_p_on) {
    tnuc = (NucRow *)(w + p.tnuc);
    unsigned long long *part = (unsigned long long *)(w + p.nucpart);
    launch_nucleus("accept_nucleus", B * (k + 1), V, inv_td, (double)top_p, target_logits, V, tstat, nch_t,
                   tnuc, 1, part, s);
    if (k > 0 && draft_nucleus) {
      dnuc = (NucRow *)draft_nucleus;
    } else if (k > 0) {
      dnuc = (NucRow *)(w + p.dnuc);
      launch_nucleus("accept_nucleus", B * k, V, inv_td, (double)top_p, draft_logits, V, dstat, nch_d, dnuc, 1, part,
                     s);
    }
  }
  launch_accept_decide(B, k, V, mode, inv_t, inv_td, target_logits, draft_logits, tstat, nch_t, dstat, nch_d, tnuc,
                       dnuc,
                       draft_tokens, u_accept, u_final, n_accept, out_tokens, sel, s);
  if (rec)
    launch_record_topk(B, k, V, inv_t, record->topk, target_logits, tstat, submax, record->logp, record->ids, s);
  if (mode == GM_SAMPLE)
    launch_residual_draw("accept_residual_chunk", "accept_residual_scan", B, V, inv_t, sel, (double *)(w + p.wsum),
                         (double *)(w + p.psum), top_p_on, s);
  return check_launch("gm_spec_accept");
}
}  // namespace gm

extern "C" gm_status gm_spec_accept(int B, int k, int V, int mode, float temperature, float top_p,
                                    const float *target_logits,
                                    const float *draft_logits, const gm_row_stats *target_stats,
                                    const gm_row_stats *draft_stats,
                                    const gm_nucleus *draft_nucleus,
                                    const int32_t *draft_tokens, const float *u_accept,
                                    const float *u_final, int32_t *n_accept, int32_t *out_tokens,
                                    const gm_record *record, void *ws, size_t ws_bytes, void *stream) {
  return spec_accept_impl(B, k, V, mode, temperature, top_p, target_logits, draft_logits, target_stats, draft_stats,
                          draft_nucleus, draft_tokens, u_accept, u_final, n_accept, out_tokens, record, ws, ws_bytes,
                          stream);
}

// ---------------------------------------------------------------- gm_dca_loss
extern "C" gm_status gm_dca_loss(int N, int K, int V, int topk, const float *head_logits, const uint16_t *rec_logp,
                                 const int32_t *rec_ids, const int32_t *n_accept, int vgm, float *loss, float *alpha,
                                 float *grad, void *ws, size_t ws_bytes, void *stream) {
  if (N < 0 || K < 1 || K > kMaxK || V < 1) return fail(GM_ERR_INVALID_ARG, "bad N=%d K=%d V=%d", N, K, V);
  if (V > kMaxVocab) return fail(GM_ERR_UNSUPPORTED, "vocab %d exceeds %d", V, kMaxVocab);
  if (topk < 1 || topk > kRecMaxTopk || topk > V)
    return fail(GM_ERR_INVALID_ARG, "topk %d outside 1..min(%d, V)", topk, kRecMaxTopk);
  if (N == 0) return GM_OK;
  if (!head_logits || !rec_logp || !rec_ids || !loss || !alpha || (vgm && !n_accept))
    return fail(GM_ERR_INVALID_ARG, "null DCA input / output");
  gm_status st = check_ws(ws, ws_bytes, dca_workspace(N, K, V));
  if (st != GM_OK) return st;
  run_dca_loss(N, K, V, topk, head_logits, rec_logp, rec_ids, n_accept, vgm, loss, alpha, grad, (char *)ws,
               (hipStream_t)stream);
  return check_launch("gm_dca_loss");
}

// ---------------------------------------------------------------- gm_kv_commit
extern "C" gm_status gm_kv_commit(const gm_kv_cache *cache, int B, int k, const int32_t *n_accept,
                                  int32_t *committed_slots, void *stream) {
  if (!cache || !cache->block_table || !cache->seq_lens) return fail(GM_ERR_INVALID_ARG, "null cache");
  if (B < 0 || k < 0 || k > kMaxK) return fail(GM_ERR_INVALID_ARG, "bad B=%d k=%d", B, k);
  if (cache->page_size < 1 || cache->max_pages_per_seq < 1) return fail(GM_ERR_INVALID_ARG, "bad page geometry");
  if (B == 0) return GM_OK;
  if (!n_accept) return fail(GM_ERR_INVALID_ARG, "null n_accept");
  launch_kv_commit(B, k, cache->page_size, cache->max_pages_per_seq, cache->block_table, cache->seq_lens, n_accept,
                   committed_slots, (hipStream_t)stream);
  return check_launch("gm_kv_commit");
}

// ---------------------------------------------------------------- gm_verify_attention
extern "C" gm_status gm_verify_attention(const gm_model_config *cfg, const gm_kv_cache *cache, int layer, int B,
                                         int k, const void *q, void *out, void *ws, size_t ws_bytes,
                                         int32_t *dev_err, void *stream) {
  gm_status st = check_config(cfg, B, k);
  if (st != GM_OK) return st;
  if (!cache) return fail(GM_ERR_INVALID_ARG, "null cache");
  if (layer < 0 || layer >= cache->n_layers) return fail(GM_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, cache->n_layers);
  st = check_cache(cfg, cache, cache->n_layers, k + 1, "gm_verify_attention");
  if (st != GM_OK) return st;
  if (B == 0) return GM_OK;
  if (!q || !out) return fail(GM_ERR_INVALID_ARG, "null q / out");
  const AttnPlan p = plan_attention(*cfg, B, k + 1, cache->max_ctx);
  st = check_ws(ws, ws_bytes, p.total);
  if (st != GM_OK) return st;
  AttnArgs a = attn_args(*cfg, *cache, layer, B, k + 1, cache->seq_lens, 0, nullptr);
  a.trace = "attn_verify";
  a.trace_combine = "attn_verify_combine";
  a.q = q;
  a.out = out;
  a.dev_err = dev_err;
  run_attention(a, p, (char *)ws, (hipStream_t)stream);
  return check_launch("gm_verify_attention");
}

// ---------------------------------------------------------------- gm_verify_forward
extern "C" gm_status gm_verify_forward(const gm_model_config *cfg, const gm_model_weights *w, const gm_kv_cache *cache,
                                       int B, int k, const int32_t *tokens, float *logits, float *hidden,
                                       float temperature, gm_row_stats *target_stats, void *ws, size_t ws_bytes,
                                       int32_t *dev_err, void *stream) {
  gm_status st = check_config(cfg, B, k);
  if (st != GM_OK) return st;
  if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers) return fail(GM_ERR_INVALID_ARG, "null model weights");
  for (int l = 0; l < cfg->n_layers; ++l)
    if ((st = check_layer(cfg, &w->layers[l], "gm_verify_forward")) != GM_OK) return st;
  st = check_cache(cfg, cache, cfg->n_layers, k + 1, "gm_verify_forward");
  if (st != GM_OK) return st;
  if (B == 0) return GM_OK;
  if (!tokens || !logits || !hidden) return fail(GM_ERR_INVALID_ARG, "null tokens / logits / hidden");
  if (target_stats && !(temperature > 0.f)) return fail(GM_ERR_INVALID_ARG, "target_stats need a temperature > 0");
  const ForwardPlan p = plan_forward(*cfg, B, k, cache->max_ctx);
  st = check_ws(ws, ws_bytes, p.total);
  if (st != GM_OK) return st;
  run_verify_forward(*cfg, *w, *cache, B, k, tokens, logits, hidden, target_stats ? 1.0f / temperature : 1.0f,
                     (RowStat *)target_stats, p, (char *)ws, dev_err, (hipStream_t)stream);
  return check_launch("gm_verify_forward");
}

// ---------------------------------------------------------------- gm_mtp_draft
extern "C" gm_status gm_mtp_draft(const gm_model_config *cfg, const gm_mtp_weights *mtp, const gm_model_weights *shared,
                                  const gm_kv_cache *mtp_cache, int B, int k, int mode, float temperature,
                                  float top_p, const float *verify_hidden, const int32_t *n_accept, const int32_t *out_tokens,
                                  const float *u_draft, int32_t *drafts, float *draft_logits,
                                  gm_row_stats *draft_stats, gm_nucleus *draft_nucleus, void *ws, size_t ws_bytes,
                                  int32_t *dev_err,
                                  void *stream) {
  gm_status st = check_config(cfg, B, k);
  if (st != GM_OK) return st;
  if (k < 1) return fail(GM_ERR_INVALID_ARG, "gm_mtp_draft needs k >= 1");
  if (mode != GM_GREEDY && mode != GM_SAMPLE) return fail(GM_ERR_INVALID_ARG, "unknown draft mode %d", mode);
  if (!(temperature > 0.f)) return fail(GM_ERR_INVALID_ARG, "temperature must be > 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(GM_ERR_INVALID_ARG, "top_p must be in (0, 1]");
  if (mode == GM_SAMPLE && top_p < 1.f && draft_stats)
    return fail(GM_ERR_UNSUPPORTED, "draft_stats are not produced with top_p < 1 (pass NULL)");
  if (!mtp || !mtp->norm_h || !mtp->norm_e || !mtp->w_proj || !mtp->final_norm) return fail(GM_ERR_INVALID_ARG, "null MTP weights");
  if ((st = check_layer(cfg, &mtp->layer, "gm_mtp_draft")) != GM_OK) return st;
  if (!shared || !shared->embed || !shared->lm_head) return fail(GM_ERR_INVALID_ARG, "null shared embedding / LM head");
  st = check_cache(cfg, mtp_cache, 1, 2 * k + 1, "gm_mtp_draft");
  if (st != GM_OK) return st;
  if (B == 0) return GM_OK;
  if (!verify_hidden || !n_accept || !out_tokens || !drafts || !draft_logits)
    return fail(GM_ERR_INVALID_ARG, "null MTP input / output");
  if (mode == GM_SAMPLE && !u_draft) return fail(GM_ERR_INVALID_ARG, "sample mode needs u_draft");
  const MtpPlan p = plan_mtp(*cfg, B, k, mtp_cache->max_ctx);
  st = check_ws(ws, ws_bytes, p.total);
  if (st != GM_OK) return st;
  run_mtp_draft(*cfg, *mtp, *shared, *mtp_cache, B, k, mode, 1.0f / temperature,
                mode == GM_SAMPLE && top_p < 1.f ? (double)top_p : 1.0, 1.0 / (double)temperature, verify_hidden,
                n_accept, out_tokens, u_draft, drafts, draft_logits, (RowStat *)draft_stats, (NucRow *)draft_nucleus, p,
                (char *)ws, dev_err,
                (hipStream_t)stream);
  return check_launch("gm_mtp_draft");
}

// ---------------------------------------------------------------- gm_mtp_reconstruct
extern "C" gm_status gm_mtp_reconstruct(const gm_model_config *cfg, const gm_mtp_weights *mtp,
                                        const gm_model_weights *shared, const gm_kv_cache *mtp_cache, int R, int K,
                                        const float *start_hidden, const int32_t *start_tokens,
                                        const int32_t *drafts, float *head_logits, void *ws, size_t ws_bytes,
                                        int32_t *dev_err, void *stream) {
  gm_status st = check_config(cfg, R, K);
  if (st != GM_OK) return st;
  if (K < 1) return fail(GM_ERR_INVALID_ARG, "gm_mtp_reconstruct needs K >= 1");
  if (!mtp || !mtp->norm_h || !mtp->norm_e || !mtp->w_proj || !mtp->final_norm) return fail(GM_ERR_INVALID_ARG, "null MTP weights");
  if ((st = check_layer(cfg, &mtp->layer, "gm_mtp_reconstruct")) != GM_OK) return st;
  if (!shared || !shared->embed || !shared->lm_head) return fail(GM_ERR_INVALID_ARG, "null shared embedding / LM head");
  st = check_cache(cfg, mtp_cache, 1, K, "gm_mtp_reconstruct");
  if (st != GM_OK) return st;
  if (R == 0) return GM_OK;
  if (!start_hidden || !start_tokens || !head_logits || (K > 1 && !drafts))
    return fail(GM_ERR_INVALID_ARG, "null reconstruction input / output");
  const MtpPlan p = plan_mtp(*cfg, R, K, mtp_cache->max_ctx);
  st = check_ws(ws, ws_bytes, p.total);
  if (st != GM_OK) return st;
  run_mtp_reconstruct(*cfg, *mtp, *shared, *mtp_cache, R, K, start_hidden, start_tokens, drafts, head_logits, p,
                      (char *)ws, dev_err, (hipStream_t)stream);
  return check_launch("gm_mtp_reconstruct");
}
