// Host-side launchers of the gfx950 kernels (internal to libgm).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gm {

// ---------------------------------------------------------------- tracing
// RAII bracket of one kernel launch by a pair of HIP events while tracing is on.
struct TraceScope {
  TraceScope(const char *name, hipStream_t s);
  ~TraceScope();
  int slot;
  hipStream_t stream;
};

// ---------------------------------------------------------------- vocabulary pass
struct RowStat {        // softmax statistics of one chunk of one row of logits
  float max;            // max of z / T over the chunk
  int argmax;           // lowest id attaining it
  double sum;           // sum of exp(z / T - max) over the chunk
};

struct RowSel {         // one inverse-CDF draw per sequence
  const float *p_row;   // logits of p (never null)
  const float *q_row;   // logits of q, or null: draw from p
  double mp, sp;        // max and normaliser of p
  double mq, sq;        // max and normaliser of q
  double u;             // the uniform
  int32_t *dst;         // where the drawn id goes
  int active;           // 0: nothing to draw for this sequence
  int pad;
  // top-p: id x of a row is kept iff key(z_x) > key, or key(z_x) == key and x <= id
  // (key 0 with id INT32_MAX keeps every id); sp / sq are then the nucleus masses
  uint32_t pkey, qkey;
  int32_t pid, qid;
};

// Nucleus (top-p set) of one row of logits: the ids ranked by logit (larger first,
// the lower id first among equal logits) up to the first at which the running
// probability reaches top_p.  The kept ids are those whose order key (see
// order_key in vocab.hip) exceeds `key`, and those equal to it up to id `idt`.
struct NucRow {
  double m;             // reference exponent z_ref / T (float64)
  double s;             // the nucleus mass: sum of exp(z / T - m) over the kept ids
  uint32_t key;         // order key of the smallest kept logit
  int32_t idt;          // the largest kept id among the logits with that key
};

constexpr int kStatThreads = 256;
constexpr int kStatVec = 16;                                   // float4 per thread
constexpr int kStatChunk = kStatThreads * kStatVec * 4;       // 16384 ids per chunk
constexpr int kScanThreads = 256;
constexpr int kScanPer = 16;                                   // ids per thread
constexpr int kScanChunk = kScanThreads * kScanPer;           // 4096 ids per chunk

inline int stat_chunks(int V) { return (V + kStatChunk - 1) / kStatChunk; }
inline int scan_chunks(int V) { return (V + kScanChunk - 1) / kScanChunk; }

// Softmax statistics per tile of a logits row (RowStat per tile), the form the
// LM-head GEMM epilogue emits; a draw from such a row needs no further pass over
// the vocabulary.  The row's ids are cut into `strips` strips of 16 and the
// strips into `tiles` tiles: tile t holds strips [t S / T, (t + 1) S / T)
// (integer division).
constexpr int kStripIds = 16;
constexpr int kMaxTileStrips = 8;              // 128 ids (fixed tiles and the tiled GEMM's statistics)
// The draw scans the ids of one tile with kDrawRun consecutive ids per lane of a
// wave, so it takes tiles of up to kMaxDrawTileIds ids (the strip ranges of the
// draft head's LM head hold up to 160).
constexpr int kDrawRun = 3;
constexpr int kMaxDrawTileIds = kDrawRun * 64;
constexpr int kMaxTiles = 4096;                // the draw stages a row's tile statistics in 64 KiB of LDS
constexpr int kMaxVocab = kMaxTiles * kMaxTileStrips * kStripIds;
struct TileGeom {
  int strips, tiles;
};
__host__ __device__ inline int tile_first_strip(const TileGeom &g, int t) { return (int)((long)t * g.strips / g.tiles); }
// tiles of 8 strips (128 ids; the last may be shorter)
inline TileGeom fixed_tiles(int V) {
  const int S = (V + kStripIds - 1) / kStripIds;
  return TileGeom{S, (S + kMaxTileStrips - 1) / kMaxTileStrips};
}
// tile statistics by a pass over rows of logits (paths without the GEMM epilogue)
void launch_tile_stats(const float *logits, long row_stride, int n_rows, int V, float inv_t, TileGeom geo,
                       RowStat *tiles, hipStream_t s);
// one draw per row from softmax(z / T) given its tile statistics: argmax (greedy) or the
// inverse-CDF draw with u[b * u_stride]; writes dst[b * dst_stride]
// row_out (may be null): the row's combined statistics at row_out[b * row_stride_out]
// next (may be null): the same launch also writes the next chain step's MTP input row b
// (mtp_input_row with h + b * H and the drawn id) into out + b * 2 * H
struct DrawNextInput {
  int dtype, H;
  float eps;
  const float *h;
  const void *E, *norm_h, *norm_e;
  void *out;
  int32_t *dev_err;
};
void launch_tile_draw(int B, int V, int mode, float inv_t, const float *logits, long row_stride, TileGeom geo,
                      const RowStat *tiles, const float *u, int u_stride, int32_t *dst, int dst_stride,
                      RowStat *row_out, int row_stride_out, hipStream_t s, const DrawNextInput *next = nullptr);

// submax (may be null): also the raw-logit maxima of every run of kRecSub ids, [row][stat_chunks(V) * 64]
void launch_row_stats(const char *name, const float *logits, long row_stride, int n_rows, int V, float inv_t,
                      RowStat *out, hipStream_t s, float *submax = nullptr);
// cycle record: the top `topk` entries of softmax(z / T) for block rows 0..k-1 of each
// sequence, from the accept's row statistics (tstat) and run maxima (submax)
constexpr int kRecSub = 256;       // ids per run maximum (one wave's load in the row-statistics pass)
constexpr int kRecMaxTopk = 64;
void launch_record_topk(int B, int k, int V, float inv_t, int topk, const float *logits, const RowStat *tstat,
                        const float *submax, uint16_t *logp, int32_t *ids, hipStream_t s);
// one RowStat per row (at out[r * out_stride]) from `tiles` tile statistics per row
void launch_tile_combine(int n_rows, int tiles, const RowStat *st, RowStat *out, int out_stride, hipStream_t s);
// tstat / dstat hold nch_t / nch_d RowStats per target / draft row (chunk statistics, or one
// combined per row); tnuc / dnuc (top-p, else null): the nuclei of the target and draft rows
void launch_accept_decide(int B, int k, int V, int mode, float inv_t, double inv_td, const float *tlog,
                          const float *dlog, const RowStat *tstat, int nch_t, const RowStat *dstat, int nch_d,
                          const NucRow *tnuc, const NucRow *dnuc,
                          const int32_t *drafts, const float *u_accept, const float *u_final,
                          int32_t *n_accept, int32_t *out_tokens, RowSel *sel, hipStream_t s);
// top-p: the nucleus of rows r = 0..n_rows-1 at logits + r * row_stride, each with nch
// statistics (chunks or tiles) at st + r * nch, into out[r * out_stride]; 0 < top_p < 1.  part (may be null):
// kNucPartBytes of scratch that lets launches of few rows split their first pass
constexpr int kNucSplitRows = 256;     // rows x workgroups per row of a split first pass
constexpr int kNucMaxSplit = 8;
constexpr size_t kNucPartBytes = (size_t)kNucSplitRows * 4096 * 8;
void launch_nucleus(const char *name, int n_rows, int V, double inv_td, double top_p, const float *logits,
                    long row_stride, const RowStat *st, int nch, NucRow *out, int out_stride,
                    unsigned long long *part, hipStream_t s);
// sel[b] := a draw from the nucleus nuc[b * nuc_stride] of row b (logits + b * row_stride)
// with the uniform u[b * u_stride], into dst[b * dst_stride]
void launch_nucleus_select(int B, const float *logits, long row_stride, const NucRow *nuc, int nuc_stride,
                           const float *u, int u_stride, int32_t *dst, int dst_stride, RowSel *sel, hipStream_t s);
// nucleus false: every row of sel keeps every id (top-p 1), and the kernels skip the nucleus tests
void launch_residual_draw(const char *chunk_name, const char *scan_name, int B, int V, float inv_t, const RowSel *sel,
                          double *wsum, double *psum, bool nucleus, hipStream_t s);

// ---------------------------------------------------------------- KV index
void launch_kv_commit(int B, int k, int page_size, int max_pages, const int32_t *block_table,
                      int32_t *seq_lens, const int32_t *n_accept, int32_t *slots, hipStream_t s);

}  // namespace gm
