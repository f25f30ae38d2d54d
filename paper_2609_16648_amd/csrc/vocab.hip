// Vocabulary-pass kernels: softmax statistics, the accept rule (Sec. 2.2,
// Eq. accept-rule), the residual / bonus draw and the draft-head draw.
//
// Logits rows are read in place; no probability matrix is written.
//  1. row_stats: per (row, chunk of 16384 ids) the max of z/T, the lowest id
//     attaining it and sum exp(z/T - max) accumulated in float64.
//  2. accept_decide (one thread per sequence): combines the chunk statistics,
//     evaluates p_i(d_i) / q_i(d_i) in float64 from the two gathered logits,
//     rounds the ratio to float32, compares it with u and stops at the first
//     rejection; greedy mode compares d_i with the row argmax instead.  It
//     prepares one draw per sequence (residual max(0, p - q) at the first
//     rejection, p_{k+1} after a full accept).
//  3. residual_chunk + residual_scan: an inverse-CDF draw in ascending id
//     order (per-id exponentials in float32, normalisers, differences and
//     running sums in float64), first as chunk masses, then a scan inside the
//     chunk that holds u * Z.
//  4. tile_stats / tile_draw: per-tile statistics (tiles of at most 128 ids; also emitted by
//     the LM-head GEMM epilogue) and a draw that needs no pass over the row.
#include <float.h>

#include "common.h"
#include "launch.h"
#include "mtp_row.h"

namespace gm {

__device__ __forceinline__ uint32_t order_key(float x) {   // larger float, larger key (-0 as +0)
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// top-p: id x with logit z is in the nucleus (key, idt) (NucRow, RowSel)
__device__ __forceinline__ bool in_nucleus(float z, int x, uint32_t key, int idt) {
  const uint32_t k = order_key(z);
  return k > key || (k == key && x <= idt);
}

// ------------------------------------------------------------------ 1. row statistics
// submax (may be null): [row][n_chunks * 64] maxima of the raw logits over runs of
// kRecSub = 256 ids (one wave's float4 load), for the cycle record's selection.
__global__ __launch_bounds__(kStatThreads) __attribute__((amdgpu_waves_per_eu(5, 8))) void row_stats_kernel(const float *__restrict__ logits,
                                                                 long row_stride, int V, float inv_t,
                                                                 int n_chunks, RowStat *__restrict__ out,
                                                                 float *__restrict__ submax) {
  __shared__ float sm_max[kStatThreads / kWave];
  __shared__ int sm_arg[kStatThreads / kWave];
  __shared__ double sm_sum[kStatThreads / kWave];
  const int r = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  const float *row = logits + (long)r * row_stride;
  const int lo = c * kStatChunk;
  const int hi = min(V, lo + kStatChunk);
  const bool vec = ((V & 3) == 0) && ((row_stride & 3) == 0);

  // The raw logits stay in registers and z / T is formed where it is used (the same
  // product each time).  With no second copy, no per-load maxima kept and straight-line
  // loads for whole chunks the kernel fits five waves per SIMD (87 registers), so the
  // 2560 workgroups of 256 rows of the 151936-id vocabulary run in two full rounds
  // rather than two and a half.
  float f[kStatVec][4];
  if (vec && hi - lo == kStatChunk) {   // a whole chunk (uniform over the workgroup): plain vector loads
#pragma unroll
    for (int j = 0; j < kStatVec; ++j) {
      const float4 g = __builtin_bit_cast(float4, load_nt(row + lo + 4 * (tid + kStatThreads * j)));   // read once
      f[j][0] = g.x; f[j][1] = g.y; f[j][2] = g.z; f[j][3] = g.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kStatVec; ++j) {
      const int e = lo + 4 * (tid + kStatThreads * j);
      if (vec && e + 3 < hi) {
        const float4 g = __builtin_bit_cast(float4, load_nt(row + e));
        f[j][0] = g.x; f[j][1] = g.y; f[j][2] = g.z; f[j][3] = g.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) f[j][q] = (e + q < hi) ? row[e + q] : -INFINITY;
      }
    }
  }
  auto rmax = [&](int j) { return fmaxf(fmaxf(f[j][0], f[j][1]), fmaxf(f[j][2], f[j][3])); };
  if (submax) {
    // maxima of the 16 runs of 256 ids this wave loaded (run j: load j of the wave), by a
    // reduce-scatter over the lanes: after the rounds with masks 32..4 lane L holds run
    // (L >> 2) & 15 reduced over its lane group, then masks 2 and 1 finish the reduction
    const int lane = tid & 63;
    float m8[8], m4[4], m2[2], m1;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const bool hi_half = lane & 32;
      const float keep = hi_half ? rmax(8 + q) : rmax(q), send = hi_half ? rmax(q) : rmax(8 + q);
      m8[q] = fmaxf(keep, __shfl_xor(send, 32, kWave));
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool hi_half = lane & 16;
      const float keep = hi_half ? m8[4 + q] : m8[q], send = hi_half ? m8[q] : m8[4 + q];
      m4[q] = fmaxf(keep, __shfl_xor(send, 16, kWave));
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const bool hi_half = lane & 8;
      const float keep = hi_half ? m4[2 + q] : m4[q], send = hi_half ? m4[q] : m4[2 + q];
      m2[q] = fmaxf(keep, __shfl_xor(send, 8, kWave));
    }
    {
      const bool hi_half = lane & 4;
      const float keep = hi_half ? m2[1] : m2[0], send = hi_half ? m2[0] : m2[1];
      m1 = fmaxf(keep, __shfl_xor(send, 4, kWave));
    }
    m1 = fmaxf(m1, __shfl_xor(m1, 2, kWave));
    m1 = fmaxf(m1, __shfl_xor(m1, 1, kWave));
    if ((lane & 3) == 0) {
      const int j = (lane >> 2) & 15, w = tid >> 6;
      // run j of wave w covers ids lo + 1024 j + 256 w .. + 255
      submax[(long)blockIdx.x * n_chunks * 64 + (long)c * 64 + 4 * j + w] = m1;
    }
  }
  // max, then the lowest id attaining it, as two branch-free wave reductions.  Each
  // pass takes an opaque copy of 1/T, so the compiler recomputes z / T there instead
  // of keeping all 64 products live beside the logits.
  auto opaque_inv_t = [&]() { float t = inv_t; asm volatile("" : "+v"(t)); return t; };
  const float t1 = opaque_inv_t();
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < kStatVec; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) m = fmaxf(m, f[j][q] * t1);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
  int am = 0x7fffffff;
  const float t2 = opaque_inv_t();
#pragma unroll
  for (int j = kStatVec - 1; j >= 0; --j)
#pragma unroll
    for (int q = 3; q >= 0; --q) am = f[j][q] * t2 == m ? lo + 4 * (tid + kStatThreads * j) + q : am;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) am = min(am, __shfl_xor(am, o, kWave));
  const int lane = tid & 63, wid = tid >> 6;
  if (lane == 0) { sm_max[wid] = m; sm_arg[wid] = am; }
  __syncthreads();
  m = sm_max[0];
  am = sm_arg[0];
#pragma unroll
  for (int w = 1; w < kStatThreads / kWave; ++w)
    if (sm_max[w] > m || (sm_max[w] == m && sm_arg[w] < am)) { m = sm_max[w]; am = sm_arg[w]; }

  double s = 0.0;
  const float t3 = opaque_inv_t();
#pragma unroll
  for (int j = 0; j < kStatVec; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) s += (double)expf(f[j][q] * t3 - m);
  s = wave_sum(s);
  if (lane == 0) sm_sum[wid] = s;
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int w = 0; w < kStatThreads / kWave; ++w) t += sm_sum[w];
    RowStat o;
    o.max = m;
    o.argmax = am;
    o.sum = t;
    out[(long)r * n_chunks + c] = o;
  }
}

void launch_row_stats(const char *name, const float *logits, long row_stride, int n_rows, int V, float inv_t,
                      RowStat *out, hipStream_t s, float *submax) {
  if (n_rows <= 0) return;
  TraceScope ts(name, s);
  dim3 grid(n_rows, stat_chunks(V));
  hipLaunchKernelGGL(row_stats_kernel, grid, dim3(kStatThreads), 0, s, logits, row_stride, V, inv_t,
                     stat_chunks(V), out, submax);
}

// max, normaliser and lowest arg-max of a whole row from its chunk statistics
__device__ __forceinline__ void combine_stats(const RowStat *st, int nch, double &M, double &S, int &am) {
  float m = -INFINITY;
  int a = 0;
  for (int c = 0; c < nch; ++c)
    if (st[c].max > m) { m = st[c].max; a = st[c].argmax; }
  double s = 0.0;
  for (int c = 0; c < nch; ++c) s += st[c].sum * exp((double)st[c].max - (double)m);
  M = (double)m;
  S = s;
  am = a;
}

// One RowStat per row from its `tiles` tile statistics (ascending id ranges): the
// largest max, the lowest id attaining it, and the normaliser rescaled to that max in
// float64.  One wave per row; each lane takes every 64th tile in order, then fixed
// shuffle trees combine the lanes, so the result does not depend on timing.
__global__ __launch_bounds__(256) void tile_combine_kernel(int n_rows, int tiles, const RowStat *__restrict__ st,
                                                           RowStat *__restrict__ out, int out_stride) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n_rows) return;
  const RowStat *t = st + (long)row * tiles;
  float m = -INFINITY;
  int am = 0x7fffffff;
  for (int i = lane; i < tiles; i += kWave)
    if (t[i].max > m) { m = t[i].max; am = t[i].argmax; }   // ascending ids: the first of equal maxima wins
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float mo = __shfl_xor(m, o, kWave);
    const int ao = __shfl_xor(am, o, kWave);
    if (mo > m || (mo == m && ao < am)) { m = mo; am = ao; }
  }
  double s = 0.0;
  for (int i = lane; i < tiles; i += kWave) s += t[i].sum * exp((double)t[i].max - (double)m);
  s = wave_sum(s);
  if (lane == 0) {
    RowStat o;
    o.max = m;
    o.argmax = am;
    o.sum = s;
    out[(long)row * out_stride] = o;
  }
}

void launch_tile_combine(int n_rows, int tiles, const RowStat *st, RowStat *out, int out_stride, hipStream_t s) {
  if (n_rows <= 0) return;
  TraceScope ts("tile_combine", s);
  hipLaunchKernelGGL(tile_combine_kernel, dim3((n_rows + 3) / 4), dim3(256), 0, s, n_rows, tiles, st, out, out_stride);
}

// ------------------------------------------------------------------ 2. accept decision
// One wave per sequence.  Lane r <= k combines the chunk statistics of target
// row r, lane k + 1 + r those of draft row r; lane i < k then evaluates the
// test for draft i (all in parallel), and the first failing lane is the first
// rejection (the rule stops there, so later tests are not looked at).
__global__ __launch_bounds__(64) void accept_decide_kernel(int B, int k, int V, int mode, float inv_t,
                                                           double inv_td,
                                                           const float *__restrict__ tlog,
                                                           const float *__restrict__ dlog,
                                                           const RowStat *__restrict__ tstat,
                                                           const RowStat *__restrict__ dstat, int nch, int nch_d,
                                                           const NucRow *__restrict__ tnuc,
                                                           const NucRow *__restrict__ dnuc,
                                                           const int32_t *__restrict__ drafts,
                                                           const float *__restrict__ u_acc,
                                                           const float *__restrict__ u_fin,
                                                           int32_t *__restrict__ n_out, int32_t *__restrict__ out_tokens,
                                                           RowSel *__restrict__ sel) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int k1 = k + 1;
  // this lane's row: target rows 0..k, then draft rows 0..k-1 (sampling only)
  const bool is_t = lane < k1, is_d = mode != GM_GREEDY && lane >= k1 && lane < k1 + k;
  double M = 0.0, S = 1.0;
  int am = 0;
  uint32_t nkey = 0;
  int nid = 0x7fffffff;
  if (is_t || is_d) {
    const RowStat *st = is_t ? tstat + (long)(b * k1 + lane) * nch : dstat + (long)(b * k + lane - k1) * nch_d;
    combine_stats(st, is_t ? nch : nch_d, M, S, am);
    if (tnuc && mode != GM_GREEDY) {   // top-p: p and q are the rows' nuclei
      const NucRow nr = is_t ? tnuc[b * k1 + lane] : dnuc[b * k + lane - k1];
      M = nr.m;
      S = nr.s;
      nkey = nr.key;
      nid = nr.idt;
    }
  }
  const bool top_p = tnuc != nullptr && mode != GM_GREEDY;
  // the draft row statistics moved to the lane of the same position
  const double Mq = __shfl(M, k1 + lane < 64 ? k1 + lane : lane, kWave);
  const double Sq = __shfl(S, k1 + lane < 64 ? k1 + lane : lane, kWave);
  const uint32_t qkey = __shfl(nkey, k1 + lane < 64 ? k1 + lane : lane, kWave);
  const int qid = __shfl(nid, k1 + lane < 64 ? k1 + lane : lane, kWave);
  bool ok = false;   // lane i < k: draft i passes its test
  int d = -1;
  if (lane < k) {
    d = drafts[b * k + lane];
    if (mode == GM_GREEDY) {
      ok = d == am;
    } else if (d >= 0 && d < V) {
      const float rt = tlog[(long)(b * k1 + lane) * V + d], rq = dlog[(long)(b * k + lane) * V + d];
      double p, q;
      if (top_p) {     // p'(d), q'(d): zero outside the nucleus, exponents in float64
        p = in_nucleus(rt, d, nkey, nid) ? exp((double)rt * inv_td - M) / S : 0.0;
        q = in_nucleus(rq, d, qkey, qid) ? exp((double)rq * inv_td - Mq) / Sq : 0.0;
      } else {
        p = exp((double)(rt * inv_t) - M) / S;
        q = exp((double)(rq * inv_t) - Mq) / Sq;
      }
      const float ratio = q > 0.0 ? (float)(p / q) : INFINITY;
      ok = u_acc[b * k + lane] < ratio;
    }
  }
  const unsigned long long fail = __ballot(lane < k && !ok);
  const int n = fail ? __ffsll((long long)fail) - 1 : k;
  // lane n holds the statistics of target row n (and of draft row n, n < k)
  const double mp = __shfl(M, n, kWave), sp = __shfl(S, n, kWave);
  const double mq = __shfl(Mq, n, kWave), sq = __shfl(Sq, n, kWave);
  const uint32_t pkey_n = __shfl(nkey, n, kWave), qkey_n = __shfl(qkey, n, kWave);
  const int pid_n = __shfl(nid, n, kWave), qid_n = __shfl(qid, n, kWave);
  const int am_n = __shfl(am, n, kWave);
  if (lane < k1) {
    int tok = -1;
    if (lane < n) tok = d;
    else if (lane == n && mode == GM_GREEDY) tok = am_n;
    if (lane != n || mode == GM_GREEDY) out_tokens[b * k1 + lane] = tok;
  }
  if (lane == 0) {
    n_out[b] = n;
    RowSel rs;
    rs.active = 0;
    rs.q_row = nullptr;
    rs.mq = 0.0;
    rs.sq = 1.0;
    rs.pad = 0;
    rs.p_row = tlog + (long)(b * k1 + n) * V;
    rs.mp = mp;
    rs.sp = sp;
    rs.u = 0.0;
    rs.dst = out_tokens + b * k1 + n;
    rs.pkey = pkey_n;
    rs.pid = pid_n;
    rs.qkey = 0;
    rs.qid = 0x7fffffff;
    if (mode != GM_GREEDY) {
      if (n < k) {
        rs.q_row = dlog + (long)(b * k + n) * V;
        rs.mq = mq;
        rs.sq = sq;
        rs.qkey = qkey_n;
        rs.qid = qid_n;
      }
      rs.u = (double)u_fin[b];
      rs.active = 1;
    }
    sel[b] = rs;
  }
}

void launch_accept_decide(int B, int k, int V, int mode, float inv_t, double inv_td, const float *tlog,
                          const float *dlog, const RowStat *tstat, int nch_t, const RowStat *dstat, int nch_d,
                          const NucRow *tnuc, const NucRow *dnuc,
                          const int32_t *drafts, const float *u_accept, const float *u_final,
                          int32_t *n_accept, int32_t *out_tokens, RowSel *sel, hipStream_t s) {
  if (B <= 0) return;
  TraceScope ts("accept_decide", s);
  hipLaunchKernelGGL(accept_decide_kernel, dim3(B), dim3(64), 0, s, B, k, V, mode, inv_t, inv_td, tlog, dlog, tstat,
                     dstat, nch_t, nch_d, tnuc, dnuc, drafts, u_accept, u_final, n_accept, out_tokens, sel);
}

// ------------------------------------------------------------------ cycle record
// The record of a cycle keeps, per draft position, the target's top-k entries of
// p_i = softmax(z_i / T) as log-probabilities with the full-vocabulary
// normaliser, in bf16 (App. "Implementing Draft-Path Reconstruction in verl").
// One block per recorded row.  The topk-th largest run maximum T (runs of
// kRecSub ids, from the row-statistics pass) bounds the topk-th largest logit
// from below (the maxima of the topk largest runs are topk distinct ids >= T),
// so every kept entry is an id with z >= T inside a run whose maximum is >= T.
// Those candidates, typically a few per run, are keyed (logit, then lower id
// first), sorted in LDS, and the first topk kept.  When more than kRecCand
// qualify (heavy ties), a bisection on the logit's order key finds the topk-th
// value v exactly; the ids above v and then the lowest ids equal to v are taken.
constexpr int kRecCand = 4096;
constexpr int kRecMaxRuns = kMaxVocab / kRecSub;

__device__ __forceinline__ unsigned long long cand_key(float x, int id) {   // larger logit first, then lower id
  return ((unsigned long long)order_key(x) << 32) | (uint32_t)(0x7fffffff - id);
}

// descending bitonic sort of n (a power of two) keys in LDS by the whole block
template <typename K>
__device__ void block_sort_desc(K *a, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (int t = threadIdx.x; t < n / 2; t += blockDim.x) {
        const int lo = 2 * t - (t & (stride - 1)), hi = lo + stride;
        const K x = a[lo], y = a[hi];
        if ((lo & size) == 0 ? x < y : x > y) { a[lo] = y; a[hi] = x; }
      }
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(1024) void record_topk_kernel(int k, int V, float inv_t, int topk,
                                                          const float *__restrict__ logits,
                                                          const RowStat *__restrict__ tstat, int nch,
                                                          const float *__restrict__ submax,
                                                          uint16_t *__restrict__ out_logp,
                                                          int32_t *__restrict__ out_ids) {
  __shared__ __attribute__((aligned(16))) float runs[kRecMaxRuns];
  __shared__ __attribute__((aligned(16))) unsigned long long cand[kRecCand];
  __shared__ unsigned long long top[kRecMaxTopk];
  __shared__ int qual[kRecMaxRuns];   // the runs whose maximum is >= T
  __shared__ int sh_cnt, sh_nq;
  __shared__ float sh_T;
  __shared__ double sh_M, sh_lse;
  const int bi = blockIdx.x, b = bi / k, i = bi % k;
  const long row = (long)b * (k + 1) + i;   // the block row that verifies draft i
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, nw = blockDim.x >> 6;
  const int nrun = nch * 64;
  const float *z = logits + row * V;
  for (int t = tid; t < nrun; t += blockDim.x) runs[t] = submax[row * nrun + t];
  if (tid == 0) {
    double M, S;
    int am;
    combine_stats(tstat + row * nch, nch, M, S, am);
    sh_M = M;
    sh_lse = log(S);
    sh_cnt = 0;
    sh_nq = 0;
  }
  __syncthreads();
  // T: the topk-th largest run maximum, i.e. a maximum with fewer than topk maxima above
  // it and at least topk at or above it (every such maximum has the same value)
  for (int t = tid; t < nrun; t += blockDim.x) {   // nrun is a multiple of 64
    const float m = runs[t];
    int gt = 0, ge = 0;
    const float4 *r4 = reinterpret_cast<const float4 *>(runs);
    for (int j = 0; j < nrun / 4; j += 4) {
      float4 r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) r[u] = r4[j + u];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        gt += (r[u].x > m) + (r[u].y > m) + (r[u].z > m) + (r[u].w > m);
        ge += (r[u].x >= m) + (r[u].y >= m) + (r[u].z >= m) + (r[u].w >= m);
      }
    }
    if (gt < topk && ge >= topk) sh_T = m;
  }
  __syncthreads();
  const float T = sh_T;
  for (int r = tid; r < nrun; r += blockDim.x)
    if (runs[r] >= T) qual[atomicAdd(&sh_nq, 1)] = r;
  __syncthreads();
  // every 4-id group of the qualifying runs, spread over the whole block, 8 groups per
  // thread in flight at once
  const int ngroups = sh_nq * (kRecSub / 4);
  for (int g0 = tid; g0 < ngroups; g0 += 8 * blockDim.x) {
    float v[8][4];
    int xb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int g = g0 + u * blockDim.x;
      xb[u] = g < ngroups ? qual[g / (kRecSub / 4)] * kRecSub + 4 * (g % (kRecSub / 4)) : V;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[u][q] = xb[u] + q < V ? z[xb[u] + q] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (xb[u] + q < V && v[u][q] >= T) {
          const int pos = atomicAdd(&sh_cnt, 1);
          if (pos < kRecCand) cand[pos] = cand_key(v[u][q], xb[u] + q);
        }
      }
    }
  }
  __syncthreads();
  const int cnt = sh_cnt;   // at least topk
  if (cnt <= 512) {
    // few candidates: each one's rank is the number of larger keys (keys are distinct;
    // the padding keys are 0, below every candidate)
    const int c8 = (cnt + 7) & ~7;
    for (int t = cnt + tid; t < c8; t += blockDim.x) cand[t] = 0ull;
    __syncthreads();
    for (int t = tid; t < cnt; t += blockDim.x) {
      const unsigned long long key = cand[t];
      int rank = 0;
      for (int j = 0; j < c8; j += 8) {
        unsigned long long c[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) c[u] = cand[j + u];
#pragma unroll
        for (int u = 0; u < 8; ++u) rank += c[u] > key;
      }
      if (rank < topk) top[rank] = key;
    }
    __syncthreads();
    for (int t = tid; t < topk; t += blockDim.x) cand[t] = top[t];
    __syncthreads();
  } else if (cnt <= kRecCand) {
    int c2 = 64;
    while (c2 < cnt) c2 <<= 1;
    for (int t = cnt + tid; t < c2; t += blockDim.x) cand[t] = 0ull;
    block_sort_desc(cand, c2);
  } else {
    // the largest order key v with at least topk ids at or above it
    __shared__ int sh_c;
    uint32_t lo_k = order_key(T), hi_k = 0xffffffffu;
    while (lo_k < hi_k) {
      const uint32_t mid = lo_k + (uint32_t)(((unsigned long long)hi_k - lo_k + 1) / 2);
      if (tid == 0) sh_c = 0;
      __syncthreads();
      int local = 0;
      for (int r = w; r < nrun; r += nw) {
        if (!(runs[r] >= T)) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int x = r * kRecSub + 4 * lane + q;
          if (x < V && order_key(z[x]) >= mid) ++local;
        }
      }
      atomicAdd(&sh_c, local);
      __syncthreads();
      if (sh_c >= topk) lo_k = mid;
      else hi_k = mid - 1;
      __syncthreads();
    }
    const uint32_t vk = lo_k;
    if (tid == 0) sh_cnt = 0;
    __syncthreads();
    for (int r = w; r < nrun; r += nw) {   // the ids above v: fewer than topk
      if (!(runs[r] >= T)) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int x = r * kRecSub + 4 * lane + q;
        if (x < V && order_key(z[x]) > vk) cand[atomicAdd(&sh_cnt, 1)] = cand_key(z[x], x);
      }
    }
    __syncthreads();
    const int gt = sh_cnt;
    if (w == 0) {   // then the lowest ids equal to v, walking the runs in id order
      int taken = 0;
      for (int r = 0; r < nrun && taken < topk - gt; ++r) {
        if (!(runs[r] >= T)) continue;
        const int x0 = r * kRecSub + 4 * lane;
        bool hit[4];
        int m = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          hit[q] = x0 + q < V && order_key(z[x0 + q]) == vk;
          m += hit[q];
        }
        int pre = m;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int n = __shfl_up(pre, o, kWave);
          if (lane >= o) pre += n;
        }
        const int tot = __shfl(pre, 63, kWave);
        int rank = taken + pre - m;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (hit[q]) {
            if (rank < topk - gt) cand[gt + rank] = cand_key(z[x0 + q], x0 + q);
            ++rank;
          }
        }
        taken += tot;
      }
    }
    __syncthreads();
    for (int t = topk + tid; t < 64; t += blockDim.x) cand[t] = 0ull;
    block_sort_desc(cand, 64);
  }
  for (int t = tid; t < topk; t += blockDim.x) {
    const int id = 0x7fffffff - (int)(uint32_t)cand[t];
    const double lp = (double)(z[id] * inv_t) - sh_M - sh_lse;   // the statistics' float32 z / T
    out_logp[(long)bi * topk + t] = f32_to_bf16((float)lp);
    out_ids[(long)bi * topk + t] = id;
  }
}

void launch_record_topk(int B, int k, int V, float inv_t, int topk, const float *logits, const RowStat *tstat,
                        const float *submax, uint16_t *logp, int32_t *ids, hipStream_t s) {
  if (B <= 0 || k <= 0) return;
  TraceScope ts("record_topk", s);
  hipLaunchKernelGGL(record_topk_kernel, dim3(B * k), dim3(1024), 0, s, k, V, inv_t, topk, logits, tstat,
                     stat_chunks(V), submax, logp, ids);
}

// ------------------------------------------------------------------ top-p nucleus
// The evaluation setting of the paper decodes with top-p truncation (App.
// "Evaluation Configuration"): the kept ids of a row are those ranked by logit
// (larger first, lower id first among equal logits) up to the first at which the
// running probability reaches top_p.  One 1024-thread block per row finds the
// last kept id by a radix selection on the order key of the raw logits, carrying
// probability mass: each id weighs exp(z / T - m) in float64 (m = z_ref / T of
// the row's argmax), held as an unsigned fixed-point integer of 2^-44 units, so
// the LDS histogram sums are exact and independent of the order of the atomic
// adds.  Three passes over the row bin the key by its top 12 bits, the next 12
// and the last 8; each pass ranks the bins from the top and keeps the one where
// the running mass (plus that of every larger key) first reaches top_p times the
// row's mass.  Ids equal to the boundary logit weigh the same, so the number of
// them the nucleus needs follows from the masses; only when it keeps some but
// not all of them is the id of the last one looked for.  The second pass only
// gathers the logits and ids of the boundary's 12-bit bin into LDS; the finer
// bins and the ties are then taken from there (a bin too large for LDS takes
// passes over the row instead).
constexpr int kNucThreads = 1024;
constexpr int kNucBins = 4096;
constexpr int kNucQueue = 12288;     // logits and ids of the boundary's 12-bit bin kept in LDS (96 KiB)
constexpr int kNucTieRank = 2048;    // ties at the boundary ranked in LDS (more: a pass over the row)

// exp(y) for -32 <= y <= 0 by Tang's table-driven reduction (ACM TOMS 15(2), 1989):
// y = (64 q + j) ln2 / 64 + r with |r| <= ln2 / 128, exp(y) = 2^q 2^(j/64) exp(r), and
// exp(r) by its Taylor polynomial to r^6 (truncation below 2^-64 at |r| <= ln2 / 128).
// ln2 / 64 is split into a 32-bit head (k times it is exact for |k| < 2^21) and a tail;
// tab[j] = 2^(j/64), filled per block (nuc_exp_table).  A few ulps in all, far below
// the 2^-44 units the masses are rounded to.
__device__ __forceinline__ double nuc_exp(double y, const double *tab) {
  constexpr double kLn2Hi = 0x1.62e42feep-1 / 64.0, kLn2Lo = 0x1.a39ef35793c76p-33 / 64.0;
  const double kd = rint(y * (64.0 / 0x1.62e42fefa39efp-1));
  double r = fma(-kd, kLn2Hi, y);
  r = fma(-kd, kLn2Lo, r);
  double p = 1.0 / 720.0;
  p = fma(p, r, 1.0 / 120.0);
  p = fma(p, r, 1.0 / 24.0);
  p = fma(p, r, 1.0 / 6.0);
  p = fma(p, r, 0.5);
  p = fma(p, r, 1.0);
  p = fma(p, r, 1.0);
  const int k = (int)kd;
  return ldexp(tab[k & 63] * p, k >> 6);
}

// the block's table of 2^(j/64), j = 0..63 (before the block's first barrier)
__device__ __forceinline__ void nuc_exp_table(double *tab) {
  if (threadIdx.x < 64) tab[threadIdx.x] = exp2((double)threadIdx.x / 64.0);
}

// mass of one id in 2^-44 units (the same operations at every call: no contraction)
__device__ __forceinline__ unsigned long long nuc_mass(float v, double inv_td, double m, const double *tab) {
#pragma clang fp contract(off)
  const double y = (double)v * inv_td - m;
  if (!(y >= -32.0)) return 0ull;          // exp(-32) 2^44 < 0.5: rounds to 0 (and -inf, NaN)
  // exp(y) 2^44 < 2^52: adding 2^52 leaves its nearest integer (ties to even) in the
  // low mantissa bits
  const double t = nuc_exp(y, tab) * 0x1p44 + 0x1p52;
  return (unsigned long long)(__double_as_longlong(t) - 0x4330000000000000ll);
}

__device__ __forceinline__ float key_value(uint32_t k) {   // inverse of order_key
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// exclusive prefix sum of one value per thread over the block; wtot >= 16 entries
__device__ __forceinline__ unsigned long long block_excl_scan_u64(unsigned long long v, unsigned long long *wtot) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  unsigned long long x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long n = __shfl_up(x, o, kWave);
    if (lane >= o) x += n;
  }
  __syncthreads();
  if (lane == 63) wtot[wid] = x;
  __syncthreads();
  unsigned long long off = 0;
  for (int w = 0; w < wid && w < nw; ++w) off += wtot[w];
  return off + x - v;
}

// The bin, ranking nbins bins from the highest key down, at which the running mass
// (starting from `above`) first reaches thr; writes it and the mass before it.  The
// running sums are exact integers, so exactly one bin qualifies when
// above < thr <= above + the bins' total.
__device__ void nuc_find_bin(const unsigned long long *hist, int nbins, unsigned long long above, double thr,
                             unsigned long long *wtot, int *sh_bin, unsigned long long *sh_above) {
  const int tid = threadIdx.x;
  const int per = (nbins + kNucThreads - 1) / kNucThreads;
  unsigned long long g = 0;
  for (int j = 0; j < per; ++j) {
    const int b = nbins - 1 - (tid * per + j);
    if (b >= 0) g += hist[b];
  }
  unsigned long long cum = above + block_excl_scan_u64(g, wtot);
  for (int j = 0; j < per; ++j) {
    const int b = nbins - 1 - (tid * per + j);
    if (b < 0) break;
    const unsigned long long nb = cum + hist[b];
    if ((double)cum < thr && (double)nb >= thr) {
      *sh_bin = b;
      *sh_above = cum;
    }
    cum = nb;
  }
  __syncthreads();
}

// f(v, x) for every id x of a row, with four 16-byte loads in flight per thread
// (rows whose ids are 16-byte aligned), else one float per load, four in flight
template <typename F>
__device__ __forceinline__ void nuc_visit(const float *__restrict__ row, int V, bool vec, F &&f) {
  const int tid = threadIdx.x;
  if (vec) {
    constexpr int kStep = kNucThreads * 16;
    for (int x0 = tid * 4; x0 < V; x0 += kStep) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int x = x0 + u * kNucThreads * 4;
        v[u] = x < V ? *reinterpret_cast<const float4 *>(row + x) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int x = x0 + u * kNucThreads * 4;
        if (x < V) {
          f(v[u].x, x);
          f(v[u].y, x + 1);
          f(v[u].z, x + 2);
          f(v[u].w, x + 3);
        }
      }
    }
  } else {
    for (int x0 = tid; x0 < V; x0 += 4 * kNucThreads) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int x = x0 + u * kNucThreads;
        v[u] = x < V ? row[x] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (x0 + u * kNucThreads < V) f(v[u], x0 + u * kNucThreads);
    }
  }
}

// The reference exponent of a row: z / T (float64) of its maximum, the lowest id
// attaining the largest statistic among its nch chunk or tile statistics.  Holds a
// barrier: the caller's LDS writes before it are visible to the block after it.
__device__ double nuc_reference(const float *__restrict__ row, const RowStat *__restrict__ st, int nch, int V,
                                double inv_td, float *red_m, int *red_a) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  float bm = -INFINITY;
  int ba = 0x7fffffff;
  for (int c = tid; c < nch; c += kNucThreads) {
    const RowStat x = st[c];
    if (x.max > bm || (x.max == bm && x.argmax < ba)) {
      bm = x.max;
      ba = x.argmax;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(bm, o, kWave);
    const int oa = __shfl_xor(ba, o, kWave);
    if (om > bm || (om == bm && oa < ba)) {
      bm = om;
      ba = oa;
    }
  }
  if (lane == 0) {
    red_m[wid] = bm;
    red_a[wid] = ba;
  }
  __syncthreads();
  bm = red_m[0];
  ba = red_a[0];
  for (int w = 1; w < kNucThreads / 64; ++w)
    if (red_m[w] > bm || (red_m[w] == bm && red_a[w] < ba)) {
      bm = red_m[w];
      ba = red_a[w];
    }
  if (ba < 0 || ba >= V) ba = 0;
  return (double)row[ba] * inv_td;
}

// Pass 1 of the selection split over S workgroups per row, for launches with too
// few rows to fill the chip: workgroup (r, s) writes the histogram of its slice of
// row r (ids [lo, hi), lo and hi multiples of 4) to part[(r S + s) kNucBins ...];
// the selection sums the S of them (exact integers: the same result as one pass).
__global__ __launch_bounds__(kNucThreads) void nucleus_hist_kernel(int V, double inv_td,
                                                                   const float *__restrict__ logits, long row_stride,
                                                                   const RowStat *__restrict__ st, int nch, int S,
                                                                   unsigned long long *__restrict__ part) {
  __shared__ unsigned long long hist[kNucBins];
  __shared__ float red_m[kNucThreads / 64];
  __shared__ int red_a[kNucThreads / 64];
  __shared__ double etab[64];
  const int r = blockIdx.x / S, sg = blockIdx.x % S, tid = threadIdx.x;
  const float *row = logits + (long)r * row_stride;
  nuc_exp_table(etab);
  for (int b = tid; b < kNucBins; b += kNucThreads) hist[b] = 0ull;
  const double m = nuc_reference(row, st + (long)r * nch, nch, V, inv_td, red_m, red_a);
  const int lo = (int)(((long)V * sg / S) & ~3l), hi = sg + 1 == S ? V : (int)(((long)V * (sg + 1) / S) & ~3l);
  const bool vec = (V & 3) == 0 && (row_stride & 3) == 0 && (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  nuc_visit(row + lo, hi - lo, vec, [&](float v, int) {
    const unsigned long long e = nuc_mass(v, inv_td, m, etab);
    if (e) atomicAdd(&hist[order_key(v) >> 20], e);
  });
  __syncthreads();
  unsigned long long *dst = part + ((long)r * S + sg) * kNucBins;
  for (int b = tid; b < kNucBins; b += kNucThreads) dst[b] = hist[b];
}

__global__ __launch_bounds__(kNucThreads) void nucleus_kernel(int V, double inv_td, double top_p,
                                                              const float *__restrict__ logits, long row_stride,
                                                              const RowStat *__restrict__ st, int nch,
                                                              const unsigned long long *__restrict__ part, int S,
                                                              NucRow *__restrict__ out, int out_stride) {
  __shared__ unsigned long long hist[kNucBins];
  __shared__ float qv[kNucQueue];
  __shared__ int qx[kNucQueue];
  __shared__ unsigned sh_qn;
  __shared__ unsigned long long wtot[kNucThreads / 64];
  __shared__ float red_m[kNucThreads / 64];
  __shared__ int red_a[kNucThreads / 64];
  __shared__ int sh_bin, sh_idt;
  __shared__ unsigned long long sh_above;
  __shared__ double etab[64];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const float *row = logits + (long)r * row_stride;

  nuc_exp_table(etab);
  for (int b = tid; b < kNucBins; b += kNucThreads) hist[b] = 0ull;
  const double m = nuc_reference(row, st + (long)r * nch, nch, V, inv_td, red_m, red_a);

  // pass 1: the top 12 bits of the key (or the sum of the S slices' histograms)
  const bool vec = (V & 3) == 0 && (row_stride & 3) == 0 && (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  if (part) {
    const unsigned long long *src = part + (long)r * S * kNucBins;
    for (int b = tid; b < kNucBins; b += kNucThreads) {
      unsigned long long t = 0;
      for (int sg = 0; sg < S; ++sg) t += src[(long)sg * kNucBins + b];
      hist[b] = t;
    }
  } else {
    nuc_visit(row, V, vec, [&](float v, int) {
      const unsigned long long e = nuc_mass(v, inv_td, m, etab);
      if (e) atomicAdd(&hist[order_key(v) >> 20], e);
    });
  }
  __syncthreads();
  unsigned long long tot = 0;
  {
    unsigned long long g = 0;
    for (int b = tid; b < kNucBins; b += kNucThreads) g += hist[b];
    tot = block_excl_scan_u64(g, wtot);   // the last thread holds the total of the others
    tot += g;
    __syncthreads();
    if (tid == kNucThreads - 1) sh_above = tot;
    __syncthreads();
    tot = sh_above;
  }
  if (tot == 0) {           // no mass (every logit -inf or NaN): keep every id
    if (tid == 0) out[(long)r * out_stride] = NucRow{m, 0.0, 0u, 0x7fffffff};
    return;
  }
  const double thr = top_p * (double)tot;
  nuc_find_bin(hist, kNucBins, 0ull, thr, wtot, &sh_bin, &sh_above);
  const uint32_t b1 = (uint32_t)sh_bin;
  unsigned long long above = sh_above;

  // pass 2: the logits of bin b1 (a few percent of the row) gathered into LDS, so that
  // the masses of the finer bins are taken by full waves, and the last bits need no
  // further pass over the row; more than kNucQueue of them (heavy ties, narrow rows of
  // equal logits) take the two finer passes over the row instead
  if (tid == 0) sh_qn = 0u;
  for (int b = tid; b < kNucBins; b += kNucThreads) hist[b] = 0ull;
  __syncthreads();
  nuc_visit(row, V, vec, [&](float v, int x) {
    if ((order_key(v) >> 20) == b1) {
      const unsigned slot = atomicAdd(&sh_qn, 1u);
      if (slot < kNucQueue) {
        qv[slot] = v;
        qx[slot] = x;
      }
    }
  });
  __syncthreads();
  const unsigned qn = sh_qn;
  const bool queued = qn <= (unsigned)kNucQueue;
  if (queued) {
    for (unsigned i = tid; i < qn; i += kNucThreads) {
      const float v = qv[i];
      atomicAdd(&hist[(order_key(v) >> 8) & 0xfffu], nuc_mass(v, inv_td, m, etab));
    }
  } else {
    nuc_visit(row, V, vec, [&](float v, int) {
      const uint32_t k = order_key(v);
      if ((k >> 20) == b1) atomicAdd(&hist[(k >> 8) & 0xfffu], nuc_mass(v, inv_td, m, etab));
    });
  }
  __syncthreads();
  nuc_find_bin(hist, kNucBins, above, thr, wtot, &sh_bin, &sh_above);
  const uint32_t pre = (b1 << 12) | (uint32_t)sh_bin;
  above = sh_above;

  // pass 3: the last 8 bits
  for (int b = tid; b < 256; b += kNucThreads) hist[b] = 0ull;
  __syncthreads();
  if (queued) {
    for (unsigned i = tid; i < qn; i += kNucThreads) {
      const float v = qv[i];
      const uint32_t k = order_key(v);
      if ((k >> 8) == pre) atomicAdd(&hist[k & 0xffu], nuc_mass(v, inv_td, m, etab));
    }
  } else {
    nuc_visit(row, V, vec, [&](float v, int) {
      const uint32_t k = order_key(v);
      if ((k >> 8) == pre) atomicAdd(&hist[k & 0xffu], nuc_mass(v, inv_td, m, etab));
    });
  }
  __syncthreads();
  nuc_find_bin(hist, 256, above, thr, wtot, &sh_bin, &sh_above);
  const uint32_t key = (pre << 8) | (uint32_t)sh_bin;
  above = sh_above;
  const unsigned long long hk = hist[sh_bin];          // cnt ids of equal mass et
  const unsigned long long et = nuc_mass(key_value(key), inv_td, m, etab);
  const long long cnt = et ? (long long)(hk / et) : 1;
  // the fewest of them that reach thr (at least one, at most all)
  long long j = (long long)ceil((thr - (double)above) / (double)et);
  if (j < 1) j = 1;
  if (j > cnt) j = cnt;
  while (j > 1 && (double)(above + (unsigned long long)(j - 1) * et) >= thr) --j;
  while (j < cnt && (double)(above + (unsigned long long)j * et) < thr) ++j;
  int idt = 0x7fffffff;
  if (j < cnt && queued && cnt <= kNucTieRank) {
    // the j-th lowest id with this key, from the gathered bin: the ids of the ties are
    // listed in LDS (the histogram's memory), and the one with j - 1 lower ids is kept
    int *ties = reinterpret_cast<int *>(hist);
    if (tid == 0) {
      sh_qn = 0u;
      sh_idt = 0x7fffffff;
    }
    __syncthreads();
    for (unsigned i = tid; i < qn; i += kNucThreads)
      if (order_key(qv[i]) == key) {
        const unsigned slot = atomicAdd(&sh_qn, 1u);
        if (slot < (unsigned)kNucTieRank) ties[slot] = qx[i];
      }
    __syncthreads();
    const int nt = (int)min(sh_qn, (unsigned)kNucTieRank);
    for (int i = tid; i < nt; i += kNucThreads) {
      const int x = ties[i];
      int below = 0;
      for (int i2 = 0; i2 < nt; ++i2) below += ties[i2] < x;
      if (below == j - 1) sh_idt = x;
    }
    __syncthreads();
    idt = sh_idt;
  } else if (j < cnt) {
    // pass 4: the j-th lowest id with this key (contiguous id ranges per thread)
    if (tid == 0) sh_idt = 0x7fffffff;   // set before the scan's barriers
    const int per = (V + kNucThreads - 1) / kNucThreads;
    const int lo = tid * per, hi = min(V, lo + per);
    unsigned long long c = 0;
    for (int x = lo; x < hi; ++x) c += order_key(row[x]) == key;
    const unsigned long long before = block_excl_scan_u64(c, wtot);
    if (before < (unsigned long long)j && (unsigned long long)j <= before + c) {
      unsigned long long n = before;
      for (int x = lo; x < hi; ++x)
        if (order_key(row[x]) == key && ++n == (unsigned long long)j) {
          sh_idt = x;
          break;
        }
    }
    __syncthreads();
    idt = sh_idt;
  }
  if (tid == 0) out[(long)r * out_stride] = NucRow{m, (double)(above + (unsigned long long)j * et) * 0x1p-44, key, idt};
}

void launch_nucleus(const char *name, int n_rows, int V, double inv_td, double top_p, const float *logits,
                    long row_stride, const RowStat *st, int nch, NucRow *out, int out_stride,
                    unsigned long long *part, hipStream_t s) {
  if (n_rows <= 0) return;
  TraceScope ts(name, s);
  // fewer than 128 rows leave CUs idle: their first pass is split over up to 8 workgroups per row
  int S = part ? kNucSplitRows / n_rows : 1;
  if (S > kNucMaxSplit) S = kNucMaxSplit;
  if (S < 2 || V < S * 4096) S = 1;
  if (S > 1)
    hipLaunchKernelGGL(nucleus_hist_kernel, dim3(n_rows * S), dim3(kNucThreads), 0, s, V, inv_td, logits, row_stride,
                       st, nch, S, part);
  hipLaunchKernelGGL(nucleus_kernel, dim3(n_rows), dim3(kNucThreads), 0, s, V, inv_td, top_p, logits, row_stride, st,
                     nch, S > 1 ? part : nullptr, S, out, out_stride);
}

__global__ void nucleus_select_kernel(int B, const float *__restrict__ logits, long row_stride,
                                      const NucRow *__restrict__ nuc, int nuc_stride, const float *__restrict__ u,
                                      int u_stride,
                                      int32_t *dst, int dst_stride, RowSel *__restrict__ sel) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const NucRow n = nuc[(long)b * nuc_stride];
  RowSel rs;
  rs.p_row = logits + (long)b * row_stride;
  rs.q_row = nullptr;
  rs.mp = n.m;
  rs.sp = n.s;
  rs.mq = 0.0;
  rs.sq = 1.0;
  rs.u = (double)u[(long)b * u_stride];
  rs.dst = dst + (long)b * dst_stride;
  rs.active = 1;
  rs.pad = 0;
  rs.pkey = n.key;
  rs.pid = n.idt;
  rs.qkey = 0;
  rs.qid = 0x7fffffff;
  sel[b] = rs;
}

void launch_nucleus_select(int B, const float *logits, long row_stride, const NucRow *nuc, int nuc_stride,
                           const float *u, int u_stride, int32_t *dst, int dst_stride, RowSel *sel, hipStream_t s) {
  if (B <= 0) return;
  hipLaunchKernelGGL(nucleus_select_kernel, dim3((B + 63) / 64), dim3(64), 0, s, B, logits, row_stride, nuc,
                     nuc_stride, u, u_stride, dst, dst_stride, sel);
}

// ------------------------------------------------------------------ 3. inverse-CDF draw
// Weight of id x: max(0, p(x) - q(x)) with q, p(x) without.  Each exponential is a
// float32 expf of z / T - max (both float32); scaling by the float64 normaliser
// and every sum are float64.
// the raw logits of kScanPer consecutive ids of one row (float4 loads when the row
// allows; -inf past the end)
__device__ __forceinline__ void load_run(const float *row, int x0, int V, float (&r)[kScanPer]) {
  if ((V & 3) == 0 && x0 + kScanPer <= V) {
#pragma unroll
    for (int j = 0; j < kScanPer; j += 4) {
      const float4 f = *reinterpret_cast<const float4 *>(row + x0 + j);
      r[j] = f.x;
      r[j + 1] = f.y;
      r[j + 2] = f.z;
      r[j + 3] = f.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) r[j] = x0 + j < V ? row[x0 + j] : -INFINITY;
  }
}

// the draw weight of id x (max(0, p - q), or p alone) and its p; under top-p, ids outside
// a row's nucleus weigh 0 in it.  NUC false (top-p 1, every row keeps every id): the same
// weights without the nucleus tests, which are about a quarter of the pass's ALU work.
template <bool NUC>
__device__ __forceinline__ void id_weight(const RowSel &s, int x, int V, float zp, float zq, bool with_q, float inv_t,
                                          float mp, float mq, double isp, double isq, double &w, double &px) {
  const bool kp = x < V && (!NUC || in_nucleus(zp, x, s.pkey, s.pid));
  px = kp ? (double)expf(zp * inv_t - mp) * isp : 0.0;
  w = px;
  if (with_q) {
    const bool kq = x < V && (!NUC || in_nucleus(zq, x, s.qkey, s.qid));
    const double qx = kq ? (double)expf(zq * inv_t - mq) * isq : 0.0;
    w = fmax(px - qx, 0.0);
  }
}

// the kScanPer draw weights of one thread's run and the sum of their p
template <bool NUC>
__device__ __forceinline__ void run_weights(const RowSel &s, int x0, int V, float inv_t, bool use_p, double isp,
                                            double isq, double (&w)[kScanPer], double &psum) {
  float rp[kScanPer], rq[kScanPer];
  load_run(s.p_row, x0, V, rp);
  const bool with_q = !use_p && s.q_row != nullptr;
  if (with_q) load_run(s.q_row, x0, V, rq);
  const float mp = (float)s.mp, mq = (float)s.mq;
  psum = 0.0;
  double px;
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    id_weight<NUC>(s, x0 + j, V, rp[j], rq[j], with_q, inv_t, mp, mq, isp, isq, w[j], px);
    psum += px;
  }
}

// the same run summed as it is formed: the sums the scan kernel takes over run_weights'
// weights, in the same order, without holding the kScanPer weights
template <bool NUC>
__device__ __forceinline__ void run_sums(const RowSel &s, int x0, int V, float inv_t, double isp, double isq,
                                         double &wsum, double &psum) {
  float rp[kScanPer], rq[kScanPer];
  load_run(s.p_row, x0, V, rp);
  const bool with_q = s.q_row != nullptr;
  if (with_q) load_run(s.q_row, x0, V, rq);
  const float mp = (float)s.mp, mq = (float)s.mq;
  psum = 0.0;
  wsum = 0.0;
  double w, px;
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) {
    id_weight<NUC>(s, x0 + j, V, rp[j], rq[j], with_q, inv_t, mp, mq, isp, isq, w, px);
    psum += px;
    wsum += w;
  }
}

// Inclusive prefix sum of one double per thread over the block (256 threads).
__device__ __forceinline__ double block_incl_scan(double v, double *wsum /* >= 4 */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(v, o, kWave);
    if (lane >= o) v += n;
  }
  if (lane == 63) wsum[wid] = v;
  __syncthreads();
  double off = 0.0;
  for (int w = 0; w < wid; ++w) off += wsum[w];
  return off + v;
}

// per-thread sums over kScanPer consecutive ids, then a block-wide inclusive scan
// over the threads (the same code in both kernels, so a chunk's mass is exactly
// the last running sum of the scan inside it)
template <bool NUC>
__global__ __launch_bounds__(kScanThreads) void residual_chunk_kernel(int V, float inv_t,
                                                                      const RowSel *__restrict__ sel,
                                                                      int nch, double *__restrict__ wsum,
                                                                      double *__restrict__ psum) {
  __shared__ double sw[kScanThreads / kWave], sp[kScanThreads / kWave];
  const int b = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  const RowSel s = sel[b];
  if (!s.active) return;
  const int x0 = c * kScanChunk + tid * kScanPer;
  const double isp = 1.0 / s.sp, isq = 1.0 / s.sq;
  double w, p;
  run_sums<NUC>(s, x0, V, inv_t, isp, isq, w, p);
  const double tw = block_incl_scan(w, sw);
  const double tp = block_incl_scan(p, sp);
  if (tid == kScanThreads - 1) {
    wsum[(long)b * nch + c] = tw;
    psum[(long)b * nch + c] = tp;
  }
}

template <bool NUC>
__global__ __launch_bounds__(kScanThreads) void residual_scan_kernel(int V, float inv_t,
                                                                     const RowSel *__restrict__ sel, int nch,
                                                                     const double *__restrict__ wsum,
                                                                     const double *__restrict__ psum) {
  extern __shared__ double chunk_sh[];   // [2 nch]: residual masses, then p masses
  __shared__ double st[kScanThreads / kWave];
  __shared__ double sh_t, sh_base;
  __shared__ int sh_chunk, sh_thread, sh_last, sh_use_p;
  const int b = blockIdx.x, tid = threadIdx.x;
  const RowSel s = sel[b];
  if (!s.active) return;
  for (int c = tid; c < nch; c += kScanThreads) {   // all chunk masses in flight at once
    chunk_sh[c] = wsum[(long)b * nch + c];
    chunk_sh[nch + c] = psum[(long)b * nch + c];
  }
  __syncthreads();
  if (tid == 0) {
    const double *W = chunk_sh;
    double Z = 0.0;
    for (int c = 0; c < nch; ++c) Z += W[c];
    int use_p = 0;
    if (!(Z > 0.0)) {          // no residual mass: draw from p
      use_p = 1;
      W = chunk_sh + nch;
      Z = 0.0;
      for (int c = 0; c < nch; ++c) Z += W[c];
    }
    const double t = s.u * Z;
    double run = 0.0;
    int cs = -1;
    for (int c = 0; c < nch; ++c) {
      if (run + W[c] > t) { cs = c; break; }
      run += W[c];
    }
    if (cs < 0) {              // rounding put u * Z past the end: last chunk with mass
      run = 0.0;
      for (int c = 0; c < nch; ++c)
        if (W[c] > 0.0) cs = c;
      if (cs < 0) cs = 0;
      for (int c = 0; c < cs; ++c) run += W[c];
    }
    sh_t = t;
    sh_base = run;
    sh_chunk = cs;
    sh_use_p = use_p;
    sh_thread = kScanThreads;
    sh_last = -1;
  }
  __syncthreads();
  const int cs = sh_chunk;
  const bool use_p = sh_use_p != 0;
  const double isp = 1.0 / s.sp, isq = 1.0 / s.sq;
  const int x0 = cs * kScanChunk + tid * kScanPer;
  double wv[kScanPer], pdummy;
  run_weights<NUC>(s, x0, V, inv_t, use_p, isp, isq, wv, pdummy);
  double w = 0.0;
#pragma unroll
  for (int j = 0; j < kScanPer; ++j) w += wv[j];
  const double incl = block_incl_scan(w, st);
  // the running sum before this thread's run: the previous thread's inclusive sum
  double excl = __shfl_up(incl, 1, kWave);
  if ((tid & 63) == 0) {   // the waves before this one, summed as the scan sums them
    excl = 0.0;
    for (int q = 0; q < (tid >> 6); ++q) excl += st[q];
  }
  if (sh_base + incl > sh_t) atomicMin(&sh_thread, tid);   // first run whose sum passes u * Z
  if (w > 0.0) atomicMax(&sh_last, tid);                  // last run with mass (rounding fallback)
  __syncthreads();
  const bool found = sh_thread < kScanThreads;
  const int th = found ? sh_thread : (sh_last >= 0 ? sh_last : 0);
  if (tid == th) {
    double acc = sh_base + excl;
    int x_last = -1, x_hit = -1;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const int x = x0 + j;
      if (x < V) {
        if (wv[j] > 0.0) x_last = x;
        acc += wv[j];
        if (found && x_hit < 0 && acc > sh_t) x_hit = x;
      }
    }
    *s.dst = x_hit >= 0 ? x_hit : (x_last >= 0 ? x_last : (x0 < V ? x0 : V - 1));
  }
}

void launch_residual_draw(const char *chunk_name, const char *scan_name, int B, int V, float inv_t, const RowSel *sel,
                          double *wsum, double *psum, bool nucleus, hipStream_t s) {
  const int nch = scan_chunks(V);
  {
    TraceScope ts(chunk_name, s);
    if (nucleus)
      hipLaunchKernelGGL(residual_chunk_kernel<true>, dim3(B, nch), dim3(kScanThreads), 0, s, V, inv_t, sel, nch,
                         wsum, psum);
    else
      hipLaunchKernelGGL(residual_chunk_kernel<false>, dim3(B, nch), dim3(kScanThreads), 0, s, V, inv_t, sel, nch,
                         wsum, psum);
  }
  {
    TraceScope ts(scan_name, s);
    if (nucleus)
      hipLaunchKernelGGL(residual_scan_kernel<true>, dim3(B), dim3(kScanThreads), 2 * nch * sizeof(double), s, V,
                         inv_t, sel, nch, wsum, psum);
    else
      hipLaunchKernelGGL(residual_scan_kernel<false>, dim3(B), dim3(kScanThreads), 2 * nch * sizeof(double), s, V,
                         inv_t, sel, nch, wsum, psum);
  }
}

// ------------------------------------------------------------------ KV commit / rollback
__global__ void kv_commit_kernel(int B, int k, int page_size, int max_pages,
                                 const int32_t *__restrict__ block_table, int32_t *__restrict__ seq_lens,
                                 const int32_t *__restrict__ n_accept, int32_t *__restrict__ slots) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int m = seq_lens[b];
  int n = n_accept[b];
  n = n < 0 ? 0 : (n > k ? k : n);
  if (slots) {
    for (int i = 0; i <= k; ++i) {
      int v = -1;
      if (i <= n) {
        const int t = m + i;
        const int pi = t / page_size;
        v = pi < max_pages ? block_table[(long)b * max_pages + pi] * page_size + t % page_size : -1;
      }
      slots[b * (k + 1) + i] = v;
    }
  }
  seq_lens[b] = m + n + 1;
}

void launch_kv_commit(int B, int k, int page_size, int max_pages, const int32_t *block_table,
                      int32_t *seq_lens, const int32_t *n_accept, int32_t *slots, hipStream_t s) {
  TraceScope ts("kv_commit", s);
  hipLaunchKernelGGL(kv_commit_kernel, dim3((B + 63) / 64), dim3(64), 0, s, B, k, page_size, max_pages,
                     block_table, seq_lens, n_accept, slots);
}

}  // namespace gm

// ------------------------------------------------------------------ tile statistics and tile draws
namespace gm {

// one wave per tile (at most 128 ids, two per lane): max of z / T, the lowest id
// attaining it, sum exp(z / T - max) (float32 terms, float64 sum)
static_assert(kMaxTileStrips * kStripIds <= 2 * kWave, "a tile is at most two ids per lane");
__global__ __launch_bounds__(256) void tile_stats_kernel(const float *__restrict__ logits, long row_stride, int V,
                                                         float inv_t, TileGeom geo, RowStat *__restrict__ out) {
  const int r = blockIdx.x, t = blockIdx.y * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (t >= geo.tiles) return;
  const float *row = logits + (long)r * row_stride;
  const int lo = tile_first_strip(geo, t) * kStripIds, hi = min(V, tile_first_strip(geo, t + 1) * kStripIds);
  const int x0 = lo + lane, x1 = x0 + 64;
  const float v0 = x0 < hi ? row[x0] * inv_t : -INFINITY, v1 = x1 < hi ? row[x1] * inv_t : -INFINITY;
  float m = v0;
  int a = x0 < hi ? x0 : 0x7fffffff;
  if (v1 > m) { m = v1; a = x1; }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, kWave);
    const int oa = __shfl_xor(a, o, kWave);
    if (om > m || (om == m && oa < a)) { m = om; a = oa; }
  }
  double s = (x0 < hi ? (double)expf(v0 - m) : 0.0) + (x1 < hi ? (double)expf(v1 - m) : 0.0);
  s = wave_sum(s);
  if (lane == 0) {
    RowStat o;
    o.max = m;
    o.argmax = a;
    o.sum = s;
    out[(long)r * geo.tiles + t] = o;
  }
}

void launch_tile_stats(const float *logits, long row_stride, int n_rows, int V, float inv_t, TileGeom geo,
                       RowStat *tiles, hipStream_t s) {
  if (n_rows <= 0) return;
  TraceScope ts("draft_tile_stats", s);
  hipLaunchKernelGGL(tile_stats_kernel, dim3(n_rows, (geo.tiles + 3) / 4), dim3(256), 0, s, logits, row_stride, V,
                     inv_t, geo, tiles);
}

// One block per row.  The row's max and arg-max come from its tile statistics
// (staged in LDS, all loads in flight at once); a sampled draw takes the tile
// masses s_t exp(m_t - M) in float64, contiguous runs of them per thread, a
// block-wide prefix sum over the runs, and the first run whose prefix passes
// u * S is walked tile by tile to the tile holding u * S.  One wave then scans
// that tile's ids (at most kMaxDrawTileIds, kDrawRun consecutive ids per lane; the
// same per-id terms exp(z / T - m_t) the tile sums were made of, scaled in float64)
// for the first running sum above u * S.
// The draw of row b by one block of 256 threads; the drawn id goes to dst[b * dst_stride]
// and to *tok_sh.  Waves other than the first may leave before the last phase.
__device__ __forceinline__ void tile_draw_row(int V, int mode, float inv_t, const float *__restrict__ logits,
                                              long row_stride, const RowStat *__restrict__ tiles, TileGeom geo,
                                              const float *__restrict__ u, int u_stride, int32_t *__restrict__ dst,
                                              int dst_stride, RowStat *__restrict__ row_out, int row_stride_out,
                                              RowStat *st, int *tok_sh) {
  const int n_tiles = geo.tiles;
  uint4 *st_raw = reinterpret_cast<uint4 *>(st);
  __shared__ float red_m[4];
  __shared__ int red_a[4];
  __shared__ double wsum[4];
  __shared__ double sh_base, sh_t;
  __shared__ int sh_tile, sh_hit, sh_last;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  auto put = [&](int x) {
    dst[(long)b * dst_stride] = x;
    *tok_sh = x;
  };
  const uint4 *src = reinterpret_cast<const uint4 *>(tiles + (long)b * n_tiles);
  float m = -INFINITY;
  int a = 0x7fffffff;
  for (int t0 = tid; t0 < n_tiles; t0 += 256 * 8) {
    uint4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int t = t0 + 256 * q;
      v[q] = t < n_tiles ? src[t] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int t = t0 + 256 * q;
      if (t < n_tiles) {
        st_raw[t] = v[q];
        const float tm = __uint_as_float(v[q].x);
        const int ta = (int)v[q].y;
        if (tm > m || (tm == m && ta < a)) { m = tm; a = ta; }
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, kWave);
    const int oa = __shfl_xor(a, o, kWave);
    if (om > m || (om == m && oa < a)) { m = om; a = oa; }
  }
  if (lane == 0) { red_m[wid] = m; red_a[wid] = a; }
  if (tid == 0) { sh_hit = 256; sh_last = -1; }
  __syncthreads();
  m = red_m[0];
  a = red_a[0];
  for (int w = 1; w < 4; ++w)
    if (red_m[w] > m || (red_m[w] == m && red_a[w] < a)) { m = red_m[w]; a = red_a[w]; }
  if (mode == GM_GREEDY && !row_out) {
    if (tid == 0) put(a);
    return;
  }
  const double M = (double)m;
  const int per = (n_tiles + 255) / 256, t0 = tid * per, t1 = min(n_tiles, t0 + per);
  double w = 0.0;
  for (int t = t0; t < t1; ++t) w += st[t].sum * exp((double)st[t].max - M);
  const double incl = block_incl_scan(w, wsum);
  const double S = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  if (row_out && tid == 0) {   // the row's statistics, for the accept of this draft
    RowStat o;
    o.max = m;
    o.argmax = a;
    o.sum = S;
    row_out[(long)b * row_stride_out] = o;
  }
  if (mode == GM_GREEDY) {
    if (tid == 0) put(a);
    return;
  }
  const double target = (double)u[(long)b * u_stride] * S;
  if (incl > target) atomicMin(&sh_hit, tid);   // first run whose prefix passes u * S
  if (w > 0.0) atomicMax(&sh_last, tid);       // last run with mass (rounding fallback)
  __syncthreads();
  const int hit = sh_hit, th = hit < 256 ? hit : (sh_last >= 0 ? sh_last : 255);
  if (tid == th) {
    double acc = incl - w;
    int tile = -1;
    for (int t = t0; t < t1; ++t) {
      const double W = st[t].sum * exp((double)st[t].max - M);
      if (hit < 256 && acc + W > target) { tile = t; break; }
      if (hit >= 256 && t == t1 - 1) { tile = t; break; }   // past the end: last tile of the last run
      acc += W;
    }
    if (tile < 0) { tile = t1 > t0 ? t1 - 1 : n_tiles - 1; }   // rounding inside the run: its last tile
    sh_tile = tile;
    sh_base = acc;
    sh_t = target;
  }
  __syncthreads();
  if (wid != 0) return;
  const int tile = sh_tile;
  const float mt = st[tile].max;
  const double scale = exp((double)mt - M);
  const float *row = logits + (long)b * row_stride;
  const int lo = tile_first_strip(geo, tile) * kStripIds, hi = min(V, tile_first_strip(geo, tile + 1) * kStripIds);
  const int x0 = lo + kDrawRun * lane;   // kDrawRun consecutive ids per lane
  double e[kDrawRun], run = 0.0;
#pragma unroll
  for (int q = 0; q < kDrawRun; ++q) {
    e[q] = x0 + q < hi ? (double)expf(row[x0 + q] * inv_t - mt) * scale : 0.0;
    run += e[q];
  }
  double incl2 = run;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double n = __shfl_up(incl2, o, kWave);
    if (lane >= o) incl2 += n;
  }
  double excl = __shfl_up(incl2, 1, kWave);
  if (lane == 0) excl = 0.0;
  // running sum after each of this lane's ids; the first id whose sum passes u * S
  double c = sh_base + excl;
  int pick = -1, lastq = -1;
#pragma unroll
  for (int q = 0; q < kDrawRun; ++q) {
    c += e[q];
    if (pick < 0 && c > sh_t) pick = q;
    if (e[q] > 0.0) lastq = q;
  }
  const unsigned long long hitm = __ballot(pick >= 0);
  const unsigned long long nz = __ballot(lastq >= 0);
  // running sums grow along lanes: the first hit lane holds the drawn id
  const int first = hitm ? __ffsll((long long)hitm) - 1 : -1;
  const int lastnz = nz ? 63 - __clzll((long long)nz) : -1;
  if (first >= 0 && lane == first) put(x0 + pick);
  if (first < 0 && lastnz >= 0 && lane == lastnz) put(x0 + lastq);
  if (first < 0 && lastnz < 0 && lane == 0) put(a);
}

// Optional second half of the draw launch: the next chain step's MTP input row
// (mtp_input_row) from the id just drawn and the layer output h, in place of a
// separate input launch.  out == nullptr: draw only.
template <typename T>
struct DrawInput {
  int H, VT;
  float eps;
  const float *h;
  const T *E, *nh, *ne;
  T *out;
  int32_t *dev_err;
};

template <typename T>
__global__ __launch_bounds__(256) void tile_draw_kernel(int V, int mode, float inv_t, const float *__restrict__ logits,
                                                        long row_stride, const RowStat *__restrict__ tiles,
                                                        TileGeom geo, const float *__restrict__ u, int u_stride,
                                                        int32_t *__restrict__ dst, int dst_stride,
                                                        RowStat *__restrict__ row_out, int row_stride_out,
                                                        DrawInput<T> in) {
  extern __shared__ uint4 st_raw[];   // [n_tiles] RowStat
  __shared__ int tok_sh;
  __shared__ float2 red[16];
  tile_draw_row(V, mode, inv_t, logits, row_stride, tiles, geo, u, u_stride, dst, dst_stride, row_out,
                row_stride_out, reinterpret_cast<RowStat *>(st_raw), &tok_sh);
  if (in.out == nullptr) return;
  __syncthreads();
  const int b = blockIdx.x;
  mtp_input_row<T>(in.VT, in.H, V, in.eps, in.h + (long)b * in.H, tok_sh, in.E, in.nh, in.ne,
                   in.out + (long)b * 2 * in.H, in.dev_err, red);
}

void launch_tile_draw(int B, int V, int mode, float inv_t, const float *logits, long row_stride, TileGeom geo,
                      const RowStat *tiles, const float *u, int u_stride, int32_t *dst, int dst_stride,
                      RowStat *row_out, int row_stride_out, hipStream_t s, const DrawNextInput *next) {
  if (B <= 0) return;
  TraceScope ts("draft_draw", s);
  const size_t lds = (size_t)geo.tiles * sizeof(RowStat);
  if (next && next->dtype == GM_BF16) {
    const DrawInput<bf16> in{next->H,       mtp_input_threads(next->H), next->eps, next->h,
                             (const bf16 *)next->E, (const bf16 *)next->norm_h, (const bf16 *)next->norm_e,
                             (bf16 *)next->out, next->dev_err};
    hipLaunchKernelGGL(tile_draw_kernel<bf16>, dim3(B), dim3(256), lds, s, V, mode, inv_t, logits, row_stride, tiles,
                       geo, u, u_stride, dst, dst_stride, row_out, row_stride_out, in);
  } else if (next) {
    const DrawInput<float> in{next->H,       mtp_input_threads(next->H), next->eps, next->h,
                              (const float *)next->E, (const float *)next->norm_h, (const float *)next->norm_e,
                              (float *)next->out, next->dev_err};
    hipLaunchKernelGGL(tile_draw_kernel<float>, dim3(B), dim3(256), lds, s, V, mode, inv_t, logits, row_stride,
                       tiles, geo, u, u_stride, dst, dst_stride, row_out, row_stride_out, in);
  } else {
    const DrawInput<float> none{};
    hipLaunchKernelGGL(tile_draw_kernel<float>, dim3(B), dim3(256), lds, s, V, mode, inv_t, logits, row_stride,
                       tiles, geo, u, u_stride, dst, dst_stride, row_out, row_stride_out, none);
  }
}

}  // namespace gm
