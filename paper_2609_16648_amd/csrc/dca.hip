// Depth-coupled acceptance loss with verify-gated masking, and its gradient in
// the head logits (Sec. "The Depth-Coupled Acceptance Loss", "Learning up to
// the First Rejection"; App. "DCA", Eqs. alpha, chain, dca, vgm, dca-partial,
// dca-tail, dca-coeff), over the cycle record's sparse support: the head
// distribution q = softmax(z) is normalised over the whole vocabulary and
// gathered at the record's ids S, and the mass outside S forms one residual
// bin (App. "Implementing Draft-Path Reconstruction in verl").
//
//  1. The row-statistics pass over the head logits (max and sum exp per chunk).
//  2. One block per cycle, one wave per draft position: q and p on S (float64),
//     alpha_k, the subgradient flags [q < p] of min, then the chain (one
//     thread): M = sum_{l<=L} prod_{i<=l} alpha_i, the loss -log M, and the
//     coefficient of position k, -(prod_{i<k} alpha_i) D_k / M (0 past L).
//  3. The gradient pass, one block per (row, 4096 ids): coef * q_x * (g_x - gbar)
//     with g_x the residual bin's flag; the block then rewrites the ids of S
//     that fall in its range with their own flags.
#include "common.h"
#include "forward.h"

namespace gm {

namespace {
struct DcaRow {          // per (cycle, position): what the gradient pass needs
  double coef, gbar, M, inv_s;
  int g_rest, pad;
};
constexpr int kDcaIds = 4096;   // ids per block of the gradient pass

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__global__ __launch_bounds__(1024) void dca_cycle_kernel(int K, int V, int topk, int vgm,
                                                         const float *__restrict__ z,
                                                         const RowStat *__restrict__ stats, int nch,
                                                         const uint16_t *__restrict__ rec_logp,
                                                         const int32_t *__restrict__ rec_ids,
                                                         const int32_t *__restrict__ n_accept,
                                                         float *__restrict__ loss, float *__restrict__ alpha_out,
                                                         DcaRow *__restrict__ rows, uint8_t *__restrict__ flags) {
  __shared__ double sh_alpha[16];
  const int n = blockIdx.x, k = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const long r = (long)n * K + k;
  // q's normaliser from the chunk statistics
  double M = 0.0, S = 1.0;
  int am = 0;
  {
    const RowStat *st = stats + r * nch;
    float m = -INFINITY;
    for (int c = 0; c < nch; ++c) m = fmaxf(m, st[c].max);
    double s = 0.0;
    for (int c = 0; c < nch; ++c) s += st[c].sum * exp((double)st[c].max - (double)m);
    M = (double)m;
    S = s;
    (void)am;
  }
  double p = 0.0, q = 0.0;
  if (lane < topk) {
    const int id = rec_ids[r * topk + lane];
    p = exp((double)bf16_to_f32(rec_logp[r * topk + lane]));
    q = (id >= 0 && id < V) ? exp((double)z[r * V + id] - M) / S : 0.0;
  }
  const double sum_p = wave_sum(p), sum_q = wave_sum(q), sum_min = wave_sum(fmin(p, q));
  const double pR = fmax(0.0, 1.0 - sum_p), qR = 1.0 - sum_q;
  const double alpha = sum_min + fmin(pR, qR);
  const int g = q < p, g_rest = qR < pR;
  const double gbar = wave_sum(lane < topk && g ? q : 0.0) + (g_rest ? qR : 0.0);
  if (lane < topk) flags[r * topk + lane] = (uint8_t)g;
  if (lane == 0) {
    sh_alpha[k] = alpha;
    alpha_out[r] = (float)alpha;
    rows[r].gbar = gbar;
    rows[r].M = M;
    rows[r].inv_s = 1.0 / S;
    rows[r].g_rest = g_rest;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int L = K;
    if (vgm) {
      const int na = n_accept[n];
      L = na + 1 < K ? (na + 1 < 1 ? 1 : na + 1) : K;
    }
    double chain = 0.0, pre = 1.0;
    for (int l = 0; l < L; ++l) {
      pre *= sh_alpha[l];
      chain += pre;
    }
    loss[n] = (float)(-log(chain));
    double before = 1.0;
    for (int kk = 0; kk < K; ++kk) {
      double coef = 0.0;
      if (kk < L) {
        double D = 0.0, t = 1.0;   // D_k = sum_{l=k}^{L} prod_{i=k+1}^{l} alpha_i
        for (int l = kk; l < L; ++l) {
          if (l > kk) t *= sh_alpha[l];
          D += t;
        }
        coef = -before * D / chain;
      }
      rows[(long)n * K + kk].coef = coef;
      before *= sh_alpha[kk];
    }
  }
}

__global__ __launch_bounds__(256) void dca_grad_kernel(int V, int topk, const float *__restrict__ z,
                                                       const DcaRow *__restrict__ rows,
                                                       const int32_t *__restrict__ rec_ids,
                                                       const uint8_t *__restrict__ flags, float *__restrict__ grad) {
  const long r = blockIdx.x;
  const int lo = blockIdx.y * kDcaIds, hi = min(V, lo + kDcaIds);
  const DcaRow d = rows[r];
  const float coef = (float)d.coef, M = (float)d.M, inv_s = (float)d.inv_s;
  const float rest = (float)((double)d.g_rest - d.gbar);
  const float *zr = z + r * V;
  float *gr = grad + r * V;
  const bool vec = (V & 3) == 0;
  for (int x = lo + 4 * threadIdx.x; x < hi; x += 4 * blockDim.x) {
    if (vec && x + 3 < hi) {
      const float4 v = *reinterpret_cast<const float4 *>(zr + x);
      float4 o;
      o.x = coef * (expf(v.x - M) * inv_s) * rest;
      o.y = coef * (expf(v.y - M) * inv_s) * rest;
      o.z = coef * (expf(v.z - M) * inv_s) * rest;
      o.w = coef * (expf(v.w - M) * inv_s) * rest;
      *reinterpret_cast<float4 *>(gr + x) = o;
    } else {
      for (int q = 0; q < 4 && x + q < hi; ++q) gr[x + q] = coef * (expf(zr[x + q] - M) * inv_s) * rest;
    }
  }
  __syncthreads();
  // the record's ids in this range carry their own flags
  if ((int)threadIdx.x < topk) {
    const int id = rec_ids[r * topk + threadIdx.x];
    if (id >= lo && id < hi) {
      const float own = (float)((double)flags[r * topk + threadIdx.x] - d.gbar);
      gr[id] = coef * (expf(zr[id] - M) * inv_s) * own;
    }
  }
}
}  // namespace

size_t dca_workspace(int N, int K, int V) {
  Carve c;
  c.take(sizeof(RowStat) * (size_t)N * K * stat_chunks(V));
  c.take(sizeof(DcaRow) * (size_t)N * K);
  c.take((size_t)N * K * kRecMaxTopk);
  return c.off;
}

void run_dca_loss(int N, int K, int V, int topk, const float *head_logits, const uint16_t *rec_logp,
                  const int32_t *rec_ids, const int32_t *n_accept, int vgm, float *loss, float *alpha, float *grad,
                  char *ws, hipStream_t s) {
  Carve c;
  RowStat *stats = (RowStat *)(ws + c.take(sizeof(RowStat) * (size_t)N * K * stat_chunks(V)));
  DcaRow *rows = (DcaRow *)(ws + c.take(sizeof(DcaRow) * (size_t)N * K));
  uint8_t *flags = (uint8_t *)(ws + c.take((size_t)N * K * kRecMaxTopk));
  launch_row_stats("dca_row_stats", head_logits, V, N * K, V, 1.0f, stats, s);
  {
    TraceScope ts("dca_cycle", s);
    hipLaunchKernelGGL(dca_cycle_kernel, dim3(N), dim3(64 * K), 0, s, K, V, topk, vgm, head_logits, stats,
                       stat_chunks(V), rec_logp, rec_ids, n_accept, loss, alpha, rows, flags);
  }
  if (grad) {
    TraceScope ts("dca_grad", s);
    hipLaunchKernelGGL(dca_grad_kernel, dim3(N * K, (V + kDcaIds - 1) / kDcaIds), dim3(256), 0, s, V, topk,
                       head_logits, rows, rec_ids, flags, grad);
  }
}

}  // namespace gm
