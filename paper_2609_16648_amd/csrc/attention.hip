// Verify attention (Sec. 3.1, Eq. verification-context): the query at block
// position i of sequence b attends causally to cache positions 0 .. m_b + i.
//
// bf16 path, one 64-lane wave per (context split, KV head, sequence):
//  * GQA packing: the (n_heads / n_kv_heads) query heads of one KV head times
//    the block rows form the rows of 16-row matrix-core tiles, so each K/V
//    byte streamed from HBM serves every query that reads it;
//  * S^T = K Q^T on v_mfma_f32_16x16x32_bf16 and O^T += V^T P^T on
//    v_mfma_f32_16x16x16_bf16: the score tile comes out of the first product
//    already in the operand layout of the second, so P never leaves registers;
//  * the KV pages are stored pre-swizzled (gm.h), so every 16-byte-per-lane
//    load reads 1 KiB contiguous straight into operand registers: no LDS
//    staging, no shuffles;
//  * P is split into bf16 hi + lo parts (two products) so the weights keep
//    ~16 mantissa bits; scores, the online softmax (exp2 domain) and O stay
//    float32;
//  * each split writes (m, l, O) partials; a combine kernel merges the splits.
// float32 path: a plain wave-per-(row, head) kernel.
#include "common.h"
#include "forward.h"

namespace gm {

namespace {
struct AttnK {
  const uint16_t *kp, *vp;
  const int32_t *bt, *base, *blen;
  const uint16_t *q;
  float *part_o;
  float2 *part_ml;
  int32_t *dev_err;
  int base_off, blen_add, R, G, n_heads, n_kv, page_size, max_pages, num_pages, split_tokens, splits, rows_pad;
  float scale_log2;
};

__device__ __forceinline__ int block_rows(const int32_t *blen, int add, int b, int R) {
  if (!blen) return R;
  const int n = blen[b] + add;
  return n < 0 ? 0 : (n > R ? R : n);
}

__device__ __forceinline__ uint32_t zero_half(uint32_t v, int hi) { return hi ? (v & 0x0000ffffu) : (v & 0xffff0000u); }

// One 16-token tile: S^T = K Q^T, online softmax (exp2 domain, rescale only when
// a row's running max grows), O^T += V^T (P_hi + P_lo).
template <int NT, bool TAIL>
__device__ __forceinline__ void attn_tile(int tb, int L, int g, float scale_log2, uint4 (&kc)[4], uint4 (&vc)[4],
                                          const bf16x8_t (&qf)[NT][4], const int (&vis)[NT], float (&mrow)[NT],
                                          float (&lsum)[NT], floatx4_t (&O)[NT][8]) {
  if (TAIL) {  // tail tile: entries past the context may hold anything, keep them out of P.V
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (tb + 4 * g + e >= L) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          if (e < 2) { vc[p].x = zero_half(vc[p].x, e); vc[p].z = zero_half(vc[p].z, e); }
          else { vc[p].y = zero_half(vc[p].y, e - 2); vc[p].w = zero_half(vc[p].w, e - 2); }
        }
      }
    }
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    floatx4_t S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) S = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kc[ii]), qf[nt][ii], S, 0, 0, 0);
    float s[4], tmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tok = tb + 4 * g + r;
      s[r] = tok < vis[nt] ? S[r] * scale_log2 : -INFINITY;
      tmax = fmaxf(tmax, s[r]);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float mnew = fmaxf(mrow[nt], tmax);
    const bool grow = mnew > mrow[nt];
    if (__any(grow)) {
      const float alpha = grow ? exp2f(mrow[nt] - mnew) : 1.f;
      lsum[nt] *= alpha;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) O[nt][mm] *= alpha;
    }
    mrow[nt] = mnew;
    const bool none = mnew == -INFINITY;
    uint16_t hi[4], lo[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float p = none ? 0.f : exp2f(s[r] - mnew);
      lsum[nt] += p;
      hi[r] = f32_to_bf16(p);
      lo[r] = f32_to_bf16(p - bf16_to_f32(hi[r]));
    }
    const uint2 phi = make_uint2(hi[0] | (uint32_t(hi[1]) << 16), hi[2] | (uint32_t(hi[3]) << 16));
    const uint2 plo = make_uint2(lo[0] | (uint32_t(lo[1]) << 16), lo[2] | (uint32_t(lo[3]) << 16));
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) {
      const uint4 &v4 = vc[mm >> 1];
      const uint2 vv = (mm & 1) ? make_uint2(v4.z, v4.w) : make_uint2(v4.x, v4.y);
      O[nt][mm] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(as_bf16x4(vv), as_bf16x4(phi), O[nt][mm], 0, 0, 0);
      O[nt][mm] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(as_bf16x4(vv), as_bf16x4(plo), O[nt][mm], 0, 0, 0);
    }
  }
}

template <int NT>
__global__ __launch_bounds__(64) void attn_mfma_kernel(AttnK a) {
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x, j = lane & 15, g = lane >> 4;
  const int m0 = a.base[b] + a.base_off;
  const int blen = block_rows(a.blen, a.blen_add, b, a.R);
  const int L = m0 + blen;
  const int t0 = split * a.split_tokens;
  if (t0 >= L) return;
  const int t1 = min(L, t0 + a.split_tokens);
  const int rows = a.G * a.R;

  bf16x8_t qf[NT][4];
  int vis[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = nt * 16 + j;
    if (r < rows) {
      const int hl = r / a.R, i = r % a.R;
      const uint16_t *qrow = a.q + (((long)b * a.R + i) * a.n_heads + kvh * a.G + hl) * 128;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) qf[nt][ii] = as_bf16x8(*reinterpret_cast<const uint4 *>(qrow + 32 * ii + 8 * g));
      vis[nt] = i < blen ? m0 + i + 1 : 0;
    } else {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) qf[nt][ii] = as_bf16x8(make_uint4(0, 0, 0, 0));
      vis[nt] = 0;
    }
  }

  float mrow[NT], lsum[NT];
  floatx4_t O[NT][8];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    mrow[nt] = -INFINITY;
    lsum[nt] = 0.f;
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) O[nt][mm] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }

  // The pages this split touches, looked up once into LDS: in the loop a lookup is then an
  // LDS read, whose counter is separate from the KV loads', so no wait drains the prefetch.
  // A page outside the pool ends the split before its first token (and is reported).
  __shared__ int page_sh[kAttnMaxSplitPages];
  __shared__ int bad_sh;
  const int p0 = t0 / a.page_size, np = (t1 - 1) / a.page_size - p0 + 1;
  if (lane == 0) bad_sh = np;
  __syncthreads();
  for (int i = lane; i < np; i += kWave) {
    const int pi = p0 + i;
    const int page = pi < a.max_pages ? a.bt[(long)b * a.max_pages + pi] : -1;
    page_sh[i] = page;
    if (page < 0 || page >= a.num_pages) atomicMin(&bad_sh, i);
  }
  __syncthreads();
  int tend = t1;
  if (bad_sh < np) {
    raise_dev_err(a.dev_err, GM_DEVERR_PAGE);
    tend = max(t0, (p0 + bad_sh) * a.page_size);
  }
  const long head_off = (long)kvh * a.page_size * 128;
  auto tile_off = [&](int tb) -> long {
    const int page = page_sh[tb / a.page_size - p0];
    return (long)page * a.n_kv * a.page_size * 128 + head_off + (long)(tb % a.page_size) * 128;
  };
  auto load_tile = [&](long off, uint4 (&kf)[4], uint4 (&vf)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) kf[i] = *reinterpret_cast<const uint4 *>(a.kp + off + i * 512 + lane * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) vf[i] = *reinterpret_cast<const uint4 *>(a.vp + off + i * 512 + lane * 8);
  };
  // full tiles: two register buffers, alternating, every load unconditional (the last
  // prefetch re-reads a valid tile), so the loads of the next tile are always in flight
  // while the current one is consumed and no register copy waits on them
  const int full_end = min(tend, (L / 16) * 16);
  const int n_full = full_end > t0 ? (full_end - t0) / 16 : 0;
  uint4 ka[4], va[4], kb[4], vb[4];
  if (n_full > 0) {
    load_tile(tile_off(t0), ka, va);
    for (int i = 0; i < n_full; i += 2) {
      load_tile(tile_off(t0 + 16 * min(i + 1, n_full - 1)), kb, vb);
      attn_tile<NT, false>(t0 + 16 * i, L, g, a.scale_log2, ka, va, qf, vis, mrow, lsum, O);
      if (i + 1 >= n_full) break;
      load_tile(tile_off(t0 + 16 * min(i + 2, n_full - 1)), ka, va);
      attn_tile<NT, false>(t0 + 16 * (i + 1), L, g, a.scale_log2, kb, vb, qf, vis, mrow, lsum, O);
    }
  }
  if (full_end < tend) {  // the partial tile at the end of the context
    load_tile(tile_off(full_end), ka, va);
    attn_tile<NT, true>(full_end, L, g, a.scale_log2, ka, va, qf, vis, mrow, lsum, O);
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float l = lsum[nt];
    l += __shfl_xor(l, 16, kWave);
    l += __shfl_xor(l, 32, kWave);
    const long prow = (((long)b * a.n_kv + kvh) * a.splits + split) * a.rows_pad + nt * 16 + j;
    if (g == 0) a.part_ml[prow] = make_float2(mrow[nt], l);
    float *po = a.part_o + prow * 128;
#pragma unroll
    for (int mm = 0; mm < 8; ++mm)
      *reinterpret_cast<float4 *>(po + 16 * mm + 4 * g) = make_float4(O[nt][mm][0], O[nt][mm][1], O[nt][mm][2], O[nt][mm][3]);
  }
}

__global__ __launch_bounds__(256) void attn_combine_kernel(AttnK a, uint16_t *__restrict__ out) {
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int m0 = a.base[b] + a.base_off;
  const int blen = block_rows(a.blen, a.blen_add, b, a.R);
  const int L = m0 + blen;
  int n_act = L > 0 ? (L + a.split_tokens - 1) / a.split_tokens : 0;
  if (n_act > a.splits) n_act = a.splits;
  const int rows = a.G * a.R;
  const long pbase = ((long)b * a.n_kv + kvh) * a.splits * a.rows_pad;
  // 32 threads per row, four channels each
  for (int idx = threadIdx.x; idx < rows * 32; idx += blockDim.x) {
    const int r = idx >> 5, d = (idx & 31) * 4;
    const int hl = r / a.R, i = r % a.R;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < blen) {
      float M = -INFINITY;
      for (int s = 0; s < n_act; ++s) M = fmaxf(M, a.part_ml[pbase + (long)s * a.rows_pad + r].x);
      if (M != -INFINITY) {
        float den = 0.f;
        float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int s = 0; s < n_act; ++s) {
          const long pr = pbase + (long)s * a.rows_pad + r;
          const float2 ml = a.part_ml[pr];
          const float w = exp2f(ml.x - M);
          const float4 o = *reinterpret_cast<const float4 *>(a.part_o + pr * 128 + d);
          den += ml.y * w;
          num.x += o.x * w;
          num.y += o.y * w;
          num.z += o.z * w;
          num.w += o.w * w;
        }
        const float inv = 1.f / den;
        v = make_float4(num.x * inv, num.y * inv, num.z * inv, num.w * inv);
      }
    }
    const uint2 packed = make_uint2(f32_to_bf16(v.x) | (uint32_t(f32_to_bf16(v.y)) << 16),
                                    f32_to_bf16(v.z) | (uint32_t(f32_to_bf16(v.w)) << 16));
    *reinterpret_cast<uint2 *>(out + (((long)b * a.R + i) * a.n_heads + kvh * a.G + hl) * 128 + d) = packed;
  }
}

// ------------------------------------------------------------------ float32 path
struct AttnF {
  const float *kp, *vp, *q;
  float *out;
  const int32_t *bt, *base, *blen;
  int32_t *dev_err;
  int base_off, blen_add, R, G, n_heads, n_kv, page_size, max_pages, num_pages;
  float scale;
};

template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnF a) {
  __shared__ float sm_m[64], sm_l[64];
  __shared__ float sm_acc[64][D + 1];
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z, t = threadIdx.x;
  const int blen = block_rows(a.blen, a.blen_add, b, a.R);
  float *orow = a.out + (((long)b * a.R + i) * a.n_heads + h) * D;
  if (i >= blen) {
    for (int c = t; c < D; c += 64) orow[c] = 0.f;
    return;
  }
  const int vis = a.base[b] + a.base_off + i + 1;
  const int kvh = h / a.G;
  const float *qrow = a.q + (((long)b * a.R + i) * a.n_heads + h) * D;
  float q[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) { q[c] = qrow[c]; acc[c] = 0.f; }
  float mx = -INFINITY, l = 0.f;
  for (int tok = t; tok < vis; tok += 64) {
    const int pi = tok / a.page_size;
    const int page = pi < a.max_pages ? a.bt[(long)b * a.max_pages + pi] : -1;
    if (page < 0 || page >= a.num_pages) {
      raise_dev_err(a.dev_err, GM_DEVERR_PAGE);
      break;
    }
    const int off = tok % a.page_size;
    const long tile = (((long)page * a.n_kv + kvh) * a.page_size + (off & ~15)) * D;
    const int s = off & 15;
    float sc = 0.f;
#pragma unroll
    for (int c = 0; c < D; ++c) sc += q[c] * a.kp[tile + k_tile_off(s, c)];
    sc *= a.scale;
    const float mn = fmaxf(mx, sc);
    const float al = expf(mx - mn), p = expf(sc - mn);
    l = l * al + p;
#pragma unroll
    for (int c = 0; c < D; ++c) acc[c] = acc[c] * al + p * a.vp[tile + v_tile_off(s, c)];
    mx = mn;
  }
  sm_m[t] = mx;
  sm_l[t] = l;
#pragma unroll
  for (int c = 0; c < D; ++c) sm_acc[t][c] = acc[c];
  __syncthreads();
  float M = -INFINITY;
  for (int u = 0; u < 64; ++u) M = fmaxf(M, sm_m[u]);
  float den = 0.f;
  for (int u = 0; u < 64; ++u) den += sm_m[u] == -INFINITY ? 0.f : sm_l[u] * expf(sm_m[u] - M);
  for (int c = t; c < D; c += 64) {
    float num = 0.f;
    for (int u = 0; u < 64; ++u) num += sm_m[u] == -INFINITY ? 0.f : sm_acc[u][c] * expf(sm_m[u] - M);
    orow[c] = num / den;
  }
}
}  // namespace

AttnPlan plan_attention(const gm_model_config &cfg, int B, int R, int max_ctx) {
  AttnPlan p{};
  const int G = cfg.n_heads / cfg.n_kv_heads;
  const int rows = G * R;
  const int nt = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
  p.rows_pad = nt * 16;
  if (cfg.dtype != GM_BF16) return p;
  const long tokens = (long)max_ctx + R;
  const long target_waves = 4096;
  long per = ((long)B * cfg.n_kv_heads * tokens + target_waves - 1) / target_waves;
  per = ((per + 63) / 64) * 64;
  if (per < 64) per = 64;
  if (per > 4096) per = 4096;
  p.split_tokens = (int)per;
  p.splits = (int)((tokens + per - 1) / per);
  Carve c;
  const size_t n = (size_t)B * cfg.n_kv_heads * p.splits * p.rows_pad;
  p.part_o = c.take(n * 128 * sizeof(float));
  p.part_ml = c.take(n * sizeof(float2));
  p.total = c.off;
  return p;
}

AttnArgs attn_args(const gm_model_config &cfg, const gm_kv_cache &c, int layer, int B, int R,
                   const int32_t *base_lens, int base_off, const int32_t *blk_len) {
  AttnArgs a{};
  a.dtype = cfg.dtype;
  a.B = B;
  a.R = R;
  a.n_heads = cfg.n_heads;
  a.n_kv = cfg.n_kv_heads;
  a.head_dim = cfg.head_dim;
  a.page_size = c.page_size;
  a.max_pages = c.max_pages_per_seq;
  a.num_pages = c.num_pages;
  a.k_pages = c.k_pages[layer];
  a.v_pages = c.v_pages[layer];
  a.block_table = c.block_table;
  a.base_lens = base_lens;
  a.base_off = base_off;
  a.blk_len = blk_len;
  a.blk_len_add = 0;
  a.scale = 1.0f / sqrtf((float)cfg.head_dim);
  a.trace = "attn";
  a.trace_combine = "attn_combine";
  return a;
}

void run_attention(const AttnArgs &a, const AttnPlan &p, char *ws, hipStream_t s) {
  if (a.B == 0) return;
  const int G = a.n_heads / a.n_kv;
  if (a.dtype == GM_BF16) {
    AttnK k{};
    k.kp = (const uint16_t *)a.k_pages;
    k.vp = (const uint16_t *)a.v_pages;
    k.bt = a.block_table;
    k.base = a.base_lens;
    k.blen = a.blk_len;
    k.q = (const uint16_t *)a.q;
    k.part_o = (float *)(ws + p.part_o);
    k.part_ml = (float2 *)(ws + p.part_ml);
    k.dev_err = a.dev_err;
    k.base_off = a.base_off;
    k.blen_add = a.blk_len_add;
    k.R = a.R;
    k.G = G;
    k.n_heads = a.n_heads;
    k.n_kv = a.n_kv;
    k.page_size = a.page_size;
    k.max_pages = a.max_pages;
    k.num_pages = a.num_pages;
    k.split_tokens = p.split_tokens;
    k.splits = p.splits;
    k.rows_pad = p.rows_pad;
    k.scale_log2 = a.scale * 1.4426950408889634f;
    dim3 grid(p.splits, a.n_kv, a.B);
    {
      TraceScope ts(a.trace, s);
      if (p.rows_pad == 16) hipLaunchKernelGGL(attn_mfma_kernel<1>, grid, dim3(64), 0, s, k);
      else if (p.rows_pad == 32) hipLaunchKernelGGL(attn_mfma_kernel<2>, grid, dim3(64), 0, s, k);
      else hipLaunchKernelGGL(attn_mfma_kernel<4>, grid, dim3(64), 0, s, k);
    }
    TraceScope ts(a.trace_combine, s);
    hipLaunchKernelGGL(attn_combine_kernel, dim3(a.n_kv, a.B), dim3(256), 0, s, k, (uint16_t *)a.out);
  } else {
    AttnF f{};
    f.kp = (const float *)a.k_pages;
    f.vp = (const float *)a.v_pages;
    f.q = (const float *)a.q;
    f.out = (float *)a.out;
    f.bt = a.block_table;
    f.base = a.base_lens;
    f.blen = a.blk_len;
    f.dev_err = a.dev_err;
    f.base_off = a.base_off;
    f.blen_add = a.blk_len_add;
    f.R = a.R;
    f.G = G;
    f.n_heads = a.n_heads;
    f.n_kv = a.n_kv;
    f.page_size = a.page_size;
    f.max_pages = a.max_pages;
    f.num_pages = a.num_pages;
    f.scale = a.scale;
    dim3 grid(a.R, a.n_heads, a.B);
    TraceScope ts(a.trace, s);
    if (a.head_dim == 64) hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, f);
    else hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, f);
  }
}

}  // namespace gm
