// Row-wise kernels of the forward and the draft head: embedding gather,
// RMSNorm, the MTP input (two RMSNorms and the concatenation), RoPE with the
// KV append into the paged cache, and row gathers.
//
// Precision: row statistics in float32; the rotary angle pos * base^(-2i/d)
// and its sine / cosine in float64 (positions reach 32K, where a float32
// angle is off by ~2e-3 rad); outputs rounded once to the model dtype.
#include "common.h"
#include "forward.h"
#include "mtp_row.h"

namespace gm {

namespace {
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(int H, int V, const int32_t *__restrict__ tok,
                                                    const T *__restrict__ E, float *__restrict__ x,
                                                    int32_t *dev_err) {
  const int r = blockIdx.x;
  const int t = tok[r];
  float *xr = x + (long)r * H;
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) raise_dev_err(dev_err, GM_DEVERR_TOKEN);
    for (int c = threadIdx.x; c < H; c += blockDim.x) xr[c] = 0.f;
    return;
  }
  const T *er = E + (long)t * H;
  for (int c = threadIdx.x; c < H; c += blockDim.x) xr[c] = Elem<T>::load(er, c);
}

// the embedding rows (float32 residual stream) and their RMSNorm in one pass
template <typename T>
__global__ __launch_bounds__(256) void embed_norm_kernel(int H, int V, const int32_t *__restrict__ tok,
                                                         const T *__restrict__ E, float *__restrict__ x,
                                                         const T *__restrict__ w, float eps, T *__restrict__ out,
                                                         int32_t *dev_err) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  const int t = tok[r];
  const bool ok = t >= 0 && t < V;
  if (!ok && threadIdx.x == 0) raise_dev_err(dev_err, GM_DEVERR_TOKEN);
  const T *er = E + (long)(ok ? t : 0) * H;
  float *xr = x + (long)r * H;
  float ss = 0.f;
  for (int c = threadIdx.x; c < H; c += blockDim.x) {
    const float v = ok ? Elem<T>::load(er, c) : 0.f;
    xr[c] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)H + eps);
  T *o = out + (long)r * H;
  for (int c = threadIdx.x; c < H; c += blockDim.x) Elem<T>::store(o, c, xr[c] * inv * Elem<T>::load(w, c));
}

// one wave per row, four channels per lane and step (H % 4 == 0)
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(int M, int H, float eps, const float *__restrict__ x,
                                                      const T *__restrict__ w, T *__restrict__ out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= M) return;
  const float *xr = x + (long)r * H;
  float ss = 0.f;
  for (int c = lane * 4; c < H; c += 256) {
    const float4 v = *reinterpret_cast<const float4 *>(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)H + eps);
  T *o = out + (long)r * H;
  for (int c = lane * 4; c < H; c += 256) {
    const float4 v = *reinterpret_cast<const float4 *>(xr + c);
    Elem<T>::store(o, c, v.x * inv * Elem<T>::load(w, c));
    Elem<T>::store(o, c + 1, v.y * inv * Elem<T>::load(w, c + 1));
    Elem<T>::store(o, c + 2, v.z * inv * Elem<T>::load(w, c + 2));
    Elem<T>::store(o, c + 3, v.w * inv * Elem<T>::load(w, c + 3));
  }
}

// MTP input row r (mtp_input_row): one block of mtp_input_threads(H) threads per row
template <typename T>
__global__ __launch_bounds__(1024) void mtp_input_kernel(int H, int V, float eps, const float *__restrict__ h,
                                                         const int32_t *__restrict__ tok, int tok_stride,
                                                         const T *__restrict__ E, const T *__restrict__ nh,
                                                         const T *__restrict__ ne, T *__restrict__ out,
                                                         int32_t *dev_err) {
  __shared__ float2 red[16];
  const int r = blockIdx.x;
  mtp_input_row<T>(blockDim.x, H, V, eps, h + (long)r * H, tok[(long)r * tok_stride], E, nh, ne, out + (long)r * 2 * H,
                   dev_err, red);
}

// One wave per (row, kRopeHeads consecutive heads): block (row, y) holds 4 such
// groups, and lane c < d/2 handles the pair (c, c + d/2) of every head of its group.
// The wave reads its heads' columns straight from the projection (or sums their
// K-split partials, in split order), all heads' loads in flight together, and
// takes the rotation of its lane's pair once for the whole group.
constexpr int kRopeHeads = 4;
template <typename T>
__global__ __launch_bounds__(256) void rope_append_kernel(RopeArgs a) {
  const int row = blockIdx.x, b = row / a.R, i = row % a.R;
  const int lane = threadIdx.x & 63;
  const int D = a.head_dim, half = D / 2;
  const int nh = a.n_heads + 2 * a.n_kv;
  const int h0 = (blockIdx.y * 4 + (threadIdx.x >> 6)) * kRopeHeads;
  if (h0 >= nh) return;
  int blen = a.R;
  if (a.blk_len) {
    blen = a.blk_len[b] + a.blk_len_add;
    blen = blen < 0 ? 0 : (blen > a.R ? a.R : blen);
  }
  const int slot = a.base_lens[b] + a.base_off + i;
  const double pos = (double)(slot + a.pos_off);
  const bool act = lane < half;
  // the pairs' two columns of every head of the group
  float x1[kRopeHeads], x2[kRopeHeads];
  const long W = (long)nh * D;
#pragma unroll
  for (int h = 0; h < kRopeHeads; ++h) {
    x1[h] = 0.f;
    x2[h] = 0.f;
    if (!act || h0 + h >= nh) continue;
    const long off = (long)row * W + (long)(h0 + h) * D + lane;
    if (a.splits > 1) {
      const long stride = (long)a.M * W;
      for (int s0 = 0; s0 < a.splits; s0 += 8) {
        float v1[8], v2[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const long sp = s0 + u < a.splits ? s0 + u : a.splits - 1;
          v1[u] = a.part[sp * stride + off];
          v2[u] = a.part[sp * stride + off + half];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (s0 + u < a.splits) {
            x1[h] += v1[u];
            x2[h] += v2[u];
          }
        }
      }
    } else {
      x1[h] = a.qkv[off];
      x2[h] = a.qkv[off + half];
    }
  }
  // the rotation of pair `lane` at this position, shared by the group's heads
  double sn = 0.0, cs = 1.0;
  if (act && h0 < a.n_heads + a.n_kv) sincos(pos * exp2(-2.0 * lane / D * log2((double)a.rope_base)), &sn, &cs);
  const T *qn = (const T *)a.q_norm, *kn = (const T *)a.k_norm;
  // the block row's page, for the K/V heads of the group
  long kv_base = -1;
  int s_in = 0;
  if (i < blen && h0 + kRopeHeads > a.n_heads) {
    const int pi = slot / a.page_size;
    const int page = pi < a.max_pages ? a.block_table[(long)b * a.max_pages + pi] : -1;
    if (page < 0 || page >= a.num_pages) {
      if (lane == 0) raise_dev_err(a.dev_err, GM_DEVERR_PAGE);
    } else {
      const int off = slot % a.page_size;
      kv_base = (((long)page * a.n_kv) * a.page_size + (off & ~15)) * D;
      s_in = off & 15;
    }
  }
#pragma unroll
  for (int h = 0; h < kRopeHeads; ++h) {
    const int hh = h0 + h;
    if (hh >= nh) break;
    const int kind = hh < a.n_heads ? 0 : (hh < a.n_heads + a.n_kv ? 1 : 2);
    float y1 = x1[h], y2 = x2[h];
    if (kind < 2 && qn) {
      const T *nw = kind == 0 ? qn : kn;
      const float ss = wave_sum(y1 * y1 + y2 * y2);
      const float inv = 1.0f / sqrtf(ss / (float)D + a.eps);
      if (act) {
        y1 = y1 * inv * Elem<T>::load(nw, lane);
        y2 = y2 * inv * Elem<T>::load(nw, lane + half);
      }
    }
    if (!act) continue;
    if (kind < 2) {
      const float r1 = (float)((double)y1 * cs - (double)y2 * sn);
      const float r2 = (float)((double)y2 * cs + (double)y1 * sn);
      y1 = r1;
      y2 = r2;
    }
    if (kind == 0) {
      T *q = (T *)a.q_out + ((long)row * a.n_heads + hh) * D;
      Elem<T>::store(q, lane, y1);
      Elem<T>::store(q, lane + half, y2);
    } else if (kv_base >= 0) {   // rows past the block's valid length append nothing
      const int head = kind == 1 ? hh - a.n_heads : hh - a.n_heads - a.n_kv;
      const long base = kv_base + (long)head * a.page_size * D;
      if (kind == 1) {
        T *kp = (T *)a.k_pages + base;
        Elem<T>::store(kp, k_tile_off(s_in, lane), y1);
        Elem<T>::store(kp, k_tile_off(s_in, lane + half), y2);
      } else {
        T *vp = (T *)a.v_pages + base;
        Elem<T>::store(vp, v_tile_off(s_in, lane), y1);
        Elem<T>::store(vp, v_tile_off(s_in, lane + half), y2);
      }
    }
  }
}

// The draft head's extend tail, one workgroup per sequence: row n_b (clamped to 0..R-1) of
// each of two row sets gathered into one row, and the head's committed length moved to
// the new boundary m_b + n_b + 1 (the length update of a commit, without a slot list).
__global__ __launch_bounds__(256) void gather_commit_kernel(int R, int C16a, const uint4 *__restrict__ src_a,
                                                            uint4 *__restrict__ dst_a, int C16b,
                                                            const uint4 *__restrict__ src_b, uint4 *__restrict__ dst_b,
                                                            const int32_t *__restrict__ sel, int32_t *__restrict__ lens) {
  const int b = blockIdx.x;
  int i = sel[b];
  i = i < 0 ? 0 : (i >= R ? R - 1 : i);
  const uint4 *sa = src_a + ((long)b * R + i) * C16a;
  const uint4 *sb = src_b + ((long)b * R + i) * C16b;
  uint4 *da = dst_a + (long)b * C16a, *db = dst_b + (long)b * C16b;
  for (int c = threadIdx.x; c < C16a; c += blockDim.x) da[c] = sa[c];
  for (int c = threadIdx.x; c < C16b; c += blockDim.x) db[c] = sb[c];
  if (threadIdx.x == 0) lens[b] += i + 1;
}

// embed_norm for bf16 rows of H % 8 == 0 channels, H <= 8 * 256 * kEmbedVec: eight channels
// per 16-byte load, each thread's loads in registers between the two passes
constexpr int kEmbedVec = 4;
__global__ __launch_bounds__(256) void embed_norm_bf16_kernel(int H, int V, const int32_t *__restrict__ tok,
                                                              const uint4 *__restrict__ E, float *__restrict__ x,
                                                              const uint4 *__restrict__ w, float eps,
                                                              uint4 *__restrict__ out, int32_t *dev_err) {
  __shared__ float red[16];
  const int r = blockIdx.x, H8 = H / 8;
  const int t = tok[r];
  const bool ok = t >= 0 && t < V;
  if (!ok && threadIdx.x == 0) raise_dev_err(dev_err, GM_DEVERR_TOKEN);
  const uint4 *er = E + (long)(ok ? t : 0) * H8;
  uint4 v[kEmbedVec];
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < kEmbedVec; ++u) {
    const int c = threadIdx.x + 256 * u;
    v[u] = (ok && c < H8) ? er[c] : make_uint4(0, 0, 0, 0);
    const uint32_t q[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
      ss += lo * lo + hi * hi;
    }
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)H + eps);
  float4 *xr = reinterpret_cast<float4 *>(x + (long)r * H);
  uint4 *o = out + (long)r * H8;
#pragma unroll
  for (int u = 0; u < kEmbedVec; ++u) {
    const int c = threadIdx.x + 256 * u;
    if (c >= H8) continue;
    const uint32_t q[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    const uint4 wv = w[c];
    const uint32_t wq[4] = {wv.x, wv.y, wv.z, wv.w};
    float f[8];
    uint32_t packed[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = __uint_as_float(q[e] << 16);
      f[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
      const float a = f[2 * e] * inv * __uint_as_float(wq[e] << 16);
      const float b = f[2 * e + 1] * inv * __uint_as_float(wq[e] & 0xffff0000u);
      packed[e] = uint32_t(f32_to_bf16(a)) | (uint32_t(f32_to_bf16(b)) << 16);
    }
    xr[2 * c] = make_float4(f[0], f[1], f[2], f[3]);
    xr[2 * c + 1] = make_float4(f[4], f[5], f[6], f[7]);
    o[c] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
  }
}
}  // namespace

void launch_embed(int dtype, int M, int H, int V, const int32_t *tokens, const void *E, float *x, int32_t *dev_err,
                  hipStream_t s) {
  if (M <= 0) return;
  TraceScope ts("embed", s);
  if (dtype == GM_BF16)
    hipLaunchKernelGGL(embed_kernel<bf16>, dim3(M), dim3(256), 0, s, H, V, tokens, (const bf16 *)E, x, dev_err);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, H, V, tokens, (const float *)E, x, dev_err);
}

void launch_embed_norm(int dtype, int M, int H, int V, const int32_t *tokens, const void *E, float *x,
                       const void *norm_w, float eps, void *out, int32_t *dev_err, hipStream_t s) {
  if (M <= 0) return;
  TraceScope ts("embed_norm", s);
  const bool aligned = ((uintptr_t)E | (uintptr_t)x | (uintptr_t)norm_w | (uintptr_t)out) % 16 == 0;
  if (dtype == GM_BF16 && H % 8 == 0 && H <= 8 * 256 * kEmbedVec && aligned)
    hipLaunchKernelGGL(embed_norm_bf16_kernel, dim3(M), dim3(256), 0, s, H, V, tokens, (const uint4 *)E, x,
                       (const uint4 *)norm_w, eps, (uint4 *)out, dev_err);
  else if (dtype == GM_BF16)
    hipLaunchKernelGGL(embed_norm_kernel<bf16>, dim3(M), dim3(256), 0, s, H, V, tokens, (const bf16 *)E, x,
                       (const bf16 *)norm_w, eps, (bf16 *)out, dev_err);
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(M), dim3(256), 0, s, H, V, tokens, (const float *)E, x,
                       (const float *)norm_w, eps, (float *)out, dev_err);
}

void launch_rmsnorm(int dtype, int M, int H, float eps, const float *x, const void *w, void *out, hipStream_t s) {
  if (M <= 0) return;
  TraceScope ts("rmsnorm", s);
  const dim3 grid((M + 3) / 4);
  if (dtype == GM_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16>, grid, dim3(256), 0, s, M, H, eps, x, (const bf16 *)w, (bf16 *)out);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, grid, dim3(256), 0, s, M, H, eps, x, (const float *)w, (float *)out);
}

void launch_rope_append(const RopeArgs &a, hipStream_t s) {
  if (a.M <= 0) return;
  TraceScope ts("rope_append", s);
  const dim3 grid(a.M, (a.n_heads + 2 * a.n_kv + 4 * kRopeHeads - 1) / (4 * kRopeHeads));
  if (a.dtype == GM_BF16) hipLaunchKernelGGL(rope_append_kernel<bf16>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(rope_append_kernel<float>, grid, dim3(256), 0, s, a);
}

void launch_mtp_input(int dtype, int M, int H, int V, float eps, const float *h, const int32_t *tok, int tok_stride,
                      const void *E, const void *norm_h, const void *norm_e, void *out, int32_t *dev_err,
                      hipStream_t s) {
  if (M <= 0) return;
  TraceScope ts("mtp_input", s);
  const int threads = mtp_input_threads(H);
  if (dtype == GM_BF16)
    hipLaunchKernelGGL(mtp_input_kernel<bf16>, dim3(M), dim3(threads), 0, s, H, V, eps, h, tok, tok_stride,
                       (const bf16 *)E, (const bf16 *)norm_h, (const bf16 *)norm_e, (bf16 *)out, dev_err);
  else
    hipLaunchKernelGGL(mtp_input_kernel<float>, dim3(M), dim3(threads), 0, s, H, V, eps, h, tok, tok_stride,
                       (const float *)E, (const float *)norm_h, (const float *)norm_e, (float *)out, dev_err);
}

void launch_gather_commit(int B, int R, int Ca, size_t elem_a, const void *src_a, void *dst_a, int Cb, size_t elem_b,
                          const void *src_b, void *dst_b, const int32_t *sel, int32_t *lens, hipStream_t s) {
  if (B <= 0) return;
  TraceScope ts("gather_commit", s);
  hipLaunchKernelGGL(gather_commit_kernel, dim3(B), dim3(256), 0, s, R, (int)((size_t)Ca * elem_a / 16),
                     (const uint4 *)src_a, (uint4 *)dst_a, (int)((size_t)Cb * elem_b / 16), (const uint4 *)src_b,
                     (uint4 *)dst_b, sel, lens);
}

}  // namespace gm
