// One row of the MTP head's input (App. "Models and Draft Heads"): the hidden
// half and the token-embedding half each pass their own RMSNorm, joined with
// the hidden half first: [RMSNorm(h) * norm_h, RMSNorm(E[tok]) * norm_e], 2H
// values in the model dtype.  Shared by the input kernel and by the draft draw,
// which builds the next chain step's input from the token it has just drawn.
#pragma once

#include "common.h"

namespace gm {

// four consecutive elements of a row (16-byte or 8-byte aligned) as float
__device__ __forceinline__ float4 load4(const float *p, long i) { return *reinterpret_cast<const float4 *>(p + i); }
__device__ __forceinline__ float4 load4(const bf16 *p, long i) {
  const uint2 v = *reinterpret_cast<const uint2 *>(p + i);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                     __uint_as_float(v.y & 0xffff0000u));
}

// The arithmetic is that of a block of VT threads (VT a multiple of 64, at most
// 1024): virtual thread v takes four channels at 4 v, 4 (v + VT), ...; each wave
// of 64 virtual threads sums its squares with one xor-shuffle tree, and the VT / 64
// wave sums are added in wave order.  The calling block (blockDim.x a multiple of
// 64) carries the virtual threads tid, tid + blockDim.x, ..., so the row comes out
// the same whatever block runs it.  Every thread of the block must call this (it
// holds a block barrier); red holds at least VT / 64 entries.
template <typename T>
__device__ __forceinline__ void mtp_input_row(int VT, int H, int V, float eps, const float *__restrict__ hr, int t,
                                              const T *__restrict__ E, const T *__restrict__ nh,
                                              const T *__restrict__ ne, T *__restrict__ o, int32_t *dev_err,
                                              float2 *red) {
  const int nt = blockDim.x, tid = threadIdx.x, lane = tid & 63;
  if (t < 0 || t >= V) {     // -1 pads a row with no token
    if (t >= V && tid == 0) raise_dev_err(dev_err, GM_DEVERR_TOKEN);
    for (int c = tid; c < 2 * H; c += nt) Elem<T>::store(o, c, 0.f);
    return;
  }
  const T *er = E + (long)t * H;
  // Every load of a pass is issued before the first use: up to kMaxVirt virtual threads per
  // thread, one four-channel group each (4 VT >= H); otherwise the general loop.
  constexpr int kMaxVirt = 4;
  if (VT * 4 >= H && VT <= kMaxVirt * nt) {
    float4 a[kMaxVirt], e[kMaxVirt];
#pragma unroll
    for (int i = 0; i < kMaxVirt; ++i) {
      const int v = i * nt + tid;
      const bool ok = i * nt + (tid & ~63) < VT && v * 4 < H;
      a[i] = ok ? load4(hr, v * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
      e[i] = ok ? load4(er, v * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < kMaxVirt; ++i) {
      if (i * nt + (tid & ~63) >= VT) continue;   // a whole virtual wave past VT
      float sh = a[i].x * a[i].x + a[i].y * a[i].y + a[i].z * a[i].z + a[i].w * a[i].w;
      float se = e[i].x * e[i].x + e[i].y * e[i].y + e[i].z * e[i].z + e[i].w * e[i].w;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        sh += __shfl_xor(sh, off, kWave);
        se += __shfl_xor(se, off, kWave);
      }
      if (lane == 0) red[(i * nt + tid) >> 6] = make_float2(sh, se);
    }
    __syncthreads();
    float sh = 0.f, se = 0.f;
    for (int i = 0; i < VT / 64; ++i) {
      sh += red[i].x;
      se += red[i].y;
    }
    const float ih = 1.0f / sqrtf(sh / (float)H + eps), ie = 1.0f / sqrtf(se / (float)H + eps);
#pragma unroll
    for (int i = 0; i < kMaxVirt; ++i) {
      const int c = (i * nt + tid) * 4;
      if (i * nt + tid >= VT || c >= H) continue;
      const float4 wh = load4(nh, c), we = load4(ne, c);
      Elem<T>::store(o, c, a[i].x * ih * wh.x);
      Elem<T>::store(o, c + 1, a[i].y * ih * wh.y);
      Elem<T>::store(o, c + 2, a[i].z * ih * wh.z);
      Elem<T>::store(o, c + 3, a[i].w * ih * wh.w);
      Elem<T>::store(o, H + c, e[i].x * ie * we.x);
      Elem<T>::store(o, H + c + 1, e[i].y * ie * we.y);
      Elem<T>::store(o, H + c + 2, e[i].z * ie * we.z);
      Elem<T>::store(o, H + c + 3, e[i].w * ie * we.w);
    }
    return;
  }
  for (int v0 = 0; v0 < VT; v0 += nt) {
    if (v0 + (tid & ~63) >= VT) continue;   // a whole virtual wave past VT
    const int v = v0 + tid;
    float sh = 0.f, se = 0.f;
    for (int c = v * 4; c < H; c += VT * 4) {
      const float4 a = load4(hr, c), e = load4(er, c);
      sh += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
      se += e.x * e.x + e.y * e.y + e.z * e.z + e.w * e.w;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      sh += __shfl_xor(sh, off, kWave);
      se += __shfl_xor(se, off, kWave);
    }
    if (lane == 0) red[v >> 6] = make_float2(sh, se);
  }
  __syncthreads();
  float sh = 0.f, se = 0.f;
  for (int i = 0; i < VT / 64; ++i) {
    sh += red[i].x;
    se += red[i].y;
  }
  const float ih = 1.0f / sqrtf(sh / (float)H + eps), ie = 1.0f / sqrtf(se / (float)H + eps);
  for (int v = tid; v < VT; v += nt) {
    for (int c = v * 4; c < H; c += VT * 4) {
      const float4 a = load4(hr, c), e = load4(er, c), wh = load4(nh, c), we = load4(ne, c);
      Elem<T>::store(o, c, a.x * ih * wh.x);
      Elem<T>::store(o, c + 1, a.y * ih * wh.y);
      Elem<T>::store(o, c + 2, a.z * ih * wh.z);
      Elem<T>::store(o, c + 3, a.w * ih * wh.w);
      Elem<T>::store(o, H + c, e.x * ie * we.x);
      Elem<T>::store(o, H + c + 1, e.y * ie * we.y);
      Elem<T>::store(o, H + c + 2, e.z * ie * we.z);
      Elem<T>::store(o, H + c + 3, e.w * ie * we.w);
    }
  }
}

// threads of the input kernel's block for hidden size H: one four-channel group per
// thread when H <= 4096
inline int mtp_input_threads(int H) {
  int threads = ((H / 4 + 63) / 64) * 64;
  return threads > 1024 ? 1024 : threads;
}

}  // namespace gm
