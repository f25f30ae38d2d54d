// Device-side helpers shared by the gfx950 kernels of the speculative step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gm.h"

namespace gm {

constexpr int kWave = 64;

// ----------------------------------------------------------------- bf16
// bfloat16 is carried as its uint16 bit pattern.
struct bf16 {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// float -> bf16, round to nearest even (inputs are finite; NaN maps to a quiet NaN)
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  b += 0x7fffu + ((b >> 16) & 1u);
  return uint16_t(b >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float *p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float *p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16> {
  static __device__ __forceinline__ float load(const bf16 *p, size_t i) { return bf16_to_f32(p[i].bits); }
  static __device__ __forceinline__ void store(bf16 *p, size_t i, float v) { p[i].bits = f32_to_bf16(v); }
};

// ----------------------------------------------------------------- MFMA operand vectors
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// 16-byte load marked non-temporal: data read once per launch (weights, KV) then does
// not displace what the launch re-reads from the caches
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_nt(const void *p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ bf16x4_t as_bf16x4(uint2 v) { return __builtin_bit_cast(bf16x4_t, v); }

// ----------------------------------------------------------------- reductions
// Orders this wave's LDS writes before its later LDS reads by other lanes (a
// wave's LDS operations complete in order; this keeps the compiler from moving
// them across and waits for the writes).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); every thread gets the result.
template <typename F>
__device__ __forceinline__ F block_sum(F v, F *smem /* >= 16 */) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) smem[wid] = v;
  __syncthreads();
  F t = 0;
  for (int i = 0; i < nw; ++i) t += smem[i];
  return t;
}

// Sum, in split order, of `splits` float4 values stride floats apart (K-split
// partials of one output element group); the loads of a batch are all issued
// before the first add (batches of 16 when there are more than 8 splits, so
// that up to 16 take one round trip).
template <int kBatch>
__device__ __forceinline__ void sum_splits_batched(const float *p, long stride, int splits, float4 &a) {
  for (int s0 = 0; s0 < splits; s0 += kBatch) {
    float4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int sp = s0 + u < splits ? s0 + u : splits - 1;
      v[u] = *reinterpret_cast<const float4 *>(p + sp * stride);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s0 + u < splits) {
        a.x += v[u].x;
        a.y += v[u].y;
        a.z += v[u].z;
        a.w += v[u].w;
      }
    }
  }
}
__device__ __forceinline__ float4 sum_splits(const float *p, long stride, int splits) {
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  if (splits > 8) sum_splits_batched<16>(p, stride, splits, a);
  else sum_splits_batched<8>(p, stride, splits, a);
  return a;
}

// ----------------------------------------------------------------- weight tile layout
// bf16 linear weights (gm.h): 1 KiB tiles of 16 rows (a strip) x 32 columns (a
// k-step); the strips come in groups of 8, and inside a group the 8 tiles of
// one k-step are consecutive, so the strips a wave or workgroup streams
// together sit in one contiguous run per k-step.
constexpr int kWGroup = 8;                      // strips per group
constexpr int kWStep = kWGroup * 512;           // elements from k-step kt to kt + 1 of a strip
// element offset of the tile (strip s, k-step kt) of a weight with `ksteps` k-steps
__device__ __forceinline__ long w_tile(int s, int kt, int ksteps) {
  return (((long)(s / kWGroup) * ksteps + kt) * kWGroup + s % kWGroup) * 512;
}

// ----------------------------------------------------------------- KV tile layout
// Offsets inside the 16-token tile of one (page, kv head); see gm.h.
__device__ __forceinline__ int k_tile_off(int s, int c) {
  return (c >> 5) * 512 + ((c & 31) >> 3) * 128 + s * 8 + (c & 7);
}
__device__ __forceinline__ int v_tile_off(int s, int c) {
  return (c >> 5) * 512 + (s >> 2) * 128 + (c & 15) * 8 + ((c >> 4) & 1) * 4 + (s & 3);
}

__device__ __forceinline__ void raise_dev_err(int32_t *err, int bit) {
  if (err) atomicOr(err, bit);
}

}  // namespace gm
