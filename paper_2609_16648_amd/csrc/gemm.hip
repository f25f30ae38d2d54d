// Dense layers of the verify forward and the draft head: Y[M,N] = X[M,K] W[N,K]^T.
//
// bf16 path: 256 threads, 128-column (or 64 SwiGLU features) x BM-row tiles,
// k-steps of 64 staged through LDS with the next step's global loads in
// flight, v_mfma_f32_16x16x32_bf16 with float32 accumulation.  The tile order
// is XCD-aware: workgroups are dealt to the 8 XCDs round-robin, so the
// logical tile index is remapped such that the M-tiles that share a weight
// tile run on the same XCD and hit its L2.  Epilogues: float32 store, float32
// residual add in place, store in the model dtype, or SwiGLU (gate and up
// columns of the same features computed by the same lanes).
// float32 path: a plain LDS-tiled FMA kernel.
#include "common.h"
#include "forward.h"

namespace gm {

namespace {
struct GemmK {
  const uint16_t *X, *W;
  void *Y;
  long ldy;
  int M, N, K, ldx, n_m, n_n;
};

constexpr int kBN = 128, kBK = 64, kLds = kBK + 8;

__device__ __forceinline__ void tile_of(int bid, int n_m, int n_n, int &tm, int &tn) {
  const int T = n_m * n_n;
  const int x = bid & 7, slot = bid >> 3, q = T >> 3, rem = T & 7;
  const int L = x * q + (x < rem ? x : rem) + slot;
  tm = L % n_m;
  tn = L / n_m;
}

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

template <int BM, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmK g) {
  __shared__ uint16_t As[BM][kLds];
  __shared__ uint16_t Bs[kBN][kLds];
  constexpr int TM = BM / 32;              // 16-row MFMA tiles per wave (waves 2 x 2)
  constexpr int AL = BM * 8 / 256;         // 16-byte A chunks per thread and k-step
  constexpr int BL = kBN * 8 / 256;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, wm = w >> 1, wn = w & 1;
  const int j = lane & 15, g4 = lane >> 4;
  int tm, tn;
  tile_of(blockIdx.x, g.n_m, g.n_n, tm, tn);
  const int m0 = tm * BM;

  // source rows of this thread's loads
  const uint16_t *asrc[AL];
  bool aval[AL];
#pragma unroll
  for (int u = 0; u < AL; ++u) {
    const int c = tid + 256 * u, row = c >> 3, kc = c & 7;
    aval[u] = m0 + row < g.M;
    asrc[u] = g.X + (long)(aval[u] ? m0 + row : 0) * g.ldx + kc * 8;
  }
  const uint16_t *bsrc[BL];
#pragma unroll
  for (int u = 0; u < BL; ++u) {
    const int c = tid + 256 * u, row = c >> 3, kc = c & 7;
    long wrow;
    if (EPI == EPI_SWIGLU) {
      const int half = row >> 6, within = row & 63, f0 = tn * 64 + half * 32;
      wrow = within < 32 ? f0 + within : (long)g.N + f0 + within - 32;
    } else {
      wrow = (long)tn * kBN + row;
    }
    bsrc[u] = g.W + wrow * g.K + kc * 8;
  }

  floatx4_t acc[TM][4];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  uint4 ra[AL], rb[BL];
#pragma unroll
  for (int u = 0; u < AL; ++u) ra[u] = aval[u] ? *reinterpret_cast<const uint4 *>(asrc[u]) : make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int u = 0; u < BL; ++u) rb[u] = *reinterpret_cast<const uint4 *>(bsrc[u]);

  for (int k0 = 0; k0 < g.K; k0 += kBK) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < AL; ++u) {
      const int c = tid + 256 * u;
      *reinterpret_cast<uint4 *>(&As[c >> 3][(c & 7) * 8]) = ra[u];
    }
#pragma unroll
    for (int u = 0; u < BL; ++u) {
      const int c = tid + 256 * u;
      *reinterpret_cast<uint4 *>(&Bs[c >> 3][(c & 7) * 8]) = rb[u];
    }
    __syncthreads();
    if (k0 + kBK < g.K) {
#pragma unroll
      for (int u = 0; u < AL; ++u)
        ra[u] = aval[u] ? *reinterpret_cast<const uint4 *>(asrc[u] + k0 + kBK) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < BL; ++u) rb[u] = *reinterpret_cast<const uint4 *>(bsrc[u] + k0 + kBK);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8_t af[TM], bfr[4];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = as_bf16x8(*reinterpret_cast<const uint4 *>(&As[wm * (BM / 2) + 16 * a + j][kk * 32 + 8 * g4]));
#pragma unroll
      for (int b = 0; b < 4; ++b)
        bfr[b] = as_bf16x8(*reinterpret_cast<const uint4 *>(&Bs[wn * 64 + 16 * b + j][kk * 32 + 8 * g4]));
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
  }

  // lane holds C[row 16a + 4 g4 + r][col 16b + j] of the wave tile
#pragma unroll
  for (int a = 0; a < TM; ++a) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * (BM / 2) + 16 * a + 4 * g4 + r;
      if (m >= g.M) continue;
      if (EPI == EPI_SWIGLU) {
        uint16_t *y = (uint16_t *)g.Y + (long)m * g.ldy;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int f = tn * 64 + wn * 32 + 16 * b + j;
          y[f] = f32_to_bf16(silu(acc[a][b][r]) * acc[a][b + 2][r]);
        }
      } else {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int n = tn * kBN + wn * 64 + 16 * b + j;
          const float v = acc[a][b][r];
          if (EPI == EPI_STORE_F32) ((float *)g.Y)[(long)m * g.ldy + n] = v;
          else if (EPI == EPI_ADD_F32) ((float *)g.Y)[(long)m * g.ldy + n] += v;
          else ((uint16_t *)g.Y)[(long)m * g.ldy + n] = f32_to_bf16(v);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ float32
struct GemmF {
  const float *X, *W;
  float *Y;
  long ldy;
  int M, N, K, ldx;
};

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmF g) {
  constexpr int TM = 16, TN = 64, TK = 32;
  constexpr int NB = EPI == EPI_SWIGLU ? 2 : 1;
  __shared__ float As[TM][TK + 1];
  __shared__ float Bs[NB][TN][TK + 1];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  float acc[NB][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += TK) {
    for (int e = tid; e < TM * TK; e += 256) {
      const int r = e / TK, c = e % TK, m = m0 + r;
      As[r][c] = (m < g.M && k0 + c < g.K) ? g.X[(long)m * g.ldx + k0 + c] : 0.f;
    }
    for (int nb = 0; nb < NB; ++nb)
      for (int e = tid; e < TN * TK; e += 256) {
        const int r = e / TK, c = e % TK, n = n0 + r;
        Bs[nb][r][c] = (n < g.N && k0 + c < g.K) ? g.W[((long)nb * g.N + n) * g.K + k0 + c] : 0.f;
      }
    __syncthreads();
    for (int c = 0; c < TK; ++c) {
      const float x = As[ty][c];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[nb][q] += x * Bs[nb][tx * 4 + q][c];
    }
    __syncthreads();
  }
  const int m = m0 + ty;
  if (m >= g.M) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int n = n0 + tx * 4 + q;
    if (n >= g.N) continue;
    float *y = g.Y + (long)m * g.ldy + n;
    if (EPI == EPI_ADD_F32) *y += acc[0][q];
    else if (EPI == EPI_SWIGLU) *y = silu(acc[0][q]) * acc[NB - 1][q];
    else *y = acc[0][q];
  }
}
}  // namespace

void launch_gemm(const char *name, int dtype, int epi, int M, int N, int K, const void *X, int ldx, const void *W,
                 void *Y, long ldy, hipStream_t s) {
  if (M <= 0) return;
  if (dtype == GM_BF16) {
    GemmK g{(const uint16_t *)X, (const uint16_t *)W, Y, ldy, M, N, K, ldx, 0, 0};
    const bool small = M <= 64;
    const int BM = small ? 64 : 128;
    g.n_m = (M + BM - 1) / BM;
    g.n_n = epi == EPI_SWIGLU ? N / 64 : N / kBN;
    const dim3 grid(g.n_m * g.n_n), block(256);
    TraceScope ts(name, s);
#define GM_GEMM_CASE(E)                                                                   \
  case E:                                                                                 \
    if (small) hipLaunchKernelGGL((gemm_bf16_kernel<64, E>), grid, block, 0, s, g);       \
    else hipLaunchKernelGGL((gemm_bf16_kernel<128, E>), grid, block, 0, s, g);            \
    break;
    switch (epi) {
      GM_GEMM_CASE(EPI_STORE_F32)
      GM_GEMM_CASE(EPI_ADD_F32)
      GM_GEMM_CASE(EPI_STORE_ACT)
      GM_GEMM_CASE(EPI_SWIGLU)
    }
#undef GM_GEMM_CASE
  } else {
    GemmF g{(const float *)X, (const float *)W, (float *)Y, ldy, M, N, K, ldx};
    const dim3 grid((N + 63) / 64, (M + 15) / 16), block(256);
    TraceScope ts(name, s);
    switch (epi) {
      case EPI_STORE_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, block, 0, s, g); break;
      case EPI_ADD_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_ADD_F32>, grid, block, 0, s, g); break;
      case EPI_STORE_ACT: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_ACT>, grid, block, 0, s, g); break;
      case EPI_SWIGLU: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, g); break;
    }
  }
}

}  // namespace gm
