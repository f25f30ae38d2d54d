// Dense layers of the verify forward and the draft head: Y[M,N] = X[M,K] W[N,K]^T.
//
// bf16 path ("streaming" GEMM for M <= 256 rows per tile, the regime of a
// verify step: every weight byte is read once and used for all M rows).
//  * Weights are stored pre-tiled (gm.h): tiles of 16 rows x 32 k (1 KiB)
//    laid out so that one 16-byte-per-lane load of a wave is the B operand of
//    v_mfma_f32_16x16x32_bf16, with the tiles of 8 strips (16-row groups) of
//    one k-step side by side.  A wave streams its strips along K, straight
//    from HBM into registers, through a prefetch ring several k-steps deep;
//    W never touches LDS.
//  * Activations (small, L2-resident) are staged in LDS in 16 or 32 KiB
//    chunks, three deep, by one extra wave of direct-to-LDS loads, one barrier
//    per chunk, shared by the 4 compute waves (5 or 7 for wide outputs, up to
//    two per SIMD, so that one wave's LDS reads overlap another's MFMAs).
//  * Small N is split along K (deterministic two-pass reduction: float32
//    partials, then a reduce kernel that sums the splits in order and applies
//    the epilogue) so that a launch fills the 256 CUs.
//  * Tile order is XCD-aware: the M tiles and K splits of one weight strip are
//    dealt to the same XCD, so a weight strip re-read by several M tiles hits
//    that XCD's L2.
//  * Epilogues: float32 store, float32 residual add in place, store in the
//    model dtype, SwiGLU (gate and up strips of the same features sit in the
//    same wave, so silu(gate) * up is formed in registers).
// float32 path: a plain LDS-tiled FMA kernel on row-major weights.
#include <atomic>
#include <type_traits>

#include "common.h"
#include "forward.h"

namespace gm {

namespace {
// Weight tiles read by one workgroup only are loaded non-temporally: they then
// do not evict the activations, which every workgroup re-reads from L2
// (measured: 5-6% off the M <= 64 LM head).  Weight strips re-read by the M
// tiles of a launch take ordinary loads, as that re-read is meant to hit L2.
template <bool STREAM>
__device__ __forceinline__ uint4 load_w(const uint16_t *p) {
  if (STREAM) return load_nt(p);
  return *reinterpret_cast<const uint4 *>(p);
}

struct GemmS {
  const uint16_t *X, *W;
  void *Y;
  float *part;        // [splits][M][Nw] float32 partials when splits > 1
  long ldy;
  int M, N, K, ldx;   // N: output columns (features for SwiGLU); Nw: weight rows
  int Nw, n_tiles, m_tiles, splits, k_iters;
  RowStat *stats;     // EPI_STATS: [M][Nw / kStatCols] tile statistics of Y / T
  float inv_t;
};

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

// CW compute waves and one A-staging wave
template <int CW> constexpr int gemm_threads() { return (CW + 1) * kWave; }
constexpr int kStatCols = kMaxTileStrips * kStripIds;   // columns per statistics tile of the tiled GEMM
constexpr int kGemmBufs = 3;              // A chunks in LDS (the loader runs two ahead)
// s_waitcnt immediates (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8; the other counters left at their maximum, i.e. not waited on)
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kVmcnt0 = waitcnt_vm(0);
// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int kSchedMfma = 0x008, kSchedDsRead = 0x100;

// logical tile index of workgroup `bid`: workgroups are dealt round-robin to
// the 8 XCDs; consecutive logical indices (same weight strip) share an XCD
__device__ __forceinline__ int xcd_remap(int bid, int T) {
  const int x = bid & 7, slot = bid >> 3, q = T >> 3, rem = T & 7;
  return x * q + (x < rem ? x : rem) + slot;
}

// MT: 16-row tiles per compute wave; NT: 16-column strips per compute wave;
// WM: compute waves along M (1 or 2); SW: weights loaded non-temporally (one M
// tile); CW: compute waves (4; for wide outputs 7, two per SIMD on three of
// the SIMDs with 224-column tiles, or 5 with 160-column tiles; the last tile of
// a launch clamped to the output).  Waves 0 .. CW - 1 compute; wave CW only
// stages the A chunks in LDS.
// The wait counter of loads is per wave, so the loader's waits for A never
// drain the compute waves' weight ring.
template <int MT, int NT, int WM, int EPI, bool SW, int CW>
__global__ __launch_bounds__(gemm_threads<CW>()) void gemm_stream_kernel(GemmS g) {
  static_assert(CW % WM == 0, "compute waves tile the rows evenly");
  constexpr int WN = CW / WM;
  constexpr int BM = 16 * MT * WM;            // rows per workgroup
  constexpr int BKA = (BM >= 256 ? 16384 : 8192) / BM;   // k per LDS chunk of A (16 KiB; 32 KiB at 256 rows)
  constexpr int SPC = BKA / 32;               // k32 steps per chunk
  constexpr int D = NT >= 4 ? 4 : 8;          // W prefetch depth (k32 steps)
  static_assert(EPI != EPI_STATS || 16 * NT * WN == kStatCols, "tile statistics cover one workgroup's columns");
  constexpr int PA = MT >= 8 ? 4 : MT;        // A fragments read ahead (all of them up to 64 rows)
  constexpr int ITER = D > SPC ? D : SPC;     // k32 steps per unrolled iteration
  constexpr int CB = BKA / 8;                 // 16-byte column blocks per A row of a chunk
  constexpr int SWZ = CB < 16 ? CB - 1 : 15;  // XOR swizzle of the column block by the row
  constexpr int AL = BM * BKA / 8 / kWave;    // 1 KiB direct-to-LDS loads per chunk
  constexpr int kVmcntAL = waitcnt_vm(AL);
  static_assert(ITER % SPC == 0 && ITER % D == 0, "unroll must cover whole chunks and ring turns");
  static_assert(ITER == 8, "plan_gemm counts K in iterations of 8 k32 steps");
  // A chunk: row r, column block p of LDS holds X[r][8 (p ^ (r & SWZ)) ...]
  __shared__ uint16_t As[kGemmBufs][BM * BKA];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // CW: the loader wave
  const int wm = w % WM, wn = w / WM;
  const int j = lane & 15, g4 = lane >> 4;
  const int T = g.n_tiles * g.m_tiles * g.splits;
  const int L = xcd_remap(blockIdx.x, T);
  const int mt = L % g.m_tiles, rest = L / g.m_tiles;
  const int ks = rest % g.splits, nt = rest / g.splits;
  const int m0 = mt * BM;
  // this split's k range, in whole unrolled iterations (at least one)
  const int it0 = (int)((long)g.k_iters * ks / g.splits), it1 = (int)((long)g.k_iters * (ks + 1) / g.splits);
  const int k_begin = it0 * ITER * 32, k_end = it1 * ITER * 32;
  const int nsteps = (k_end - k_begin) / 32;
  const int nchunks = nsteps / SPC;

  // weight strips of this wave: strip index (16-row groups of W)
  int strip[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (EPI == EPI_SWIGLU) {
      // NT/2 gate strips then the NT/2 up strips of the same 16 * NT/2 features
      const int f_strip = (nt * WN + wn) * (NT / 2) + (t % (NT / 2));
      strip[t] = (t < NT / 2) ? f_strip : g.N / 16 + f_strip;
    } else {
      strip[t] = (nt * WN + wn) * NT + t;
    }
  }

  floatx4_t acc[MT][NT];
#pragma unroll
  for (int a = 0; a < MT; ++a)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[a][t] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  // Barrier c (c = 0 .. nchunks) closes "loader stored chunk c" and "compute
  // finished chunk c - 1".  Chunk c lives in As[c % 3]; the buffer was last used
  // by chunk c - 3, finished before barrier c - 2, so the loader starts chunk c
  // right after barrier c - 2 and has two chunks of compute time to land it.
  if (w == CW) {
    // Direct-to-LDS loads: lane l of load u fills the 16 bytes at u KiB + 16 l of the
    // chunk, i.e. row e / CB, block e % CB (e = 64 u + l); the lane fetches the
    // global block that the swizzle puts there.  No registers hold A, and this
    // wave's own waits (before each barrier) are the only ones A costs.
    auto issue = [&](int c) {
      const int chunk_k = k_begin + c * BKA;
      uint16_t *dst = &As[c % kGemmBufs][0];
#pragma unroll
      for (int u = 0; u < AL; ++u) {   // rows past M re-read row M - 1 (never stored)
        const int e = lane + kWave * u, row = e / CB, p = e % CB;
        const uint16_t *src = g.X + (long)min(m0 + row, g.M - 1) * g.ldx + chunk_k + 8 * (p ^ (row & SWZ));
        __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(dst + u * 512), 16, 0, 0);
      }
    };
    issue(0);
    if (nchunks > 1) issue(1);
    for (int c = 0; c < nchunks; ++c) {
      // chunk c landed: at most the AL loads of chunk c + 1 still in flight
      if (c + 1 < nchunks) __builtin_amdgcn_s_waitcnt(kVmcntAL);
      else __builtin_amdgcn_s_waitcnt(kVmcnt0);
      __builtin_amdgcn_s_barrier();   // barrier c
      if (c + 2 < nchunks) issue(c + 2);
    }
    __builtin_amdgcn_s_barrier();     // barrier nchunks
  } else {
    // The weight ring is loaded unconditionally (indices clamped to the last
    // step, a re-read near the end), so the loop is one straight path: every
    // wait counts exactly the loads still in flight and the ring stays full
    // across iterations and chunk barriers.
    const int kt_total = g.K / 32;
    const uint16_t *wbase[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)   // strips past the weight (the last wide tile) re-read the last one
      wbase[t] = g.W + w_tile(CW == 4 ? strip[t] : min(strip[t], g.Nw / 16 - 1), k_begin / 32, kt_total) + lane * 8;
    // Slot d of the ring holds step d mod D.  Each step first refills the slot
    // consumed by the step before (its registers are dead), then consumes its
    // own: a load never targets a register still waiting for its reader, so the
    // ring keeps fixed registers across loop turns and no wait drains it.
    uint4 ring[D][NT];
#pragma unroll
    for (int s = 0; s < D - 1; ++s) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < NT; ++t) ring[s][t] = load_w<SW>(wbase[t] + (long)min(s, nsteps - 1) * kWStep);
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();     // barrier 0

    for (int s0 = 0; s0 < nsteps; s0 += ITER) {
#pragma unroll
      for (int u = 0; u < ITER; ++u) {
        const int s = s0 + u;                 // global k32 step
        const int buf = (s / SPC) % kGemmBufs;
        const int ko = (u % SPC) * 32;        // offset inside the chunk
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < NT; ++t)
          ring[(u + D - 1) % D][t] = load_w<SW>(wbase[t] + (long)min(s + D - 1, nsteps - 1) * kWStep);
        __builtin_amdgcn_sched_barrier(0);
        const uint4 (&wv)[NT] = ring[u % D];
        // A fragments from LDS, PA reads ahead of the MFMAs that use them; left to itself the
        // compiler keeps only two in flight and waits out their latency before every pair
        bf16x8_t af[MT];
        auto read_a = [&](int a) {
          const int rr = wm * 16 * MT + 16 * a + j;
          const int p = ((ko >> 3) + g4) ^ (rr & SWZ);
          af[a] = as_bf16x8(*reinterpret_cast<const uint4 *>(&As[buf][rr * BKA + 8 * p]));
        };
#pragma unroll
        for (int a = 0; a < PA; ++a) read_a(a);
#pragma unroll
        for (int a = 0; a < MT; ++a) {
          if (a + PA < MT) read_a(a + PA);
#pragma unroll
          for (int t = 0; t < NT; ++t)
            acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], as_bf16x8(wv[t]), acc[a][t], 0, 0, 0);
        }
        if (PA < MT) {   // the order above, held against the scheduler: PA reads, then a read per MFMA group
          __builtin_amdgcn_sched_group_barrier(kSchedDsRead, PA, 0);
#pragma unroll
          for (int a = 0; a < MT; ++a) {
            if (a + PA < MT) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, NT, 0);
          }
        }
        if ((u % SPC) == SPC - 1) __syncthreads();   // barrier s / SPC + 1: done with this chunk
      }
    }
  }

  // The statistics come first: the barriers they need wait for every outstanding memory
  // operation, and the logits' stores, issued last, then drain after the waves have left
  // (the next workgroup on this CU starts streaming meanwhile).
  if (EPI == EPI_STATS) {
    // Softmax statistics of this workgroup's kStatCols columns, per row.  The A buffers are
    // free once the K loop is done: the tile of z / T goes there in parts of RP rows (row
    // stride LS floats), then each thread reduces one row over the kStatCols columns in
    // ascending id order -- the max, the first id attaining it, and the float64 sum of
    // float32 terms exp(z / T - max).  No cross-lane reductions.
    constexpr int RP = BM >= 256 ? 128 : 64;
    constexpr int LS = kStatCols + 4;   // a lane's float4 reads of consecutive rows fall on distinct banks
    static_assert(RP * LS * 4 <= kGemmBufs * BM * BKA * 2, "a part of the tile fits the A buffers");
    float *tl = reinterpret_cast<float *>(&As[0][0]);
#pragma unroll
    for (int h = 0; h < BM / RP; ++h) {
      __syncthreads();
      if (w < CW) {
#pragma unroll
        for (int a = 0; a < MT; ++a) {
          const int r0 = wm * 16 * MT + 16 * a;
          if (r0 < h * RP || r0 >= (h + 1) * RP) continue;
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t)
              tl[(r0 + 4 * g4 + r - h * RP) * LS + wn * 16 * NT + 16 * t + j] = acc[a][t][r] * g.inv_t;
        }
      }
      __syncthreads();
      for (int rl = tid; rl < RP; rl += gemm_threads<CW>()) {
        const int m = m0 + h * RP + rl;
        if (m >= g.M) continue;
        const float4 *src = reinterpret_cast<const float4 *>(tl + rl * LS);
        float mx = -INFINITY;
        int arg = 0;
#pragma unroll 8
        for (int c = 0; c < kStatCols / 4; ++c) {
          const float4 v = src[c];
          if (v.x > mx) { mx = v.x; arg = 4 * c; }
          if (v.y > mx) { mx = v.y; arg = 4 * c + 1; }
          if (v.z > mx) { mx = v.z; arg = 4 * c + 2; }
          if (v.w > mx) { mx = v.w; arg = 4 * c + 3; }
        }
        double sum = 0.0;
#pragma unroll 8
        for (int c = 0; c < kStatCols / 4; ++c) {
          const float4 v = src[c];
          sum += (double)expf(v.x - mx) + (double)expf(v.y - mx) + (double)expf(v.z - mx) + (double)expf(v.w - mx);
        }
        RowStat o;
        o.max = mx;
        o.argmax = nt * kStatCols + arg;
        o.sum = sum;
        g.stats[(long)m * (g.Nw / kStatCols) + nt] = o;
      }
    }
  }

  if (w < CW) {
  // lane holds C[row 16a + 4 g4 + r][col 16t + j] of the wave tile
#pragma unroll
  for (int a = 0; a < MT; ++a) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * 16 * MT + 16 * a + 4 * g4 + r;
      if (m >= g.M) continue;
      if (g.splits > 1) {
        float *p = g.part + ((long)ks * g.M + m) * g.Nw;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (CW != 4 && (EPI == EPI_SWIGLU ? strip[t % (NT / 2)] >= g.N / 16 : strip[t] >= g.Nw / 16)) continue;
          p[strip[t] * 16 + j] = acc[a][t][r];
        }
      } else if (EPI == EPI_SWIGLU) {
        uint16_t *y = (uint16_t *)g.Y + (long)m * g.ldy;
#pragma unroll
        for (int t = 0; t < NT / 2; ++t) {
          if (CW != 4 && strip[t] >= g.N / 16) continue;   // features past the output (last tile)
          y[strip[t] * 16 + j] = f32_to_bf16(silu(acc[a][t][r]) * acc[a][t + NT / 2][r]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (CW != 4 && strip[t] >= g.Nw / 16) continue;
          const long o = (long)m * g.ldy + strip[t] * 16 + j;
          const float v = acc[a][t][r];
          if (EPI == EPI_STORE_F32 || EPI == EPI_STATS) ((float *)g.Y)[o] = v;
          else if (EPI == EPI_ADD_F32) ((float *)g.Y)[o] += v;
          else ((uint16_t *)g.Y)[o] = f32_to_bf16(v);
        }
      }
    }
  }

  }
}

// sum of the K-split partials in split order, then the epilogue
template <int EPI>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(GemmS g) {
  // four consecutive columns per thread (N % 4 == 0)
  const long total = (long)g.M * (g.N / 4);
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const int m = (int)(i / (g.N / 4)), n = (int)(i % (g.N / 4)) * 4;
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < g.splits; ++s) {
      const float *p = g.part + ((long)s * g.M + m) * g.Nw;
      const float4 x = *reinterpret_cast<const float4 *>(p + n);
      a.x += x.x; a.y += x.y; a.z += x.z; a.w += x.w;
      if (EPI == EPI_SWIGLU) {
        const float4 y = *reinterpret_cast<const float4 *>(p + g.N + n);
        b.x += y.x; b.y += y.y; b.z += y.z; b.w += y.w;
      }
    }
    const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
    const long o = (long)m * g.ldy + n;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (EPI == EPI_STORE_F32 || EPI == EPI_STATS) ((float *)g.Y)[o + q] = av[q];
      else if (EPI == EPI_ADD_F32) ((float *)g.Y)[o + q] += av[q];
      else if (EPI == EPI_SWIGLU) ((uint16_t *)g.Y)[o + q] = f32_to_bf16(silu(av[q]) * bv[q]);
      else ((uint16_t *)g.Y)[o + q] = f32_to_bf16(av[q]);
    }
  }
}

// The K-split partials of a [M][N] float32 output summed in split order (plus the
// residual already in Y for EPI_ADD_F32) into Y, followed by the RMSNorm of each
// row into `out` (model dtype, weight w): the reduce and the norm that always
// follows it in one pass.  One block per row, a float4 column group per thread
// and step (N % 4 == 0), the row kept in LDS between the two passes.
template <typename T, int EPI>
__global__ __launch_bounds__(1024) void reduce_norm_kernel(int M, int N, int splits, const float *__restrict__ part,
                                                           float *__restrict__ Y, const T *__restrict__ w, float eps,
                                                           T *__restrict__ out) {
  extern __shared__ float row_sh[];   // [N]
  __shared__ float red[16];
  const int m = blockIdx.x;
  float *y = Y + (long)m * N;
  float ss = 0.f;
  for (int n = threadIdx.x * 4; n < N; n += blockDim.x * 4) {
    float4 a = sum_splits(part + (long)m * N + n, (long)M * N, splits);
    if (EPI == EPI_ADD_F32) {
      const float4 r = *reinterpret_cast<const float4 *>(y + n);
      a = make_float4(r.x + a.x, r.y + a.y, r.z + a.z, r.w + a.w);
    }
    *reinterpret_cast<float4 *>(y + n) = a;
    *reinterpret_cast<float4 *>(row_sh + n) = a;
    ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)N + eps);
  T *o = out + (long)m * N;
  for (int n = threadIdx.x * 4; n < N; n += blockDim.x * 4) {
    const float4 a = *reinterpret_cast<const float4 *>(row_sh + n);
    Elem<T>::store(o, n, a.x * inv * Elem<T>::load(w, n));
    Elem<T>::store(o, n + 1, a.y * inv * Elem<T>::load(w, n + 1));
    Elem<T>::store(o, n + 2, a.z * inv * Elem<T>::load(w, n + 2));
    Elem<T>::store(o, n + 3, a.w * inv * Elem<T>::load(w, n + 3));
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

// ------------------------------------------------------------------ LM head, M <= 64
// Persistent strip ranges: as many waves as the chip holds, each owning a
// contiguous range of 16-column weight strips (at most kLmStrips, balanced to
// within one strip over all waves) over the whole K.  A wave streams its weight
// tiles through a kLmRing-step register ring with unconditional loads (kLmStrips
// or kLmStrips - 1 strips, the last one again where its range is shorter, so
// the four waves of a workgroup keep pace).  The activation fragments (64
// rows) are shared by the workgroup's four waves: each stages a quarter of every
// kLmChunk-step chunk in LDS, in the A-operand order, with direct-to-LDS loads one
// chunk ahead, and one barrier per chunk hands the chunk over (measured at 64
// rows: 144-147 us per launch against 152-158 us with every wave reading its own
// fragments from L2).  EPI_STATS: the softmax statistics of Y / T are taken per
// row over the wave's own range (float32 terms, summed per lane in float32, the
// 16 lane sums of a row in float64), one RowStat per (row, wave): the tiles of
// the draw are the waves' ranges.
constexpr int kLmStrips = 10;
// Two slots: one k-step (10 KiB of weights per wave) in flight while the other is consumed.
// With four waves per CU that is about as much as the HBM queues serve best; deeper rings put
// more in flight and were slower (measured at 64 rows: 2 slots 146 us per launch, 4 slots
// 151 us, 5 slots 152 us).
constexpr int kLmRing = 2;
// k-steps per activation chunk (4 KiB per k-step for 64 rows; two chunk buffers).  Two-step
// chunks, two ahead, took 151-153 us; an odd count makes the ring slot of a step dynamic.
constexpr int kLmChunk = 4;
static_assert(kLmChunk % kLmRing == 0, "a chunk covers whole ring turns");
static_assert(kLmChunk * kLmStrips <= 63, "the chunk's wait counts its weight loads in the 6-bit vmcnt");
static_assert(kLmStrips * kStripIds <= kMaxDrawTileIds, "the draw scans a whole strip range");

struct GemmL {
  const uint16_t *X, *W;
  float *Y;
  long ldy;
  int M, K, ldx;
  TileGeom geo;       // strips = N / 16, tiles = waves
  RowStat *stats;     // EPI_STATS: [M][waves]
  float inv_t;
};

template <int EPI>
__global__ __launch_bounds__(256) void lm_strips_kernel(GemmL g) {
  const int lane = threadIdx.x & 63, j = lane & 15, g4 = lane >> 4;
  const int wv = threadIdx.x >> 6;
  const int wid = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + wv);
  // a wave past the last range still stages its share of the activations and meets the
  // barriers (streaming strip 0), then leaves before the epilogue
  const bool active = wid < g.geo.tiles;
  const int s0 = active ? tile_first_strip(g.geo, wid) : 0;
  const int n = active ? tile_first_strip(g.geo, wid + 1) - s0 : 1;   // 1 .. kLmStrips
  const int ksteps = g.K / 32;   // a multiple of kLmChunk
  const int nchunks = ksteps / kLmChunk;
  const uint16_t *wb[kLmStrips];
#pragma unroll
  for (int t = 0; t < kLmStrips; ++t) wb[t] = g.W + w_tile(s0 + min(t, n - 1), 0, ksteps) + lane * 8;

  floatx4_t acc[4][kLmStrips];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int t = 0; t < kLmStrips; ++t) acc[a][t] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  // Activation chunk c in As[c % 2], 1 KiB per (k-step st, row tile a) at (4 st + a) KiB:
  // lane l holds row 16 a + (l & 15) (rows past M re-read row M - 1), k 8 (l >> 4) ..
  // of that step, i.e. the A operand as the MFMA takes it.  Wave w stages the loads
  // u = kLmChunk w .. kLmChunk (w + 1) - 1.
  __shared__ uint16_t As[2][kLmChunk * 4 * 512];
  auto issue_a = [&](int c) {
    const int cc = min(c, nchunks - 1);   // past the end: the last chunk again, into the free buffer
    uint16_t *dst = &As[c % 2][0];
#pragma unroll
    for (int q = 0; q < kLmChunk; ++q) {
      const int u = wv * kLmChunk + q, st = u >> 2, a = u & 3;
      const uint16_t *src = g.X + (long)min(16 * a + j, g.M - 1) * g.ldx + (kLmChunk * cc + st) * 32 + 8 * g4;
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)(dst + u * 512), 16, 0, 0);
    }
  };
  // The K loop for a wave that streams NS strips: kLmStrips where its range has that many,
  // else kLmStrips - 1 (the last strip of a shorter range again where it has fewer), so
  // that a CU's four waves load 37-38 strips per k-step rather than 40.  The load order
  // fixes the waits: A(0), the weights of steps 0 .. kLmRing - 2; then per chunk c: A(c + 1),
  // and per step s the weights of step s + kLmRing - 1.
  auto k_loop = [&](auto ns_tag) {
    constexpr int NS = decltype(ns_tag)::value;
    uint4 rw[kLmRing][NS];
    auto load_w_step = [&](int slot, int step) {
#pragma unroll
      for (int t = 0; t < NS; ++t) rw[slot][t] = load_w<true>(wb[t] + (long)step * kWStep);
    };
    __builtin_amdgcn_sched_barrier(0);
    issue_a(0);
#pragma unroll
    for (int d = 0; d < kLmRing - 1; ++d) load_w_step(d, d);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((kLmRing - 1) * NS));   // A(0) landed
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    for (int c = 0; c < nchunks; ++c) {
#pragma unroll
      for (int d = 0; d < kLmChunk; ++d) {
        const int s = kLmChunk * c + d;
        __builtin_amdgcn_sched_barrier(0);
        if (d == 0) issue_a(c + 1);   // into the buffer of chunk c - 1, released by the last barrier
        load_w_step((d + kLmRing - 1) % kLmRing, min(s + kLmRing - 1, ksteps - 1));
        __builtin_amdgcn_sched_barrier(0);
        bf16x8_t af[4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
          af[a] = as_bf16x8(*reinterpret_cast<const uint4 *>(&As[c % 2][(d * 4 + a) * 512 + lane * 8]));
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int t = 0; t < NS; ++t)
            acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], as_bf16x8(rw[d % kLmRing][t]), acc[a][t], 0, 0, 0);
      }
      // A(c + 1) landed: issued after it, the weights of this chunk's kLmChunk steps
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(kLmChunk * NS));
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (n == kLmStrips) k_loop(std::integral_constant<int, kLmStrips>{});
  else k_loop(std::integral_constant<int, kLmStrips - 1>{});
  __builtin_amdgcn_s_waitcnt(kVmcnt0);   // the clamped re-reads past the end, before the waves leave
  if (!active) return;

  // lane holds C[row 16 a + 4 g4 + r][col 16 (s0 + t) + j]
#pragma unroll
  for (int a = 0; a < 4; ++a) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 16 * a + 4 * g4 + r;
      if (m < g.M) {
        float *y = g.Y + (long)m * g.ldy + (long)s0 * 16 + j;
#pragma unroll
        for (int t = 0; t < kLmStrips; ++t)
          if (t < n) y[16 * t] = acc[a][t][r];
      }
    }
  }
  if (EPI == EPI_STATS) {
    // Softmax statistics of the range per row.  A row's values sit in the 16 lanes
    // of one lane group (j) times the range's strips.  Each lane's per-row partials
    // go through this wave's slice of LDS, where lane L then owns row L: the
    // partial maxima (and lowest ids) meet there, the row maxima go back to the
    // lanes, and their partial sums of exp(z / T - max) (float32, at most
    // kLmStrips terms) meet again and are added in float64.  No cross-lane
    // shuffles and no branches on the lane.
    __shared__ float sh_part[4][64 * 17];   // [row][lane group j], padded
    __shared__ int sh_arg[4][64 * 17];
    __shared__ float sh_rmax[4][64];
    float *pf = sh_part[wv], *rmax = sh_rmax[wv];
    int *pa = sh_arg[wv];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float vmax = -INFINITY;
        int varg = 0x7fffffff;
#pragma unroll
        for (int t = 0; t < kLmStrips; ++t) {
          const float v = acc[a][t][r] * g.inv_t;
          if (t < n && v > vmax) { vmax = v; varg = (s0 + t) * 16 + j; }   // ascending ids per lane
        }
        const int row = 16 * a + 4 * g4 + r;
        pf[row * 17 + j] = vmax;
        pa[row * 17 + j] = varg;
      }
    }
    wave_lds_sync();
    float M = -INFINITY;
    int A = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const float mq = pf[lane * 17 + q];
      const int aq = pa[lane * 17 + q];
      if (mq > M || (mq == M && aq < A)) { M = mq; A = aq; }
    }
    rmax[lane] = M;
    wave_lds_sync();
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * a + 4 * g4 + r;
        const float mr = rmax[row];
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < kLmStrips; ++t)
          if (t < n) sum += expf(acc[a][t][r] * g.inv_t - mr);
        pf[row * 17 + j] = sum;
      }
    }
    wave_lds_sync();
    double S = 0.0;
#pragma unroll
    for (int q = 0; q < 16; ++q) S += (double)pf[lane * 17 + q];
    if (lane < g.M) {
      RowStat st;
      st.max = M;
      st.argmax = A;
      st.sum = S;
      g.stats[(long)lane * g.geo.tiles + wid] = st;
    }
  }
}

// waves of lm_strips_kernel the device holds at once (queried once per device)
int lm_resident_waves() {
  static std::atomic<int> cache[16];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 1024;
  int v = cache[dev].load();
  if (v > 0) return v;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, lm_strips_kernel<EPI_STATS>, 256, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || per_cu < 1 || cus < 1) {
    (void)hipGetLastError();
    return 1024;
  }
  v = per_cu * cus * 4;
  cache[dev].store(v);
  return v;
}

template <int MT, int NT, int WM, int EPI, int CW>
void launch_stream(const GemmS &g, hipStream_t s) {
  const dim3 grid(g.n_tiles * g.m_tiles * g.splits);
  if (g.m_tiles == 1)
    hipLaunchKernelGGL((gemm_stream_kernel<MT, NT, WM, EPI, true, CW>), grid, dim3(gemm_threads<CW>()), 0, s, g);
  else
    hipLaunchKernelGGL((gemm_stream_kernel<MT, NT, WM, EPI, false, CW>), grid, dim3(gemm_threads<CW>()), 0, s, g);
}

template <int EPI>
void launch_stream_shape(int shape, int cw, const GemmS &g, hipStream_t s) {
  // four compute waves: 128-column tiles, one tile-statistics block each; five or seven
  // (no statistics): 160- or 224-column tiles
  if constexpr (EPI != EPI_STATS) {
    if (cw == 5) {
      launch_stream<8, 2, 1, EPI, 5>(g, s);                   // 128 x 160 tiles
      return;
    }
    if (cw == 7) {
      if (shape == 1) launch_stream<8, 2, 1, EPI, 7>(g, s);   // 128 x 224 tiles
      else launch_stream<16, 2, 1, EPI, 7>(g, s);             // 256 x 224 tiles
      return;
    }
  }
  switch (shape) {
    case 0: launch_stream<4, 2, 1, EPI, 4>(g, s); break;    // 64 x 128 tiles
    case 1: launch_stream<8, 2, 1, EPI, 4>(g, s); break;    // 128 x 128 tiles
    default: launch_stream<16, 2, 1, EPI, 4>(g, s); break;  // 256 x 128 tiles
  }
}
}  // namespace

// Tile shape and K split.  Every launch streams each weight byte from HBM
// once; the choices trade workgroup count (to keep the CUs streaming) against
// extra traffic:
//  * wide outputs (>= 256 column tiles, e.g. the LM head) with 65..256 rows
//    take 128- or 256-row tiles, so each weight strip is fetched once (at 256
//    rows measured 270 us against 330 us with four 64-row tiles per strip);
//  * everything else uses 64-row tiles: the M tiles of one strip run on the
//    same XCD and re-read it from that XCD's L2, plus, for narrow outputs, a
//    K split.  The split takes the most workgroups that still fit one per CU:
//    a CU that gets a second workgroup streams twice the bytes and holds up
//    the launch (measured at 64 rows: down projection 19 us with 13 splits,
//    260 workgroups; 14 us with 10).  It is capped so that the float32
//    partials (written, then read) move at most half as many bytes as the
//    weights at one M tile, as many at several (where each workgroup carries
//    more fixed cost per weight byte: 256 rows, o projection 17 us with 3
//    splits, 19 us with 2).
GemmPlan plan_gemm(int dtype, int epi, int M, int N, int K) {
  GemmPlan p{};
  if (dtype != GM_BF16 || M <= 0) return p;
  const int cols = 128;                             // weight rows per workgroup
  p.Nw = epi == EPI_SWIGLU ? 2 * N : N;
  p.n_tiles = p.Nw / cols;
  const int target = 256;                           // workgroups that keep every CU streaming
  // Every shape is 128 columns wide, so tile statistics (kStatCols columns per workgroup)
  // take any of them.  Past 256 rows the M tiles already fill the chip, and taller tiles
  // cut the L2 re-reads of each weight strip (M / BM of them): 256-row tiles, except
  // 128-row ones for outputs of 128..255 column tiles, whose 256-row launch leaves 2.4
  // workgroups per CU (measured at 1024 rows: QKV, O, down and the MTP projection fastest
  // at 256 rows, gate/up at 128).
  if (M > 256) p.shape = (p.n_tiles >= 128 && p.n_tiles < target) ? 1 : 2;
  else p.shape = (M > 64 && p.n_tiles >= target) ? (M <= 128 ? 1 : 2) : 0;
  const int BM = p.shape == 2 ? 256 : p.shape == 1 ? 128 : 64;
  const int ITER = 8;                               // k32 steps per unrolled iteration (see kernel)
  p.m_tiles = (M + BM - 1) / BM;
  p.k_iters = K / (ITER * 32);
  int splits = target / (p.n_tiles * p.m_tiles);
  // 2 * S * M * Nw * 4 <= Nw * K * 2 / 2 (one M tile), <= Nw * K * 2 (several), and up to
  // 4 Nw * K * 2 past 256 rows, where the weights are re-read from L2 by every M tile anyway
  // (1024 rows, O projection: 33 us with 3 splits, 47 us unsplit)
  const int cap = M > 256 ? K / M : p.m_tiles > 1 ? K / (4 * M) : K / (8 * M);
  if (splits > cap) splits = cap;
  if (splits > p.k_iters) splits = p.k_iters;
  if (splits < 1 || epi == EPI_STATS) splits = 1;   // tile statistics need whole dot products
  p.splits = splits;
  p.part_bytes = splits > 1 ? (size_t)splits * M * p.Nw * sizeof(float) : 0;
  // Wide outputs at 128- and 256-row tiles with no K split take seven compute waves and
  // 224-column tiles: two waves per SIMD overlap one's LDS fragment reads with the other's
  // MFMAs, and a workgroup re-reads its activations for 224 columns instead of 128
  // (measured on the LM head, V 151936, at 96 / 128 / 200 / 256 rows: 176 / 183 / 249 /
  // 258 us against 187 / 196 / 271 / 280 us with four).
  p.cw = 4;
  if (p.shape != 0 && splits == 1 && p.n_tiles >= target &&
      (epi == EPI_STORE_F32 || epi == EPI_ADD_F32 || epi == EPI_STORE_ACT)) {
    p.cw = 7;
    p.n_tiles = (p.Nw + 7 * cols / 4 - 1) / (7 * cols / 4);
  }
  // SwiGLU outputs (gate/up) of 128..255 column tiles past 64 rows, one K split: the tile
  // shapes measured fastest on the Qwen3-4B gate/up (19456 weight rows, K 2560), against
  // the rules above: 96 / 128 rows, 128-row tiles: 31 / 34 us against 37 / 40; 256 rows,
  // 128 x 224 tiles: 43 against 53; 512 rows, 256 x 224: 69 against 83; 1024 rows,
  // 128 x 224: 127 against 138 (160 and 192 rows: 38-39 us either way).  With two
  // 128-row M tiles, 160-column tiles (five compute waves) where they still fit one
  // workgroup per CU: each CU streams fewer weight bytes per activation read (256 rows,
  // 244 workgroups: 43.9 us against 46.9 with 128 x 224 and 45.1 with 128 x 192).
  if (epi == EPI_SWIGLU && M > 64 && p.n_tiles >= 128 && p.n_tiles < target) {
    const bool tall = M > 384 && M <= 768;
    p.shape = tall ? 2 : 1;
    p.m_tiles = tall ? (M + 255) / 256 : (M + 127) / 128;
    p.splits = 1;
    p.part_bytes = 0;
    if (M > 128) {
      p.cw = 7;
      p.n_tiles = (p.Nw + 7 * cols / 4 - 1) / (7 * cols / 4);
      const int n5 = (p.Nw + 5 * cols / 4 - 1) / (5 * cols / 4);
      if (p.shape == 1 && p.m_tiles == 2 && 2 * n5 <= target) {   // the five-wave tiles are 128 rows tall
        p.cw = 5;
        p.n_tiles = n5;
      }
    }
  }
  return p;
}

// Tile geometry of the LM head's softmax statistics at M rows: the strip-range
// kernel's waves (bf16, M <= 64), else tiles of 8 strips (128 ids).
TileGeom plan_lm_head(int dtype, int M, int V, int K, bool *strips_kernel) {
  if (strips_kernel) *strips_kernel = false;
  if (dtype != GM_BF16 || M > 64 || V % kStripIds || K % (32 * kLmChunk)) return fixed_tiles(V);
  const int S = V / kStripIds;
  int waves = lm_resident_waves();
  if (waves > S) waves = S;
  if (waves < (S + kLmStrips - 1) / kLmStrips) waves = (S + kLmStrips - 1) / kLmStrips;
  if (waves > kMaxTiles) return fixed_tiles(V);
  if (strips_kernel) *strips_kernel = true;
  return TileGeom{S, waves};
}

int launch_gemm(const char *name, int dtype, int epi, int M, int N, int K, const void *X, int ldx, const void *W,
                void *Y, long ldy, float *part, hipStream_t s, RowStat *tile_stats, float inv_t, bool defer_reduce) {
  if (M <= 0) return 1;
  if (dtype == GM_BF16 && epi == EPI_STATS) {
    bool strips = false;
    const TileGeom geo = plan_lm_head(dtype, M, N, K, &strips);
    if (strips) {
      GemmL l{(const uint16_t *)X, (const uint16_t *)W, (float *)Y, ldy, M, K, ldx, geo, tile_stats, inv_t};
      TraceScope ts(name, s);
      hipLaunchKernelGGL(lm_strips_kernel<EPI_STATS>, dim3((geo.tiles + 3) / 4), dim3(256), 0, s, l);
      return 1;
    }
  }
  if (dtype == GM_BF16) {
    const GemmPlan p = plan_gemm(dtype, epi, M, N, K);
    GemmS g{(const uint16_t *)X, (const uint16_t *)W, Y, part, ldy, M, N, K, ldx, p.Nw, p.n_tiles, p.m_tiles,
            p.splits, p.k_iters, tile_stats, inv_t};
    {
      TraceScope ts(name, s);
      switch (epi) {
        case EPI_STORE_F32: launch_stream_shape<EPI_STORE_F32>(p.shape, p.cw, g, s); break;
        case EPI_ADD_F32: launch_stream_shape<EPI_ADD_F32>(p.shape, p.cw, g, s); break;
        case EPI_STORE_ACT: launch_stream_shape<EPI_STORE_ACT>(p.shape, p.cw, g, s); break;
        case EPI_SWIGLU: launch_stream_shape<EPI_SWIGLU>(p.shape, p.cw, g, s); break;
        case EPI_STATS: launch_stream_shape<EPI_STATS>(p.shape, p.cw, g, s); break;
      }
    }
    if (p.splits > 1 && defer_reduce) return p.splits;
    if (p.splits > 1) {
      TraceScope ts("gemm_split_reduce", s);
      const long total = (long)M * (N / 4);
      const int blocks = (int)((total + 255) / 256 < 2048 ? (total + 255) / 256 : 2048);
      switch (epi) {
        case EPI_STORE_F32: hipLaunchKernelGGL(gemm_reduce_kernel<EPI_STORE_F32>, dim3(blocks), dim3(256), 0, s, g); break;
        case EPI_ADD_F32: hipLaunchKernelGGL(gemm_reduce_kernel<EPI_ADD_F32>, dim3(blocks), dim3(256), 0, s, g); break;
        case EPI_STORE_ACT: hipLaunchKernelGGL(gemm_reduce_kernel<EPI_STORE_ACT>, dim3(blocks), dim3(256), 0, s, g); break;
        case EPI_SWIGLU: hipLaunchKernelGGL(gemm_reduce_kernel<EPI_SWIGLU>, dim3(blocks), dim3(256), 0, s, g); break;
      }
    }
    return 1;
  } else {
    GemmF g{(const float *)X, (const float *)W, (float *)Y, ldy, M, N, K, ldx};
    const dim3 grid((N + 63) / 64, (M + 15) / 16), block(256);
    if (epi == EPI_STATS) {     // no fused epilogue on this path: a pass over the output rows
      {
        TraceScope ts(name, s);
        hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, block, 0, s, g);
      }
      launch_tile_stats((const float *)Y, ldy, M, N, inv_t, plan_lm_head(dtype, M, N, K), tile_stats, s);
      return 1;
    }
    TraceScope ts(name, s);
    switch (epi) {
      case EPI_STORE_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, block, 0, s, g); break;
      case EPI_ADD_F32: hipLaunchKernelGGL(gemm_f32_kernel<EPI_ADD_F32>, grid, block, 0, s, g); break;
      case EPI_STORE_ACT: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_ACT>, grid, block, 0, s, g); break;
      case EPI_SWIGLU: hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, g); break;
    }
  }
  return 1;
}

void launch_reduce_norm(int dtype, int epi, int M, int N, int splits, const float *part, float *Y, const void *norm_w,
                        float eps, void *out, hipStream_t s) {
  if (M <= 0) return;
  TraceScope ts("reduce_norm", s);
  int threads = ((N / 4 + 63) / 64) * 64;   // one float4 column group per thread when N <= 4096
  if (threads > 1024) threads = 1024;
  const dim3 grid(M), block(threads);
  const size_t lds = (size_t)N * sizeof(float);
  if (dtype == GM_BF16) {
    if (epi == EPI_ADD_F32)
      hipLaunchKernelGGL((reduce_norm_kernel<bf16, EPI_ADD_F32>), grid, block, lds, s, M, N, splits, part, Y,
                         (const bf16 *)norm_w, eps, (bf16 *)out);
    else
      hipLaunchKernelGGL((reduce_norm_kernel<bf16, EPI_STORE_F32>), grid, block, lds, s, M, N, splits, part, Y,
                         (const bf16 *)norm_w, eps, (bf16 *)out);
  } else {
    if (epi == EPI_ADD_F32)
      hipLaunchKernelGGL((reduce_norm_kernel<float, EPI_ADD_F32>), grid, block, lds, s, M, N, splits, part, Y,
                         (const float *)norm_w, eps, (float *)out);
    else
      hipLaunchKernelGGL((reduce_norm_kernel<float, EPI_STORE_F32>), grid, block, lds, s, M, N, splits, part, Y,
                         (const float *)norm_w, eps, (float *)out);
  }
}

}  // namespace gm
