// Verify attention (Sec. 3.1, Eq. verification-context): the query at block
// position i of sequence b attends causally to cache positions 0 .. m_b + i.
//
// bf16 path.  Work partition: the 16-token tiles of all sequences, laid end
// to end, are cut into P equal ranges, P = the number of workgroups the chip
// holds at once; workgroup (p, head group) takes range p for its heads, so
// every wave streams the same number of tiles whatever the length mix, and a
// range that crosses sequences yields one partial per sequence.  A combine
// kernel merges the partials of each sequence.  One 64-lane wave per KV head and
// one or two 16-row query tiles (two: the k = 7 block, 32 rows, streams each KV
// tile once for both):
//  * GQA packing: the (n_heads / n_kv_heads) query heads of one KV head times
//    the block rows form the rows of 16-row matrix-core tiles, so each K/V
//    byte streamed from HBM serves every query that reads it;
//  * S^T = K Q^T on v_mfma_f32_16x16x32_bf16; the score tile comes out in the
//    operand layout of the P V product, so P never leaves registers;
//  * P is split into bf16 hi + lo parts that ride in the two halves of the
//    32-deep reduction of one v_mfma_f32_16x16x32_bf16 (V repeated), so the
//    weights keep ~16 mantissa bits at the cost of a single product;
//  * the KV pages are stored pre-swizzled (gm.h), so every 16-byte-per-lane
//    load reads 1 KiB contiguous straight into operand registers;
//  * K/V tiles stream through a ring of register buffers, every load
//    unconditional, so kAttnRing - 1 tiles are always in flight;
//  * tiles wholly inside every query's causal window skip the mask; the
//    online softmax (exp2 domain) rescales only when a running max grows by
//    more than 2^kLazyLog2, so most tiles need no rescale.
// float32 path: a plain wave-per-(row, head) kernel.
#include <atomic>

#include "common.h"
#include "forward.h"

namespace gm {

namespace {
constexpr int kAttnWavesPerGroup = 4;   // waves per workgroup (KV heads x query row tiles)
// Dynamic LDS a workgroup reserves (unused) so that a CU holds one at a time:
// with two per CU the older one wins the SIMD arbitration, finishes early and
// leaves the CU half idle for the rest of the launch (measured); one per CU
// keeps all ranges in step.
constexpr int kAttnLdsReserve = 84 * 1024;
constexpr int kAttnRing = 3;            // K/V register buffers per wave
constexpr float kLazyLog2 = 8.f;        // rescale threshold of the running max (log2 units)

struct AttnK {
  const uint16_t *kp, *vp;
  const int32_t *bt, *base, *blen;
  const uint16_t *q;
  float *part_o;        // [P + B slots][n_kv][rows_pad][128]
  float2 *part_ml;      // [P + B slots][n_kv][rows_pad]
  int32_t *cum;         // [B + 1] tiles before sequence b (written by workgroup (0, 0))
  int32_t *dev_err;
  int B, base_off, blen_add, R, G, n_heads, n_kv, page_size, max_pages, num_pages, rows_pad;
  int parts, heads_per_group, row_tiles, waves_per_head;
  float scale_log2;
};

__device__ __forceinline__ int block_rows(const int32_t *blen, int add, int b, int R) {
  if (!blen) return R;
  const int n = blen[b] + add;
  return n < 0 ? 0 : (n > R ? R : n);
}

// 16-token tiles of sequence b: its context is base + base_off + valid block rows
__device__ __forceinline__ int seq_tiles(const AttnK &a, int b) {
  const int L = a.base[b] + a.base_off + block_rows(a.blen, a.blen_add, b, a.R);
  return L > 0 ? (L + 15) >> 4 : 0;
}

// first tile of range p when TT tiles are cut into P ranges
__device__ __forceinline__ int part_begin(int p, int TT, int P) { return (int)((long)p * TT / P); }

// exclusive block-wide prefix sum (blockDim.x a multiple of 64, <= 1024); *total gets the sum
__device__ __forceinline__ int block_excl_scan(int v, int *sh, int *total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  int off = 0, t = 0;
  for (int i = 0; i < nw; ++i) {
    const int u = sh[i];
    off += i < wid ? u : 0;
    t += u;
  }
  *total = t;
  return off + x - v;
}

__device__ __forceinline__ uint32_t zero_half(uint32_t v, int hi) { return hi ? (v & 0x0000ffffu) : (v & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {   // round to nearest even
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2_t{a, b}, bf16x2_t));
}

template <bool STREAM>
__device__ __forceinline__ uint4 load_kv(const uint16_t *p) {
  if (STREAM) return load_nt(p);
  return *reinterpret_cast<const uint4 *>(p);
}

struct TileBuf {
  uint4 k[4], v[4];
};

// One 16-token tile for the RT 16-row query tiles of a wave: S^T = K Q^T, online softmax,
// O^T += V^T (P_hi + P_lo).  MASK: apply the causal window (token < vis) and keep tokens
// past the context (t >= L, whose slots may hold anything) out of P V.  Each step runs
// for every query tile before the next, so the tiles' dependency chains interleave and
// the V operands of P V are formed once for all of them; each tile's arithmetic is the
// same as on its own.
template <bool MASK, int RT>
__device__ __forceinline__ void attn_tiles(int tb, int L, int g, float scale_log2, TileBuf &t,
                                           const bf16x8_t (&qf)[RT][4], const int (&vis)[RT], float (&m)[RT],
                                           float (&l)[RT], floatx4_t (&O)[RT][8]) {
  if (MASK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (tb + 4 * g + e >= L) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          if (e < 2) { t.v[p].x = zero_half(t.v[p].x, e); t.v[p].z = zero_half(t.v[p].z, e); }
          else { t.v[p].y = zero_half(t.v[p].y, e - 2); t.v[p].w = zero_half(t.v[p].w, e - 2); }
        }
      }
    }
  }
  floatx4_t S[RT];
#pragma unroll
  for (int u = 0; u < RT; ++u) S[u] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ii = 0; ii < 4; ++ii)
#pragma unroll
    for (int u = 0; u < RT; ++u)
      S[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(t.k[ii]), qf[u][ii], S[u], 0, 0, 0);
  float s[RT][4], tmax[RT];
#pragma unroll
  for (int u = 0; u < RT; ++u) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      s[u][r] = S[u][r] * scale_log2;
      if (MASK && tb + 4 * g + r >= vis[u]) s[u][r] = -INFINITY;
    }
    tmax[u] = fmaxf(fmaxf(s[u][0], s[u][1]), fmaxf(s[u][2], s[u][3]));
  }
#pragma unroll
  for (int u = 0; u < RT; ++u) tmax[u] = fmaxf(tmax[u], __shfl_xor(tmax[u], 16, kWave));
#pragma unroll
  for (int u = 0; u < RT; ++u) tmax[u] = fmaxf(tmax[u], __shfl_xor(tmax[u], 32, kWave));
  // Each row decides for itself (m = -inf and a finite score also count as growth);
  // rows that did not grow keep alpha = 1 exactly, so a row's result never depends
  // on the other rows of the tile.  The branch only skips tiles where no row grew.
#pragma unroll
  for (int u = 0; u < RT; ++u) {
    const bool up = tmax[u] > m[u] + kLazyLog2;
    if (__any(up)) {
      const float mn = up ? fmaxf(m[u], tmax[u]) : m[u];
      const float alpha = (!up || mn == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m[u] - mn);
      l[u] *= alpha;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) O[u][mm] *= alpha;
      m[u] = mn;
    }
  }
  // s <= m + kLazyLog2 here, so p <= 2^kLazyLog2
  bf16x8_t pb[RT];
#pragma unroll
  for (int u = 0; u < RT; ++u) {
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      p[r] = __builtin_amdgcn_exp2f(s[u][r] - m[u]);
      if (MASK && s[u][r] == -INFINITY) p[r] = 0.f;
      l[u] += p[r];
    }
    const uint32_t h01 = pack_bf16(p[0], p[1]), h23 = pack_bf16(p[2], p[3]);
    const uint32_t l01 = pack_bf16(p[0] - __uint_as_float(h01 << 16), p[1] - __uint_as_float(h01 & 0xffff0000u));
    const uint32_t l23 = pack_bf16(p[2] - __uint_as_float(h23 << 16), p[3] - __uint_as_float(h23 & 0xffff0000u));
    pb[u] = as_bf16x8(make_uint4(h01, h23, l01, l23));
  }
#pragma unroll
  for (int mm = 0; mm < 8; ++mm) {
    const uint4 &v4 = t.v[mm >> 1];
    const uint4 va = (mm & 1) ? make_uint4(v4.z, v4.w, v4.z, v4.w) : make_uint4(v4.x, v4.y, v4.x, v4.y);
#pragma unroll
    for (int u = 0; u < RT; ++u) O[u][mm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(va), pb[u], O[u][mm], 0, 0, 0);
  }
}

// RT: 16-row query tiles per wave.  A wave streams the KV tiles of its head once and
// runs the score / softmax / PV products of its RT query tiles on each of them; the
// waves_per_head = row_tiles / RT waves of one head split its query tiles.
// STREAM: every KV tile has exactly one reader (one wave per KV head), so its loads are
// marked non-temporal and do not displace the lines other waves re-read; where two waves
// read the same tiles the second read is meant to hit the cache (measured: non-temporal
// loads there cost 20%).
template <bool STREAM, int RT>
__global__ __launch_bounds__(64 * kAttnWavesPerGroup) void attn_mfma_kernel(AttnK a) {
  const int part = blockIdx.x, grp = blockIdx.y;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index, uniform per wave
  const int lane = threadIdx.x & 63, j = lane & 15, g = lane >> 4;
  const int kvh = grp * a.heads_per_group + w / a.waves_per_head, rt0 = (w % a.waves_per_head) * RT;
  const bool wave_ok = kvh < a.n_kv;
  const int rows = a.G * a.R;

  __shared__ int scan_sh[16];
  __shared__ int page_sh[kAttnMaxSplitPages];
  __shared__ int bad_sh, first_sh, first_cum_sh;

  // Total tiles TT, then the first sequence of this workgroup's range [s, e): a chunked
  // block scan over the sequences (workgroup (0, 0) also stores the prefix sums for the
  // combine).  Every workgroup computes the same sums.
  // (a batch that fits one block needs a single scan)
  const bool one_chunk = a.B <= (int)blockDim.x;
  int TT = 0, T1 = 0, cb1 = 0;
  if (one_chunk) {
    T1 = (int)threadIdx.x < a.B ? seq_tiles(a, threadIdx.x) : 0;
    cb1 = block_excl_scan(T1, scan_sh, &TT);
  } else {
    for (int c = 0; c < a.B; c += blockDim.x) {
      const int b = c + threadIdx.x;
      int tot;
      block_excl_scan(b < a.B ? seq_tiles(a, b) : 0, scan_sh, &tot);
      TT += tot;
    }
  }
  const int s = part_begin(part, TT, a.parts), e = part_begin(part + 1, TT, a.parts);
  if (threadIdx.x == 0) first_sh = a.B;
  __syncthreads();
  const bool writer = part == 0 && grp == 0;
  auto visit = [&](int b, int T, int cb) {
    if (b >= a.B) return;
    if (writer) a.cum[b] = cb;
    if (T > 0 && cb <= s && s < cb + T) {   // the sequence holding tile s (unique)
      first_sh = b;
      first_cum_sh = cb;
    }
  };
  if (one_chunk) {
    visit(threadIdx.x, T1, cb1);
  } else {
    int run = 0;
    for (int c = 0; c < a.B; c += blockDim.x) {
      const int b = c + threadIdx.x;
      const int T = b < a.B ? seq_tiles(a, b) : 0;
      int tot;
      const int cb = run + block_excl_scan(T, scan_sh, &tot);
      visit(b, T, cb);
      run += tot;
    }
  }
  if (writer && threadIdx.x == 0) a.cum[a.B] = TT;
  __syncthreads();
  if (s >= e) return;   // an empty range (fewer tiles than workgroups)
  int b = __builtin_amdgcn_readfirstlane(first_sh);
  int cb = __builtin_amdgcn_readfirstlane(first_cum_sh);
  const long head_off = (long)kvh * a.page_size * 128;

  for (; b < a.B && cb < e; ++b) {
    const int m0 = __builtin_amdgcn_readfirstlane(a.base[b] + a.base_off);
    const int blen = __builtin_amdgcn_readfirstlane(block_rows(a.blen, a.blen_add, b, a.R));
    const int L = m0 + blen;
    const int T = L > 0 ? (L + 15) >> 4 : 0;
    const int ta = max(s, cb) - cb, tz = min(e, cb + T) - cb;
    cb += T;
    if (ta >= tz) continue;
    const int t0 = 16 * ta, t1 = min(L, 16 * tz);

    // The pages of [t0, t1), looked up once into LDS: in the loop a lookup is then an LDS
    // read, whose counter is separate from the KV loads', so no wait drains the prefetch.
    // A page outside the pool ends the segment before its first token (and is reported).
    const int p0 = t0 / a.page_size;
    int np = (t1 - 1) / a.page_size - p0 + 1;
    __syncthreads();   // the previous segment is done with page_sh
    if (threadIdx.x == 0) bad_sh = np;
    if (np > kAttnMaxSplitPages) {   // lengths beyond the planned maximum: stop at the table's end
      np = kAttnMaxSplitPages;
      if (threadIdx.x == 0) bad_sh = np;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < np; i += blockDim.x) {
      const int pi = p0 + i;
      const int page = pi < a.max_pages ? a.bt[(long)b * a.max_pages + pi] : -1;
      page_sh[i] = page;
      if (page < 0 || page >= a.num_pages) atomicMin(&bad_sh, i);
    }
    __syncthreads();
    if (!wave_ok) continue;   // spare waves of the last head group (they still join the barriers)
    int tend = t1;
    const int bad = __builtin_amdgcn_readfirstlane(bad_sh);
    if (bad < (t1 - 1) / a.page_size - p0 + 1) {
      raise_dev_err(a.dev_err, GM_DEVERR_PAGE);
      tend = max(t0, (p0 + bad) * a.page_size);
    }

    bf16x8_t qf[RT][4];
    int vis[RT];
    float m[RT], l[RT];
    floatx4_t O[RT][8];
#pragma unroll
    for (int u = 0; u < RT; ++u) {
      const int r = (rt0 + u) * 16 + j;
      vis[u] = 0;
      if (r < rows) {
        const int hl = r / a.R, i = r % a.R;
        const uint16_t *qrow = a.q + (((long)b * a.R + i) * a.n_heads + kvh * a.G + hl) * 128;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) qf[u][ii] = as_bf16x8(*reinterpret_cast<const uint4 *>(qrow + 32 * ii + 8 * g));
        vis[u] = i < blen ? m0 + i + 1 : 0;
      } else {
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) qf[u][ii] = as_bf16x8(make_uint4(0, 0, 0, 0));
      }
      m[u] = -INFINITY;
      l[u] = 0.f;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) O[u][mm] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    }

    auto tile_off = [&](int tb) -> long {
      const int page = page_sh[tb / a.page_size - p0];
      return (long)page * a.n_kv * a.page_size * 128 + head_off + (long)(tb % a.page_size) * 128;
    };
    auto load_tile = [&](long off, TileBuf &t) {
#pragma unroll
      for (int i = 0; i < 4; ++i) t.k[i] = load_kv<STREAM>(a.kp + off + i * 512 + lane * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i) t.v[i] = load_kv<STREAM>(a.vp + off + i * 512 + lane * 8);
    };

    // Tiles [t0, t0 + 16 n) lie below position m0 + 1, inside the window of every valid
    // query row, and inside the context: no mask.  The rest (the causal diagonal and the
    // partial tile at the end of the context) take the mask; the mask zeroes the V entries
    // past the context in place.  Rows that are not valid queries (past the block, or
    // padding) compute finite values nobody reads.  All nt tiles stream through the ring,
    // the masked ones too, so the segment's end is as pipelined as its body.
    const int nm_end = min(tend, m0 + 1);
    const int n = __builtin_amdgcn_readfirstlane(nm_end > t0 ? (nm_end - t0) / 16 : 0);
    const int nt = __builtin_amdgcn_readfirstlane(tend > t0 ? (tend - t0 + 15) / 16 : 0);
    auto consume = [&](int i, TileBuf &t) {
      if (i < n) attn_tiles<false, RT>(t0 + 16 * i, L, g, a.scale_log2, t, qf, vis, m, l, O);
      else attn_tiles<true, RT>(t0 + 16 * i, L, g, a.scale_log2, t, qf, vis, m, l, O);
    };
    if (nt > 0) {
      // whole turns of the ring run unguarded (one straight path, so every wait counts
      // exactly the loads still in flight); the last < kAttnRing tiles are already in
      // the ring when the loop ends
      TileBuf ring[kAttnRing];
      const int n_pipe = nt - nt % kAttnRing;
#pragma unroll
      for (int d = 0; d < kAttnRing - 1; ++d) load_tile(tile_off(t0 + 16 * min(d, nt - 1)), ring[d]);
      for (int i = 0; i < n_pipe; i += kAttnRing) {
#pragma unroll
        for (int d = 0; d < kAttnRing; ++d) {
          // refill the buffer consumed last step (a re-read of the last tile near the end);
          // the scheduling barriers keep each refill after the step that frees its buffer,
          // so the ring keeps fixed registers and no copy waits on a load in flight
          __builtin_amdgcn_sched_barrier(0);
          load_tile(tile_off(t0 + 16 * min(i + d + kAttnRing - 1, nt - 1)), ring[(d + kAttnRing - 1) % kAttnRing]);
          __builtin_amdgcn_sched_barrier(0);
          consume(i + d, ring[d]);
        }
      }
#pragma unroll
      for (int d = 0; d < kAttnRing - 1; ++d)
        if (n_pipe + d < nt) consume(n_pipe + d, ring[d]);
    }

#pragma unroll
    for (int u = 0; u < RT; ++u) {
      float lu = l[u];
      lu += __shfl_xor(lu, 16, kWave);
      lu += __shfl_xor(lu, 32, kWave);
      const long prow = ((long)(part + b) * a.n_kv + kvh) * a.rows_pad + (rt0 + u) * 16 + j;
      if (g == 0) a.part_ml[prow] = make_float2(m[u], lu);
      float *po = a.part_o + prow * 128;
#pragma unroll
      for (int mm = 0; mm < 8; ++mm)
        *reinterpret_cast<float4 *>(po + 16 * mm + 4 * g) =
            make_float4(O[u][mm][0], O[u][mm][1], O[u][mm][2], O[u][mm][3]);
    }
  }
}

// Merge the partials of sequence b: the ranges that hold its tiles are parts
// p_first .. p_last (empty ranges among them wrote nothing and are skipped);
// the partial of (part p, sequence b) sits in slot p + b.  One thread per
// (KV head, row, four channels); the partials are read kCombineBatch at a
// time with every load issued before the first use, and merged in one pass.
constexpr int kCombineBatch = 8;

__global__ __launch_bounds__(256) void attn_combine_kernel(AttnK a, uint16_t *__restrict__ out) {
  const int b = blockIdx.y;
  const int rows = a.G * a.R;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= a.n_kv * rows * 32) return;
  const int d = (idx & 31) * 4, r = (idx >> 5) % rows, kvh = (idx >> 5) / rows;
  const int hl = r / a.R, i = r % a.R;
  const int blen = block_rows(a.blen, a.blen_add, b, a.R);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < blen) {
    const int TT = a.cum[a.B], cb = a.cum[b], T = a.cum[b + 1] - cb;
    const int P = a.parts;
    if (T > 0) {
      int pf = (int)(((long)(cb + 1) * P - 1) / TT), pl = (int)(((long)(cb + T) * P - 1) / TT);
      pf = pf < P - 1 ? pf : P - 1;
      pl = pl < P - 1 ? pl : P - 1;
      float M = -INFINITY, den = 0.f;
      float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int p0 = pf; p0 <= pl; p0 += kCombineBatch) {
        float2 ml[kCombineBatch];
        float4 o[kCombineBatch];
#pragma unroll
        for (int u = 0; u < kCombineBatch; ++u) {
          const int p = min(p0 + u, pl);
          const long pr = ((long)(p + b) * a.n_kv + kvh) * a.rows_pad + r;
          ml[u] = a.part_ml[pr];
          o[u] = *reinterpret_cast<const float4 *>(a.part_o + pr * 128 + d);
        }
#pragma unroll
        for (int u = 0; u < kCombineBatch; ++u) {
          const int p = p0 + u;
          if (p > pl || part_begin(p, TT, P) == part_begin(p + 1, TT, P) || ml[u].x == -INFINITY) continue;
          const float mn = fmaxf(M, ml[u].x);
          const float sc = __builtin_amdgcn_exp2f(M - mn), w = __builtin_amdgcn_exp2f(ml[u].x - mn);   // M = -inf: sc = 0
          den = den * sc + ml[u].y * w;
          num.x = num.x * sc + o[u].x * w;
          num.y = num.y * sc + o[u].y * w;
          num.z = num.z * sc + o[u].z * w;
          num.w = num.w * sc + o[u].w * w;
          M = mn;
        }
      }
      if (M != -INFINITY) {
        const float inv = 1.f / den;
        v = make_float4(num.x * inv, num.y * inv, num.z * inv, num.w * inv);
      }
    }
  }
  const uint2 packed = make_uint2(f32_to_bf16(v.x) | (uint32_t(f32_to_bf16(v.y)) << 16),
                                  f32_to_bf16(v.z) | (uint32_t(f32_to_bf16(v.w)) << 16));
  *reinterpret_cast<uint2 *>(out + (((long)b * a.R + i) * a.n_heads + kvh * a.G + hl) * 128 + d) = packed;
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

// Geometry of the bf16 launch: row tiles per KV head, heads per workgroup, groups.
struct AttnGeom {
  int row_tiles, rt_per_wave, waves_per_head, heads_per_group, groups, block;
};
AttnGeom attn_geom(const gm_model_config &cfg, int rows_pad) {
  AttnGeom g;
  g.row_tiles = rows_pad / 16;
  g.rt_per_wave = g.row_tiles >= 2 ? 2 : 1;
  g.waves_per_head = g.row_tiles / g.rt_per_wave;
  g.heads_per_group = kAttnWavesPerGroup / g.waves_per_head;
  if (g.heads_per_group > cfg.n_kv_heads) g.heads_per_group = cfg.n_kv_heads;
  if (g.heads_per_group < 1) g.heads_per_group = 1;
  g.groups = (cfg.n_kv_heads + g.heads_per_group - 1) / g.heads_per_group;
  g.block = 64 * g.heads_per_group * g.waves_per_head;
  return g;
}

// Workgroups of `block` threads that one device holds at once (queried once per
// block size and device; a fixed guess when no device answers).  The LDS
// reservation makes this one per CU.
int resident_groups(int block) {
  static std::atomic<int> cache[16][kAttnWavesPerGroup + 1];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 256;
  const int wv = block / 64;
  int v = cache[dev][wv].load();
  if (v > 0) return v;
  int per_cu = 0, cus = 0;
  const void *kernels[] = {(const void *)attn_mfma_kernel<true, 1>, (const void *)attn_mfma_kernel<true, 2>,
                           (const void *)attn_mfma_kernel<false, 2>};
  bool ok = true;
  for (const void *f : kernels)
    ok = ok && hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, kAttnLdsReserve) == hipSuccess;
  if (!ok || hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_mfma_kernel<true, 2>, block, kAttnLdsReserve) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || per_cu < 1 || cus < 1) {
    (void)hipGetLastError();
    return 256;
  }
  v = per_cu * cus;
  cache[dev][wv].store(v);
  return v;
}
}  // namespace

AttnPlan plan_attention(const gm_model_config &cfg, int B, int R, int max_ctx) {
  AttnPlan p{};
  const int G = cfg.n_heads / cfg.n_kv_heads;
  const int rows = G * R;
  const int nt = rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
  p.rows_pad = nt * 16;
  if (cfg.dtype != GM_BF16) return p;
  const AttnGeom g = attn_geom(cfg, p.rows_pad);
  long parts = resident_groups(g.block) / g.groups;
  // bound the tiles of one range so its pages fit the workgroup's page table
  const long tiles_max = (long)B * (((long)max_ctx + R + 15) / 16);
  const long need = (tiles_max + kAttnMaxSplitTokens / 16 - 1) / (kAttnMaxSplitTokens / 16);
  if (parts < need) parts = need;
  if (parts < 1) parts = 1;
  p.parts = (int)parts;
  Carve c;
  const size_t n = (size_t)(p.parts + B) * cfg.n_kv_heads * p.rows_pad;
  p.part_o = c.take(n * 128 * sizeof(float));
  p.part_ml = c.take(n * sizeof(float2));
  p.cum = c.take((size_t)(B + 1) * sizeof(int32_t));
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
    gm_model_config cfg{};
    cfg.n_kv_heads = a.n_kv;
    const AttnGeom geo = attn_geom(cfg, p.rows_pad);
    AttnK k{};
    k.kp = (const uint16_t *)a.k_pages;
    k.vp = (const uint16_t *)a.v_pages;
    k.bt = a.block_table;
    k.base = a.base_lens;
    k.blen = a.blk_len;
    k.q = (const uint16_t *)a.q;
    k.part_o = (float *)(ws + p.part_o);
    k.part_ml = (float2 *)(ws + p.part_ml);
    k.cum = (int32_t *)(ws + p.cum);
    k.dev_err = a.dev_err;
    k.B = a.B;
    k.base_off = a.base_off;
    k.blen_add = a.blk_len_add;
    k.R = a.R;
    k.G = G;
    k.n_heads = a.n_heads;
    k.n_kv = a.n_kv;
    k.page_size = a.page_size;
    k.max_pages = a.max_pages;
    k.num_pages = a.num_pages;
    k.rows_pad = p.rows_pad;
    k.parts = p.parts;
    k.heads_per_group = geo.heads_per_group;
    k.row_tiles = geo.row_tiles;
    k.waves_per_head = geo.waves_per_head;
    k.scale_log2 = a.scale * 1.4426950408889634f;
    {
      TraceScope ts(a.trace, s);
      const dim3 grid(p.parts, geo.groups), block(geo.block);
      if (geo.rt_per_wave == 1)
        hipLaunchKernelGGL((attn_mfma_kernel<true, 1>), grid, block, kAttnLdsReserve, s, k);
      else if (geo.waves_per_head == 1)
        hipLaunchKernelGGL((attn_mfma_kernel<true, 2>), grid, block, kAttnLdsReserve, s, k);
      else
        hipLaunchKernelGGL((attn_mfma_kernel<false, 2>), grid, block, kAttnLdsReserve, s, k);
    }
    TraceScope ts(a.trace_combine, s);
    const int items = a.n_kv * G * a.R * 32;
    hipLaunchKernelGGL(attn_combine_kernel, dim3((items + 255) / 256, a.B), dim3(256), 0, s, k, (uint16_t *)a.out);
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
