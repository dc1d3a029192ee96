// Score pass of LAST (arXiv 2607.27952, Sec. 3.3, Eq. 6-8) for gfx950.
//
// The attention row of the last query token is recomputed from q and the key
// cache instead of being read from a materialised P x P map (same numbers,
// O(P) instead of O(P^2) work per head). The row needs a softmax over the
// whole prefix while the keys are streamed in chunks, so the pass is split:
//
//   (no plan pass) every block finds the request it works on itself: a wave
//                     scans the per-request chunk (or slice) counts, 64
//                     requests at a time, up to the block's index. Batches of
//                     more than kScanMaxR requests run k_score_prefix first
//                     (one block: the count prefixes) and search those.
//   k_score_stream    one block per (layer, chunk of tokens). The chunk's key
//                     rows for all KV heads are one contiguous byte range,
//                     streamed once: 8 lanes cover one row with 16-byte loads
//                     (a wave reads 8 rows = 2 KB per instruction pair for
//                     Dh = 128 bf16). Each lane keeps one KV head for the whole
//                     block, so the query slices of that head's Hq/Hkv query
//                     heads stay in registers; bf16 dots use v_dot2_f32_bf16,
//                     fp32 dots use FMAs. A row's dot is reduced over its 8
//                     lanes with DPP and lane j of the row stores query head
//                     j's logit into the chunk's token-major LDS tile. Then
//                     all threads form, per head, the chunk's max m and the
//                     sums of exp(l - m) over every token (Z) and over the
//                     visual tokens (V), and copy the visual logits out.
//   k_score_partial   fallback for KV-head counts that do not divide 32: one
//                     block per (layer, chunk, KV head, query-head group), the
//                     chunk's logits staged in LDS.
//   k_score_merge     one wave per (request, layer, head) row: merges the
//                     row's chunk statistics into its max M and normaliser Z,
//                     and its share V / Z of the visual mass S = sum V / Z,
//                     which equals sum_i s_i (Eq. 8).
//   k_score_finalize  one block per slice of a request's visual tokens: S
//                     from the rows' shares, then
//                     s_i = sum_{l,h} exp(l_i - M) / Z   (Eq. 6-7), over S,
//                     so no second pass over s is needed.
//
// Every reduction has a fixed order, so results are bitwise reproducible.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 6;                  // row groups (8 rows each) in flight per wave

// Key rows are read exactly once: non-temporal loads stream them without
// displacing cache lines that other blocks still use (on this part a plain
// read stream reaches about 6.1 TB/s, a non-temporal one about 7.1 TB/s).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load(const void *p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
constexpr int64_t kWgBytes = 96 * 1024;     // key bytes per stream block
constexpr int kMaxChunk = 4096;             // tokens per chunk (fallback kernel), upper bound
constexpr int kLdsLogitFloats = 8192;
constexpr int kSliceTokens = 256;           // visual tokens per finalize block
constexpr int kMaxPairs = 4096;             // G * Hq handled by the finalize block
constexpr int kScanMaxR = 1024;             // larger batches search count prefixes instead

// Logits are kept in base-2 units (the softmax scale times log2 e, folded
// into the dot's one multiply), so that every exponential is exp2f: one
// v_exp_f32 plus the rescaling that keeps results below 2^-126 (which that
// instruction flushes) as denormals, as expf does, in about half of expf's
// instructions.

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

template <typename T, int DH>
struct RowShape {
  static constexpr int kBytes = DH * (int)sizeof(T);
  static constexpr int kNP = kBytes / 16 / 8;           // 16-byte pieces per lane per row
  static constexpr int kEP = 16 / (int)sizeof(T);       // elements per piece
  static constexpr int kElems = kNP * kEP;              // elements per lane per row
};

__device__ __forceinline__ void widen(const uint4 v, float *f, uint16_t) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
__device__ __forceinline__ void widen(const uint4 v, float *f, float) {
  f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b),
                                         c, false);
}

// Count prefixes for batches of more than kScanMaxR requests (one block):
// chunk_off[r] = sum over r' < r of ceil(P_r' / CH), slice_off likewise over
// ceil(N_r' / SL).
__global__ __launch_bounds__(kThreads) void k_score_prefix(
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ row_pos, int R, int CH, int SL, int32_t *__restrict__ chunk_off,
    int32_t *__restrict__ slice_off) {
  __shared__ int sh[kThreads / 64];
  int carry_c = 0, carry_s = 0;
  for (int base = 0; base < R; base += kThreads) {
    const int r = base + (int)threadIdx.x;
    int nc = 0, ns = 0;
    if (r < R) {
      const int P = row_pos ? row_pos[r] + 1 : cu_seqlens[r + 1] - cu_seqlens[r];
      const int N = cu_vis[r + 1] - cu_vis[r];
      nc = (P + CH - 1) / CH;
      ns = (N + SL - 1) / SL;
    }
    int tc, ts;
    const int pc = block_exclusive_scan(nc, sh, &tc) + carry_c;
    const int ps = block_exclusive_scan(ns, sh, &ts) + carry_s;
    if (r < R) {
      chunk_off[r] = pc;
      slice_off[r] = ps;
    }
    carry_c += tc;
    carry_s += ts;
  }
  if (threadIdx.x == 0) {
    chunk_off[R] = carry_c;
    slice_off[R] = carry_s;
  }
}

// Where a block's item lies. Items are numbered request by request: request r
// owns ceil(P_r / CH) chunks and ceil(N_r / SL) visual slices. Given a chunk
// index (by_slice false) or a slice index (by_slice true), finds the request r
// and the indices of its first chunk and first slice. With the prefixes of
// k_score_prefix (batches over kScanMaxR) a binary search; otherwise wave 0
// scans the counts 64 requests at a time. Every thread calls it; the result is
// block-uniform (through LDS; the function ends with a block barrier).
struct Where {
  int r, c0, s0;
};
__device__ Where locate(int64_t x, bool by_slice, int R, int CH, int SL, const int32_t *__restrict__ cu_seqlens,
                        const int32_t *__restrict__ cu_vis, const int32_t *__restrict__ row_pos,
                        const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ slice_off,
                        int *s_where) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    if (R > kScanMaxR) {
      if (lane == 0) {
        const int32_t *off = by_slice ? slice_off : chunk_off;
        int lo = 0, hi = R - 1;   // last r with off[r] <= x
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (off[mid] <= x) lo = mid; else hi = mid - 1;
        }
        s_where[0] = lo;
        s_where[1] = chunk_off[lo];
        s_where[2] = slice_off[lo];
      }
    } else {
      int base_c = 0, base_s = 0;
      for (int r0 = 0; r0 < R; r0 += 64) {
        const int r = r0 + lane;
        int nc = 0, ns = 0;
        if (r < R) {
          const int P = row_pos ? row_pos[r] + 1 : cu_seqlens[r + 1] - cu_seqlens[r];
          const int N = cu_vis[r + 1] - cu_vis[r];
          nc = (P + CH - 1) / CH;
          ns = (N + SL - 1) / SL;
        }
        int ic = nc, is = ns;   // inclusive scans over the lanes
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int yc = __shfl_up(ic, o), ys = __shfl_up(is, o);
          if (lane >= o) {
            ic += yc;
            is += ys;
          }
        }
        const int64_t end = (int64_t)(by_slice ? base_s + is : base_c + ic);
        const unsigned long long hit = __ballot(r < R && end > x);
        if (hit) {
          const int f = (int)__ffsll((long long)hit) - 1;
          if (lane == f) {
            s_where[0] = r;
            s_where[1] = base_c + ic - nc;
            s_where[2] = base_s + is - ns;
          }
          break;
        }
        base_c += __shfl(ic, 63);
        base_s += __shfl(is, 63);
      }
    }
  }
  __syncthreads();
  return Where{s_where[0], s_where[1], s_where[2]};
}

// Per-lane query slices: bf16 kept packed for v_dot2_f32_bf16, fp32 as is.
template <typename T, int DH, int GQ>
struct QSlice;
template <int DH, int GQ>
struct QSlice<uint16_t, DH, GQ> {
  using RS = RowShape<uint16_t, DH>;
  uint32_t w[GQ][RS::kElems / 2];
  __device__ void load(const uint16_t *q0, int DHs, int sub) {
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh)
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p) {
        const uint4 v = *reinterpret_cast<const uint4 *>(q0 + (int64_t)hh * DHs + (sub + 8 * p) * RS::kEP);
        w[hh][p * 4 + 0] = v.x;
        w[hh][p * 4 + 1] = v.y;
        w[hh][p * 4 + 2] = v.z;
        w[hh][p * 4 + 3] = v.w;
      }
  }
  __device__ void dots(const uint4 (&kv)[RS::kNP], float (&acc)[GQ]) const {
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
      float a = 0.f;
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p) {
        a = dot2_bf16(kv[p].x, w[hh][p * 4 + 0], a);
        a = dot2_bf16(kv[p].y, w[hh][p * 4 + 1], a);
        a = dot2_bf16(kv[p].z, w[hh][p * 4 + 2], a);
        a = dot2_bf16(kv[p].w, w[hh][p * 4 + 3], a);
      }
      acc[hh] = a;
    }
  }
};
template <int DH, int GQ>
struct QSlice<float, DH, GQ> {
  using RS = RowShape<float, DH>;
  float f[GQ][RS::kElems];
  __device__ void load(const float *q0, int DHs, int sub) {
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh)
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p) {
        const uint4 v = *reinterpret_cast<const uint4 *>(q0 + (int64_t)hh * DHs + (sub + 8 * p) * RS::kEP);
        widen(v, &f[hh][p * RS::kEP], float());
      }
  }
  __device__ void dots(const uint4 (&kv)[RS::kNP], float (&acc)[GQ]) const {
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) acc[hh] = 0.f;
#pragma unroll
    for (int p = 0; p < RS::kNP; ++p) {
      float kf[RS::kEP];
      widen(kv[p], kf, float());
#pragma unroll
      for (int e = 0; e < RS::kEP; ++e)
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) acc[hh] = fmaf(kf[e], f[hh][p * RS::kEP + e], acc[hh]);
    }
  }
};

// A chunk's logits, token-major in LDS ([nt][Hq], scaled), into the chunk's
// statistics per head (max over every token, then the sums of exp(l - max)
// over every token and over the visual ones) and its visual logits (and every
// logit when rows are asked). Called by all threads after the logits landed.
__device__ __forceinline__ void chunk_epilogue(const float *s_log, float4 *s_part, int nt, int Hq, int l, int r,
                                               int64_t c, int R, int64_t C_total, int64_t T_total, int64_t tok0,
                                               int t_begin, const int32_t *__restrict__ vis_start,
                                               const int32_t *__restrict__ cu_vis, float *__restrict__ vlog,
                                               float4 *__restrict__ stats, float *__restrict__ rows) {
  // tph threads per head take every tph-th token; their partials merge in a
  // fixed order.
  const int v_lo = vis_start[r] - t_begin;
  const int v_hi = v_lo + (cu_vis[r + 1] - cu_vis[r]);
  const int tph = max(1, kThreads / Hq);
  for (int h0 = 0; h0 < Hq; h0 += kThreads / tph) {
    const int h = h0 + (int)threadIdx.x / tph, sl = (int)threadIdx.x % tph;
    const bool act = (int)threadIdx.x / tph < kThreads / tph && h < Hq;
    float m = -INFINITY, z = 0.f, v = 0.f;
    if (act) {
      for (int t = sl; t < nt; t += tph) m = fmaxf(m, s_log[t * Hq + h]);
      for (int t = sl; t < nt; t += tph) {
        const float e = exp2f(s_log[t * Hq + h] - m);
        z += e;
        if (t >= v_lo && t < v_hi) v += e;
      }
    }
    s_part[threadIdx.x] = make_float4(m, z, v, 0.f);
    __syncthreads();
    if (act && sl == 0) {
      float M = -INFINITY;
      for (int x = 0; x < tph; ++x) M = fmaxf(M, s_part[threadIdx.x + x].x);
      float Z = 0.f, V = 0.f;
      for (int x = 0; x < tph; ++x) {
        const float4 e = s_part[threadIdx.x + x];
        const float f = e.x == -INFINITY ? 0.f : exp2f(e.x - M);
        Z = fmaf(e.y, f, Z);
        V = fmaf(e.z, f, V);
      }
      stats[((int64_t)l * Hq + h) * C_total + c] = make_float4(M, Z, V, 0.f);
    }
    __syncthreads();
  }

  // Visual logits, layer-major ([layer][visual token][head]): this block's
  // are one contiguous run of whole cache lines, stored non-temporally (the
  // finalize reads them once, after the whole pass; kept in cache they
  // displace key lines still in flight). Every logit if rows are asked.
  const int vb = max(0, v_lo), ve = min(nt, v_hi);
  const int64_t vtok0 = (int64_t)cu_vis[r] - vis_start[r] + t_begin;
  for (int e = vb * Hq + (int)threadIdx.x; e < ve * Hq; e += kThreads) {
    const int t = e / Hq, h = e - t * Hq;
    __builtin_nontemporal_store(s_log[e], &vlog[((int64_t)l * cu_vis[R] + vtok0 + t) * Hq + h]);
  }
  if (rows)
    for (int e = threadIdx.x; e < nt * Hq; e += kThreads) {
      const int t = e / Hq, h = e - t * Hq;
      rows[((int64_t)l * Hq + h) * T_total + tok0 + t_begin + t] = s_log[e];
    }
}

// Requires (8 * kWaves) % Hkv == 0, so that every lane keeps one KV head.
// LDS holds the chunk's logits token-major, [CH][Hq].
template <typename T, int DH, int GQ>
__global__ __launch_bounds__(kThreads) void k_score_stream(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ slice_off,
    const int32_t *__restrict__ row_pos, int R, int Hq, int Hkv, int CH, int64_t C_total,
    int64_t T_total, float scale, float *__restrict__ vlog, float4 *__restrict__ stats,
    float *__restrict__ rows) {
  using RS = RowShape<T, DH>;
  extern __shared__ float s_log[];          // [CH][Hq]
  __shared__ float4 s_part[kThreads];
  __shared__ int s_where[3];

  const int64_t c = blockIdx.x % C_total;
  const int l = (int)(blockIdx.x / C_total);
  const Where wh = locate(c, false, R, CH, kSliceTokens, cu_seqlens, cu_vis, row_pos, chunk_off, slice_off,
                          s_where);
  const int r = wh.r;
  const int c_local = (int)(c - wh.c0);
  const int64_t tok0 = cu_seqlens[r];
  // the scored row sits at position P - 1 and sees keys 0 .. P - 1 (causal)
  const int P = row_pos ? row_pos[r] + 1 : cu_seqlens[r + 1] - (int)tok0;
  const int t_begin = c_local * CH;
  const int nt = min(P - t_begin, CH);
  if (nt <= 0) return;
  const int nrows = nt * Hkv;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rr = lane >> 3, sub = lane & 7;
  const int kvh = (8 * wave + rr) % Hkv;

  QSlice<T, DH, GQ> qs;
  qs.load(q + (((int64_t)l * R + r) * Hq + kvh * GQ) * DH, DH, sub);

  const T *kchunk = k + ((int64_t)l * T_total + tok0 + t_begin) * Hkv * DH;
  const int ngroups = (nrows + 7) >> 3;
  for (int j = 0; wave + kWaves * j < ngroups; j += kUnroll) {
    uint4 buf[kUnroll][RS::kNP];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int row = min((wave + kWaves * (j + u)) * 8 + rr, nrows - 1);
      const T *kp = kchunk + (int64_t)row * DH;
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p)
        buf[u][p] = stream_load(kp + (sub + 8 * p) * RS::kEP);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      float acc[GQ];
      qs.dots(buf[u], acc);
      float mine = 0.f;
#pragma unroll
      for (int hh = 0; hh < GQ; ++hh) {
        const float s = sum8(acc[hh]);
        if (sub == hh) mine = s;
      }
      const int row = (wave + kWaves * (j + u)) * 8 + rr;
      if (row < nrows && sub < GQ) s_log[row * GQ + sub] = mine * scale;   // = [t][kvh*GQ+sub]
    }
  }
  __syncthreads();
  chunk_epilogue(s_log, s_part, nt, Hq, l, r, c, R, C_total, T_total, tok0, t_begin, vis_start, cu_vis,
                 vlog, stats, rows);
}

template <typename T, int DH, int GM>
__global__ __launch_bounds__(kThreads) void k_score_partial(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ slice_off,
    const int32_t *__restrict__ row_pos, int R, int Hq, int Hkv, int g, int HG, int CH,
    int64_t C_total, int64_t T_total, float scale, float *__restrict__ vlog,
    float4 *__restrict__ stats, float *__restrict__ rows) {
  using RS = RowShape<T, DH>;
  extern __shared__ float s_logit[];   // [GM][CH]
  __shared__ float s_red[kWaves][GM];
  __shared__ int s_where[3];

  int64_t bid = blockIdx.x;
  const int hg = (int)(bid % HG);
  bid /= HG;
  const int kv = (int)(bid % Hkv);
  bid /= Hkv;
  const int64_t c = bid % C_total;
  const int l = (int)(bid / C_total);
  const Where wh = locate(c, false, R, CH, kSliceTokens, cu_seqlens, cu_vis, row_pos, chunk_off, slice_off,
                          s_where);
  const int r = wh.r;
  const int c_local = (int)(c - wh.c0);
  const int64_t tok0 = cu_seqlens[r];
  const int P = row_pos ? row_pos[r] + 1 : cu_seqlens[r + 1] - (int)tok0;
  const int t_begin = c_local * CH;
  const int nt = min(P - t_begin, CH);
  if (nt <= 0) return;
  const int h0 = kv * g + hg * GM;
  const int gh = min(GM, g - hg * GM);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rr = lane >> 3, sub = lane & 7;

  float qf[GM][RS::kElems];
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) {
    const int h = h0 + min(hh, gh - 1);
    const T *qp = q + (((int64_t)l * R + r) * Hq + h) * DH;
#pragma unroll
    for (int p = 0; p < RS::kNP; ++p) {
      const uint4 v = *reinterpret_cast<const uint4 *>(qp + (sub + 8 * p) * RS::kEP);
      widen(v, &qf[hh][p * RS::kEP], T());
    }
  }

  const T *kbase = k + (((int64_t)l * T_total + tok0 + t_begin) * Hkv + kv) * DH;
  const int64_t kstride = (int64_t)Hkv * DH;
  const int ngroups = (nt + 7) >> 3;

  for (int g0 = wave * kUnroll; g0 < ngroups; g0 += kWaves * kUnroll) {
    uint4 buf[kUnroll][RS::kNP];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int t = min((g0 + u) * 8 + rr, nt - 1);
      const T *kp = kbase + (int64_t)t * kstride;
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p)
        buf[u][p] = stream_load(kp + (sub + 8 * p) * RS::kEP);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      float acc[GM];
#pragma unroll
      for (int hh = 0; hh < GM; ++hh) acc[hh] = 0.f;
#pragma unroll
      for (int p = 0; p < RS::kNP; ++p) {
        float kf[RS::kEP];
        widen(buf[u][p], kf, T());
#pragma unroll
        for (int e = 0; e < RS::kEP; ++e)
#pragma unroll
          for (int hh = 0; hh < GM; ++hh) acc[hh] = fmaf(kf[e], qf[hh][p * RS::kEP + e], acc[hh]);
      }
      float mine = 0.f;
#pragma unroll
      for (int hh = 0; hh < GM; ++hh) {
        const float s = sum8(acc[hh]);
        if (sub == hh) mine = s;
      }
      const int t = (g0 + u) * 8 + rr;
      if (t < nt && sub < gh) s_logit[sub * CH + t] = mine * scale;
    }
  }
  __syncthreads();

  const int v_r = vis_start[r];
  const int N_r = cu_vis[r + 1] - cu_vis[r];
  const int vb = max(0, v_r - t_begin), ve = min(nt, v_r + N_r - t_begin);
  float m[GM];
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) {
    float x = -INFINITY;
    if (hh < gh)
      for (int t = threadIdx.x; t < nt; t += kThreads) x = fmaxf(x, s_logit[hh * CH + t]);
    x = wave_max(x);
    if (lane == 0) s_red[wave][hh] = x;
  }
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) {
    float x = s_red[0][hh];
    for (int w = 1; w < kWaves; ++w) x = fmaxf(x, s_red[w][hh]);
    m[hh] = x;
  }
  __syncthreads();
  float zs[GM], vs[GM];
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) {
    float z = 0.f, v = 0.f;
    if (hh < gh)
      for (int t = threadIdx.x; t < nt; t += kThreads) {
        const float e = exp2f(s_logit[hh * CH + t] - m[hh]);
        z += e;
        if (t >= vb && t < ve) v += e;
      }
    zs[hh] = wave_sum(z);
    vs[hh] = wave_sum(v);
  }
#pragma unroll
  for (int hh = 0; hh < GM; ++hh)
    if (lane == 0) s_red[wave][hh] = zs[hh];
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) {
    float x = 0.f;
    for (int w = 0; w < kWaves; ++w) x += s_red[w][hh];
    zs[hh] = x;
  }
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < GM; ++hh)
    if (lane == 0) s_red[wave][hh] = vs[hh];
  __syncthreads();
  if (threadIdx.x < gh) {
    const int hh = threadIdx.x;
    float x = 0.f;
    for (int w = 0; w < kWaves; ++w) x += s_red[w][hh];
    float zz = 0.f, mm = 0.f;
#pragma unroll
    for (int j = 0; j < GM; ++j)
      if (j == hh) {
        zz = zs[j];
        mm = m[j];
      }
    stats[((int64_t)l * Hq + h0 + hh) * C_total + c] = make_float4(mm, zz, x, 0.f);
  }

  const int64_t vtok0 = (int64_t)cu_vis[r] + t_begin - v_r;
  for (int hh = 0; hh < gh; ++hh) {
    for (int t = vb + threadIdx.x; t < ve; t += kThreads)
      vlog[((int64_t)l * cu_vis[R] + vtok0 + t) * Hq + h0 + hh] = s_logit[hh * CH + t];
    if (rows) {
      float *rd = rows + ((int64_t)l * Hq + h0 + hh) * T_total + tok0 + t_begin;
      for (int t = threadIdx.x; t < nt; t += kThreads) rd[t] = s_logit[hh * CH + t];
    }
  }
}

// The first chunk of request r: sum over r' < r of ceil(P_r' / CH), scanned
// by wave 0 64 requests at a time (or read from the k_score_prefix output for
// batches over kScanMaxR). Block-uniform, through LDS.
__device__ int chunk_first(int r, int R, int CH, const int32_t *__restrict__ cu_seqlens,
                           const int32_t *__restrict__ row_pos, const int32_t *__restrict__ chunk_off,
                           int *s_out) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int base = 0;
    if (R > kScanMaxR) {
      base = chunk_off[r];
    } else {
      for (int r0 = 0; r0 < r; r0 += 64) {
        const int q = r0 + lane;
        int nc = 0;
        if (q < r) {
          const int P = row_pos ? row_pos[q] + 1 : cu_seqlens[q + 1] - cu_seqlens[q];
          nc = (P + CH - 1) / CH;
        }
        for (int o = 1; o < 64; o <<= 1) nc += __shfl_xor(nc, o);
        base += nc;
      }
    }
    if (lane == 0) s_out[0] = base;
  }
  __syncthreads();
  return s_out[0];
}

// Merge the chunk statistics of every (request, layer, head) row into its max
// M and 1/Z, and its share V / Z of the request's visual mass
// S = sum_{l,h} V / Z (= sum_i s_i). One wave per row, kWaves rows a block:
// lanes merge the row's chunks lane-strided with the online rule, then the
// wave combines the lanes (log-sum-exp over (max, sum) pairs).
__global__ __launch_bounds__(kThreads) void k_score_merge(
    const float4 *__restrict__ stats, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ row_pos, const int32_t *__restrict__ chunk_off, int R, int GH, int CH,
    int64_t C_total, float2 *__restrict__ rowstat, float *__restrict__ rowmass) {
  __shared__ int s_first[1];
  const int bpr = (GH + kWaves - 1) / kWaves;   // blocks per request
  const int r = blockIdx.x / bpr;
  const int c0 = chunk_first(r, R, CH, cu_seqlens, row_pos, chunk_off, s_first);
  const int P = row_pos ? row_pos[r] + 1 : cu_seqlens[r + 1] - cu_seqlens[r];
  const int c1 = c0 + (P + CH - 1) / CH;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int p = (blockIdx.x % bpr) * kWaves + wave;
  if (p >= GH) return;
  const float4 *st = stats + (int64_t)p * C_total;
  float m = -INFINITY, z = 0.f, v = 0.f;
  for (int c = c0 + lane; c < c1; c += 64) {
    const float4 e = st[c];
    if (e.x > m) {
      const float f = m == -INFINITY ? 0.f : exp2f(m - e.x);
      z = fmaf(z, f, e.y);
      v = fmaf(v, f, e.z);
      m = e.x;
    } else {
      const float f = exp2f(e.x - m);
      z = fmaf(e.y, f, z);
      v = fmaf(e.z, f, v);
    }
  }
  const float M = wave_max(m);
  const float f = m == -INFINITY ? 0.f : exp2f(m - M);
  const float Z = wave_sum(z * f), V = wave_sum(v * f);
  if (lane == 0) {
    rowstat[(int64_t)r * GH + p] = make_float2(M, 1.0f / Z);
    rowmass[(int64_t)r * GH + p] = V / Z;
  }
}

// s_i = sum_{l,h} exp(l_i - M) / Z (Eq. 6-7), divided by S (Eq. 8), for one
// slice of a request's visual tokens; a thread per token reads its layers'
// Hq contiguous logits directly (every load independent of the others).
__global__ __launch_bounds__(kThreads) void k_score_finalize(
    const float *__restrict__ vlog, const float2 *__restrict__ rowstat, const float *__restrict__ rowmass,
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ row_pos,
    const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ slice_off, int R, int G, int Hq, int CH,
    int SL, int64_t N_total, float *__restrict__ scores) {
  const int GH = G * Hq;
  __shared__ float2 sMZ[kMaxPairs];
  __shared__ float s_red[kWaves];
  __shared__ int s_where[3];
  const Where wh = locate(blockIdx.x, true, R, CH, SL, cu_seqlens, cu_vis, row_pos, chunk_off, slice_off,
                          s_where);
  const int r = wh.r, sl = (int)(blockIdx.x - wh.s0);
  // S = sum over the request's rows of V / Z: each thread its rows p = t,
  // t + kThreads, ... in order, then the wave and the waves in a fixed order
  float part = 0.f;
  for (int p = threadIdx.x; p < GH; p += kThreads) {
    sMZ[p] = rowstat[(int64_t)r * GH + p];
    part += rowmass[(int64_t)r * GH + p];
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = part;
  __syncthreads();
  float S = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) S += s_red[w];
  const float invS = 1.0f / S;
  const int64_t n0 = cu_vis[r];
  const int N_r = cu_vis[r + 1] - (int)n0;
  const int end = min(N_r, (sl + 1) * SL);
  // a row before the end of the visual span sees only the tokens up to itself
  const int seen = row_pos ? min(N_r, row_pos[r] - vis_start[r] + 1) : N_r;
  for (int i = sl * SL + threadIdx.x; i < end; i += kThreads) {
    if (i >= seen) {
      scores[n0 + i] = 0.f;
      continue;
    }
    // (layer, head) pairs p = l * Hq + h in increasing order; layer l's logits
    // of this token are Hq contiguous floats
    float acc = 0.f;
    for (int l = 0; l < G; ++l) {
      const float *lg = vlog + ((int64_t)l * N_total + n0 + i) * Hq;
      const float2 *mz = sMZ + l * Hq;
      if ((Hq & 3) == 0) {
        for (int h = 0; h < Hq; h += 4) {
          const float4 x = *reinterpret_cast<const float4 *>(lg + h);
          acc = fmaf(exp2f(x.x - mz[h].x), mz[h].y, acc);
          acc = fmaf(exp2f(x.y - mz[h + 1].x), mz[h + 1].y, acc);
          acc = fmaf(exp2f(x.z - mz[h + 2].x), mz[h + 2].y, acc);
          acc = fmaf(exp2f(x.w - mz[h + 3].x), mz[h + 3].y, acc);
        }
      } else {
        for (int h = 0; h < Hq; ++h) acc = fmaf(exp2f(lg[h] - mz[h].x), mz[h].y, acc);
      }
    }
    scores[n0 + i] = acc * invS;
  }
}

// The same as k_score_finalize, for Hq % 4 == 0 and G * Hq <= 4 kFinQ: the
// slice's logits of a layer are one contiguous run of 256 Hq floats, read by
// the whole block as 16-byte pieces in order (every load instruction covers
// consecutive lines), all layers' pieces in flight at once. A piece holds 4
// heads of one token; its share sum_h exp(l - M) / Z goes to LDS, and each
// thread then adds its token's shares layer by layer, heads ascending (a fixed
// order, as everywhere in the score pass).
constexpr int kFinQMax = 32;   // pieces a thread, over all layers
template <int kFinQ>
__global__ __launch_bounds__(kThreads) void k_score_finalize_c(
    const float *__restrict__ vlog, const float2 *__restrict__ rowstat, const float *__restrict__ rowmass,
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ row_pos,
    const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ slice_off, int R, int G, int Hq, int CH,
    int64_t N_total, float *__restrict__ scores) {
  extern __shared__ float s_part[];   // [G][kThreads][PS]
  const int GH = G * Hq, P = Hq / 4, PS = P | 1, GP = G * P;
  __shared__ float2 sMZ[4 * kFinQ];
  __shared__ float s_red[kWaves];
  __shared__ int s_where[3];
  const Where wh = locate(blockIdx.x, true, R, CH, kThreads, cu_seqlens, cu_vis, row_pos, chunk_off, slice_off,
                          s_where);
  const int r = wh.r, sl = (int)(blockIdx.x - wh.s0);
  const int t = threadIdx.x;
  const int64_t n0 = cu_vis[r];
  const int N_r = cu_vis[r + 1] - (int)n0;
  const int tok0 = sl * kThreads, cnt = min(N_r - tok0, kThreads);
  // piece q of this thread: layer q / P, piece k = (q % P) kThreads + t of the
  // layer's run, token k / P (exact in fp32 for k < 2^13: the quotient's
  // fraction is at least 1 / (2P) from the next integer)
  const float invP = 1.0f / (float)P;
  auto tok_of = [&](int k) { return (int)(((float)k + 0.5f) * invP); };
  // every piece of every layer first: layer l's run starts at token tok0
  float4 x[kFinQ];
  {
    int l = 0, j = 0;
#pragma unroll
    for (int q = 0; q < kFinQ; ++q) {
      if (q < GP) {
        const int k = j * kThreads + t;
        if (tok_of(k) < cnt)
          x[q] = *reinterpret_cast<const float4 *>(vlog + ((int64_t)l * N_total + n0 + tok0) * Hq + 4 * (int64_t)k);
      }
      ++j;
      l += j == P ? 1 : 0;
      j = j == P ? 0 : j;
    }
  }
  float part = 0.f;
  for (int p = t; p < GH; p += kThreads) {
    sMZ[p] = rowstat[(int64_t)r * GH + p];
    part += rowmass[(int64_t)r * GH + p];
  }
  part = wave_sum(part);
  if ((t & 63) == 0) s_red[t >> 6] = part;
  __syncthreads();
  float S = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) S += s_red[w];
  const float invS = 1.0f / S;
  {
    int l = 0, j = 0;
#pragma unroll
    for (int q = 0; q < kFinQ; ++q) {
      if (q < GP) {
        const int k = j * kThreads + t, tok = tok_of(k), jj = k - tok * P;
        if (tok < cnt) {
          const float2 *mz = sMZ + l * Hq + 4 * jj;
          float v = exp2f(x[q].x - mz[0].x) * mz[0].y;
          v = fmaf(exp2f(x[q].y - mz[1].x), mz[1].y, v);
          v = fmaf(exp2f(x[q].z - mz[2].x), mz[2].y, v);
          v = fmaf(exp2f(x[q].w - mz[3].x), mz[3].y, v);
          s_part[(l * kThreads + tok) * PS + jj] = v;
        }
      }
      ++j;
      l += j == P ? 1 : 0;
      j = j == P ? 0 : j;
    }
  }
  __syncthreads();
  if (t >= cnt) return;
  // a row before the end of the visual span sees only the tokens up to itself
  const int seen = row_pos ? min(N_r, row_pos[r] - vis_start[r] + 1) : N_r;
  float acc = 0.f;
  for (int l = 0; l < G; ++l)
    for (int j = 0; j < P; ++j) acc += s_part[(l * kThreads + t) * PS + j];
  scores[n0 + tok0 + t] = tok0 + t < seen ? acc * invS : 0.f;
}

// Optional full rows A[p*, :] for inspection: raw logits -> probabilities.
__global__ __launch_bounds__(kThreads) void k_rows_finalize(
    const float4 *__restrict__ stats, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ chunk_off, int R, int64_t C_total, int64_t T_total,
    float *__restrict__ rows) {
  const int p = blockIdx.x / R, r = blockIdx.x % R;
  const float4 *st = stats + (int64_t)p * C_total;
  const int c0 = chunk_off[r], c1 = chunk_off[r + 1];
  float M = -INFINITY;
  for (int c = c0; c < c1; ++c) M = fmaxf(M, st[c].x);
  float Z = 0.f;
  for (int c = c0; c < c1; ++c) Z = fmaf(st[c].y, exp2f(st[c].x - M), Z);
  const float invZ = 1.0f / Z;
  float *row = rows + (int64_t)p * T_total;
  for (int t = cu_seqlens[r] + threadIdx.x; t < cu_seqlens[r + 1]; t += kThreads)
    row[t] = exp2f(row[t] - M) * invZ;
}

template <typename T, int DH>
hipError_t launch_stream_dh(const last_batch *b, const last::ScorePlan &p, const last::ScoreWs &w,
                            const void *q, const void *k, const int32_t *row_pos, float *attn_rows,
                            float scale, hipStream_t s) {
  const int g = b->Hq / b->Hkv;
  const int64_t blocks = (int64_t)b->G * p.C_total;
  const size_t lds = (size_t)p.chunk_tokens * b->Hq * sizeof(float);
  last::launch_begin("score_stream", s);
#define LAST_LAUNCH_GQ(GQV)                                                                        \
  hipLaunchKernelGGL((k_score_stream<T, DH, GQV>), dim3((unsigned)blocks), dim3(kThreads), lds, s, \
                     (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis,          \
                     w.chunk_off, w.slice_off, row_pos, b->R, b->Hq, b->Hkv, p.chunk_tokens,     \
                     p.C_total, p.T_total, scale, w.vlog, w.stats, attn_rows)
  switch (g) {
    case 1: LAST_LAUNCH_GQ(1); break;
    case 2: LAST_LAUNCH_GQ(2); break;
    case 3: LAST_LAUNCH_GQ(3); break;
    case 4: LAST_LAUNCH_GQ(4); break;
    case 5: LAST_LAUNCH_GQ(5); break;
    case 6: LAST_LAUNCH_GQ(6); break;
    case 7: LAST_LAUNCH_GQ(7); break;
    default: LAST_LAUNCH_GQ(8); break;
  }
#undef LAST_LAUNCH_GQ
  return last::launch_end(s);
}

template <typename T, int DH>
hipError_t launch_partial_dh(const last_batch *b, const last::ScorePlan &p,
                             const last::ScoreWs &w, const void *q, const void *k,
                             const int32_t *row_pos, float *attn_rows, float scale, hipStream_t s) {
  const int g = b->Hq / b->Hkv;
  const int64_t blocks = (int64_t)b->G * p.C_total * b->Hkv * p.head_groups;
  const size_t lds = (size_t)p.g_max * p.chunk_tokens * sizeof(float);
  last::launch_begin("score_partial", s);
#define LAST_LAUNCH_GM(GMV)                                                                     \
  hipLaunchKernelGGL((k_score_partial<T, DH, GMV>), dim3((unsigned)blocks), dim3(kThreads), lds, \
                     s, (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis,      \
                     w.chunk_off, w.slice_off, row_pos, b->R, b->Hq, b->Hkv, g, p.head_groups,  \
                     p.chunk_tokens, p.C_total, p.T_total, scale, w.vlog, w.stats,               \
                     attn_rows)
  switch (p.g_max) {
    case 1: LAST_LAUNCH_GM(1); break;
    case 2: LAST_LAUNCH_GM(2); break;
    case 4: LAST_LAUNCH_GM(4); break;
    default: LAST_LAUNCH_GM(8); break;
  }
#undef LAST_LAUNCH_GM
  return last::launch_end(s);
}

}  // namespace

namespace last {

ScorePlan make_score_plan(const last_batch *b, const int32_t *row_pos_h) {
  ScorePlan p{};
  const int g = b->Hq / b->Hkv;
  p.T_total = b->cu_seqlens_h[b->R];
  p.N_total = b->cu_vis_h[b->R];
  p.slice_tokens = kSliceTokens;
  const int64_t elt = b->qk_dtype == LAST_BF16 ? 2 : 4;
  // The streaming kernel keeps one KV head per lane; that needs Hkv | 32 and at
  // most 8 query heads per KV head.
  p.stream = (8 * kWaves) % b->Hkv == 0 && g <= 8;
  if (p.stream) {
    p.g_max = g;
    p.head_groups = 1;
    const int64_t tok_bytes = (int64_t)b->Hkv * b->Dh * elt;
    int64_t ch = (kWgBytes + tok_bytes - 1) / tok_bytes;
    ch = std::min<int64_t>(ch, kLdsLogitFloats / b->Hq);   // the chunk's logits live in LDS
    p.chunk_tokens = (int32_t)std::max<int64_t>(1, ch);
  } else {
    p.g_max = g <= 1 ? 1 : g <= 2 ? 2 : g <= 4 ? 4 : 8;
    p.head_groups = (g + p.g_max - 1) / p.g_max;
    // ~2048 blocks while each chunk's logits fit in LDS
    const int64_t rows = (int64_t)b->G * b->Hkv * p.head_groups * p.T_total;
    int64_t ch = (rows + 2047) / 2048;
    ch = (ch + 63) / 64 * 64;
    const int64_t ch_cap = std::min<int64_t>(kMaxChunk, kLdsLogitFloats / p.g_max);
    p.chunk_tokens = (int32_t)std::max<int64_t>(256, std::min<int64_t>(ch, ch_cap));
  }
  p.C_total = 0;
  p.S_total = 0;
  for (int r = 0; r < b->R; ++r) {
    const int64_t P = row_pos_h ? (int64_t)row_pos_h[r] + 1 : b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r];
    const int64_t N = b->cu_vis_h[r + 1] - b->cu_vis_h[r];
    p.C_total += (P + p.chunk_tokens - 1) / p.chunk_tokens;
    p.S_total += (N + p.slice_tokens - 1) / p.slice_tokens;
  }
  return p;
}

ScoreWs carve_score_ws(void *ws, const last_batch *b, const ScorePlan &p, size_t *bytes) {
  Carver cv(ws);
  ScoreWs w{};
  w.chunk_off = cv.take<int32_t>(b->R + 1);
  w.slice_off = cv.take<int32_t>(b->R + 1);
  w.stats = cv.take<float4>((size_t)b->G * b->Hq * p.C_total);
  w.vlog = cv.take<float>((size_t)b->G * b->Hq * p.N_total);
  w.rowstat = cv.take<float2>((size_t)b->R * b->G * b->Hq);
  w.rowmass = cv.take<float>((size_t)b->R * b->G * b->Hq);
  *bytes = cv.size();
  return w;
}

int score_max_pairs() { return kMaxPairs; }

hipError_t launch_score_plan(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                             const int32_t *row_pos, hipStream_t s, bool always) {
  if (b->R <= kScanMaxR && !always) return hipSuccess;   // the blocks scan the counts themselves
  launch_begin("score_prefix", s);
  hipLaunchKernelGGL(k_score_prefix, dim3(1), dim3(kThreads), 0, s, b->cu_seqlens, b->cu_vis, row_pos, b->R,
                     p.chunk_tokens, p.slice_tokens, w.chunk_off, w.slice_off);
  return launch_end(s);
}

hipError_t launch_score_tail(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                             const int32_t *row_pos, float *scores, hipStream_t s) {
  const int GH = b->G * b->Hq;
  launch_begin("score_merge", s);
  hipLaunchKernelGGL(k_score_merge, dim3((unsigned)((int64_t)b->R * ((GH + kWaves - 1) / kWaves))), dim3(kThreads),
                     0, s, w.stats, b->cu_seqlens, row_pos, w.chunk_off, b->R, GH, p.chunk_tokens, p.C_total,
                     w.rowstat, w.rowmass);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;
  launch_begin("score_finalize", s);
  if (b->Hq % 4 == 0 && GH <= 4 * kFinQMax && p.slice_tokens == kThreads) {
    const size_t lds = (size_t)b->G * kThreads * ((b->Hq / 4) | 1) * sizeof(float);
    const int q = GH / 4;   // pieces a thread
#define LAST_FIN(Q)                                                                                               \
  hipLaunchKernelGGL(k_score_finalize_c<Q>, dim3((unsigned)p.S_total), dim3(kThreads), lds, s, w.vlog, w.rowstat, \
                     w.rowmass, b->cu_seqlens, b->cu_vis, b->vis_start, row_pos, w.chunk_off, w.slice_off, b->R,   \
                     b->G, b->Hq, p.chunk_tokens, p.N_total, scores)
    if (q <= 4) LAST_FIN(4);
    else if (q <= 8) LAST_FIN(8);
    else if (q <= 16) LAST_FIN(16);
    else LAST_FIN(32);
#undef LAST_FIN
  } else {
    hipLaunchKernelGGL(k_score_finalize, dim3((unsigned)p.S_total), dim3(kThreads), 0, s, w.vlog, w.rowstat,
                       w.rowmass, b->cu_seqlens, b->cu_vis, b->vis_start, row_pos, w.chunk_off, w.slice_off, b->R,
                       b->G, b->Hq, p.chunk_tokens, p.slice_tokens, p.N_total, scores);
  }
  return launch_end(s);
}

hipError_t launch_scores(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                         const void *q, const void *k, const int32_t *row_pos, float *scores,
                         float *attn_rows, float scale, hipStream_t s) {
  // the debug rows read the chunk prefixes directly, so they are always computed then
  hipError_t e = launch_score_plan(b, p, w, row_pos, s, attn_rows != nullptr);
  if (e != hipSuccess) return e;
  // logits in base-2 units
  scale = (float)((double)scale * 1.4426950408889634);

  const bool bf = b->qk_dtype == LAST_BF16;
  if (p.stream)
    e = bf ? (b->Dh == 64 ? launch_stream_dh<uint16_t, 64>(b, p, w, q, k, row_pos, attn_rows, scale, s)
                          : launch_stream_dh<uint16_t, 128>(b, p, w, q, k, row_pos, attn_rows, scale, s))
           : (b->Dh == 64 ? launch_stream_dh<float, 64>(b, p, w, q, k, row_pos, attn_rows, scale, s)
                          : launch_stream_dh<float, 128>(b, p, w, q, k, row_pos, attn_rows, scale, s));
  else
    e = bf ? (b->Dh == 64 ? launch_partial_dh<uint16_t, 64>(b, p, w, q, k, row_pos, attn_rows, scale, s)
                          : launch_partial_dh<uint16_t, 128>(b, p, w, q, k, row_pos, attn_rows, scale, s))
           : (b->Dh == 64 ? launch_partial_dh<float, 64>(b, p, w, q, k, row_pos, attn_rows, scale, s)
                          : launch_partial_dh<float, 128>(b, p, w, q, k, row_pos, attn_rows, scale, s));
  if (e != hipSuccess) return e;

  e = launch_score_tail(b, p, w, row_pos, scores, s);
  if (e != hipSuccess || !attn_rows) return e;

  launch_begin("score_rows", s);
  hipLaunchKernelGGL(k_rows_finalize, dim3((unsigned)(b->G * b->Hq * b->R)), dim3(kThreads), 0, s,
                     w.stats, b->cu_seqlens, w.chunk_off, b->R, p.C_total, p.T_total, attn_rows);
  return launch_end(s);
}

}  // namespace last
