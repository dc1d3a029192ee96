// Score pass of LAST (arXiv 2607.27952, Sec. 3.3, Eq. 6-8) for gfx950.
//
// The attention row of the last query token is recomputed from q and the key
// cache instead of being read from a materialised P x P map (same numbers,
// O(P) instead of O(P^2) work per head). The row needs a softmax over the
// whole prefix while the keys are streamed in chunks, so the pass is split:
//
//   k_score_plan      one block: per-request chunk/slice prefix sums and the
//                     chunk -> request / slice -> request maps.
//   k_score_partial   one block per (layer, chunk of tokens, KV head, query-head
//                     group). Streams the chunk's key rows once (each row is
//                     Dh * elt bytes; 8 lanes cover one row with 16-byte loads,
//                     so a wave reads 8 rows per instruction), forms the logits
//                     of every query head sharing that KV head with exact
//                     bf16 -> fp32 widening and fp32 FMAs, reduces each row over
//                     its 8 lanes with DPP, and keeps the chunk's logits in LDS.
//                     It then writes, per head, the chunk's max m, sum of
//                     exp(l - m) over all tokens Z and over the visual tokens V,
//                     and the raw logits of the visual columns.
//   k_score_finalize  one block per slice of a request's visual tokens. Merges
//                     the chunk statistics of every (layer, head) row into the
//                     row's max M and normaliser Z, forms
//                     s_i = sum_{l,h} exp(l_i - M) / Z   (Eq. 6-7)
//                     and divides by the visual mass sum_{l,h} V / Z, which is
//                     sum_i s_i (Eq. 8), so no second pass over s is needed.
//
// Every reduction has a fixed order, so results are bitwise reproducible.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 4;          // row groups (8 rows each) in flight per wave
constexpr int kMaxChunk = 4096;     // tokens per chunk, upper bound
constexpr int kLdsLogitFloats = 8192;
constexpr int kSliceTokens = 256;   // visual tokens per finalize block
constexpr int kMaxPairs = 4096;     // G * Hq handled by the finalize block

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

// Exclusive scan of one int per thread over the block; returns the prefix and
// writes the block total. `sh` needs blockDim/64 ints.
__device__ int block_exclusive_scan(int v, int *sh, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int before = 0, tot = 0;
  for (int w = 0; w < nw; ++w) {
    const int s = sh[w];
    if (w < wave) before += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return before + x - v;
}

__global__ __launch_bounds__(kThreads) void k_score_plan(
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ cu_vis, int R, int CH,
    int SL, int64_t C_cap, int64_t S_cap, int32_t *__restrict__ chunk_off,
    int32_t *__restrict__ chunk_req, int32_t *__restrict__ slice_off,
    int32_t *__restrict__ slice_req) {
  __shared__ int sh[kThreads / 64];
  int carry_c = 0, carry_s = 0;
  for (int base = 0; base < R; base += kThreads) {
    const int r = base + (int)threadIdx.x;
    int nc = 0, ns = 0;
    if (r < R) {
      const int P = cu_seqlens[r + 1] - cu_seqlens[r];
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
      for (int c = 0; c < nc; ++c)
        if (pc + c < C_cap) chunk_req[pc + c] = r;
      for (int c = 0; c < ns; ++c)
        if (ps + c < S_cap) slice_req[ps + c] = r;
    }
    carry_c += tc;
    carry_s += ts;
  }
  if (threadIdx.x == 0) {
    chunk_off[R] = carry_c;
    slice_off[R] = carry_s;
  }
}

template <typename T, int DH, int GM>
__global__ __launch_bounds__(kThreads) void k_score_partial(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ chunk_off, const int32_t *__restrict__ chunk_req, int R, int Hq,
    int Hkv, int g, int HG, int CH, int64_t C_total, int64_t T_total, int64_t N_total,
    float scale, float *__restrict__ vlog, float4 *__restrict__ stats,
    float *__restrict__ rows) {
  using RS = RowShape<T, DH>;
  extern __shared__ float s_logit[];   // [GM][CH]
  __shared__ float s_red[kWaves][GM];

  int64_t bid = blockIdx.x;
  const int hg = (int)(bid % HG);
  bid /= HG;
  const int kv = (int)(bid % Hkv);
  bid /= Hkv;
  const int64_t c = bid % C_total;
  const int l = (int)(bid / C_total);
  const int r = chunk_req[c];
  const int c_local = (int)(c - chunk_off[r]);
  const int64_t tok0 = cu_seqlens[r];
  const int P = cu_seqlens[r + 1] - (int)tok0;
  const int t_begin = c_local * CH;
  const int nt = min(P - t_begin, CH);
  if (nt <= 0) return;
  const int h0 = kv * g + hg * GM;
  const int gh = min(GM, g - hg * GM);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rr = lane >> 3, sub = lane & 7;

  // This lane's slice of every query vector, widened to fp32 once.
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
        buf[u][p] = *reinterpret_cast<const uint4 *>(kp + (sub + 8 * p) * RS::kEP);
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

  // Chunk statistics per head: max over every token, then sums of exp(l - m)
  // over every token and over the visual ones.
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
        const float e = expf(s_logit[hh * CH + t] - m[hh]);
        z += e;
        if (t >= vb && t < ve) v += e;
      }
    z = wave_sum(z);
    v = wave_sum(v);
    zs[hh] = z;
    vs[hh] = v;
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

  // Raw scaled logits of the visual columns (and of every column if asked).
  const int64_t vdst0 = (int64_t)cu_vis[r] + t_begin - v_r;
  for (int hh = 0; hh < gh; ++hh) {
    float *dst = vlog + ((int64_t)l * Hq + h0 + hh) * N_total + vdst0;
    for (int t = vb + threadIdx.x; t < ve; t += kThreads) dst[t] = s_logit[hh * CH + t];
    if (rows) {
      float *rd = rows + ((int64_t)l * Hq + h0 + hh) * T_total + tok0 + t_begin;
      for (int t = threadIdx.x; t < nt; t += kThreads) rd[t] = s_logit[hh * CH + t];
    }
  }
}

__global__ __launch_bounds__(kThreads) void k_score_finalize(
    const float *__restrict__ vlog, const float4 *__restrict__ stats,
    const int32_t *__restrict__ cu_vis, const int32_t *__restrict__ chunk_off,
    const int32_t *__restrict__ slice_off, const int32_t *__restrict__ slice_req, int GH,
    int64_t C_total, int64_t N_total, int SL, float *__restrict__ scores) {
  __shared__ float sM[kMaxPairs], sInvZ[kMaxPairs], sMass[kMaxPairs];
  __shared__ float s_red[kWaves];
  const int b = blockIdx.x;
  const int r = slice_req[b];
  const int sl = b - slice_off[r];
  const int c0 = chunk_off[r], c1 = chunk_off[r + 1];
  for (int p = threadIdx.x; p < GH; p += kThreads) {
    const float4 *st = stats + (int64_t)p * C_total;
    float M = -INFINITY;
    for (int c = c0; c < c1; ++c) M = fmaxf(M, st[c].x);
    float Z = 0.f, V = 0.f;
    for (int c = c0; c < c1; ++c) {
      const float4 s = st[c];
      const float e = expf(s.x - M);
      Z = fmaf(s.y, e, Z);
      V = fmaf(s.z, e, V);
    }
    sM[p] = M;
    sInvZ[p] = 1.0f / Z;
    sMass[p] = V / Z;
  }
  __syncthreads();
  float part = 0.f;
  for (int p = threadIdx.x; p < GH; p += kThreads) part += sMass[p];
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = part;
  __syncthreads();
  float S = 0.f;
  for (int w = 0; w < kWaves; ++w) S += s_red[w];
  const float invS = 1.0f / S;

  const int64_t n0 = cu_vis[r];
  const int N_r = cu_vis[r + 1] - (int)n0;
  const int end = min(N_r, (sl + 1) * SL);
  for (int i = sl * SL + threadIdx.x; i < end; i += kThreads) {
    float acc = 0.f;
    for (int p = 0; p < GH; ++p) acc = fmaf(expf(vlog[(int64_t)p * N_total + n0 + i] - sM[p]), sInvZ[p], acc);
    scores[n0 + i] = acc * invS;
  }
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
  for (int c = c0; c < c1; ++c) Z = fmaf(st[c].y, expf(st[c].x - M), Z);
  const float invZ = 1.0f / Z;
  float *row = rows + (int64_t)p * T_total;
  for (int t = cu_seqlens[r] + threadIdx.x; t < cu_seqlens[r + 1]; t += kThreads)
    row[t] = expf(row[t] - M) * invZ;
}

template <typename T, int DH>
hipError_t launch_partial_dh(const last_batch *b, const last::ScorePlan &p,
                             const last::ScoreWs &w, const void *q, const void *k,
                             float *attn_rows, float scale, hipStream_t s) {
  const int g = b->Hq / b->Hkv;
  const int64_t blocks = (int64_t)b->G * p.C_total * b->Hkv * p.head_groups;
  const size_t lds = (size_t)p.g_max * p.chunk_tokens * sizeof(float);
  last::launch_begin("score_partial", s);
#define LAST_LAUNCH_GM(GMV)                                                                     \
  hipLaunchKernelGGL((k_score_partial<T, DH, GMV>), dim3((unsigned)blocks), dim3(kThreads), lds, \
                     s, (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis,      \
                     w.chunk_off, w.chunk_req, b->R, b->Hq, b->Hkv, g, p.head_groups,           \
                     p.chunk_tokens, p.C_total, p.T_total, p.N_total, scale, w.vlog, w.stats,    \
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

ScorePlan make_score_plan(const last_batch *b) {
  ScorePlan p{};
  const int g = b->Hq / b->Hkv;
  p.g_max = g <= 1 ? 1 : g <= 2 ? 2 : g <= 4 ? 4 : 8;
  p.head_groups = (g + p.g_max - 1) / p.g_max;
  p.T_total = b->cu_seqlens_h[b->R];
  p.N_total = b->cu_vis_h[b->R];
  // Aim for ~2048 blocks (8 per CU) while keeping each chunk's logits in LDS.
  const int64_t rows = (int64_t)b->G * b->Hkv * p.head_groups * p.T_total;
  int64_t ch = (rows + 2047) / 2048;
  ch = (ch + 63) / 64 * 64;
  const int64_t ch_cap = std::min<int64_t>(kMaxChunk, kLdsLogitFloats / p.g_max);
  p.chunk_tokens = (int32_t)std::max<int64_t>(256, std::min<int64_t>(ch, ch_cap));
  p.slice_tokens = kSliceTokens;
  p.C_total = 0;
  p.S_total = 0;
  for (int r = 0; r < b->R; ++r) {
    const int64_t P = b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r];
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
  w.chunk_req = cv.take<int32_t>(p.C_total);
  w.slice_off = cv.take<int32_t>(b->R + 1);
  w.slice_req = cv.take<int32_t>(p.S_total);
  w.stats = cv.take<float4>((size_t)b->G * b->Hq * p.C_total);
  w.vlog = cv.take<float>((size_t)b->G * b->Hq * p.N_total);
  *bytes = cv.size();
  return w;
}

int score_max_pairs() { return kMaxPairs; }

hipError_t launch_scores(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                         const void *q, const void *k, float *scores, float *attn_rows,
                         float scale, hipStream_t s) {
  launch_begin("score_plan", s);
  hipLaunchKernelGGL(k_score_plan, dim3(1), dim3(kThreads), 0, s, b->cu_seqlens, b->cu_vis,
                     b->R, p.chunk_tokens, p.slice_tokens, p.C_total, p.S_total, w.chunk_off,
                     w.chunk_req, w.slice_off, w.slice_req);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;

  if (b->qk_dtype == LAST_BF16)
    e = b->Dh == 64 ? launch_partial_dh<uint16_t, 64>(b, p, w, q, k, attn_rows, scale, s)
                    : launch_partial_dh<uint16_t, 128>(b, p, w, q, k, attn_rows, scale, s);
  else
    e = b->Dh == 64 ? launch_partial_dh<float, 64>(b, p, w, q, k, attn_rows, scale, s)
                    : launch_partial_dh<float, 128>(b, p, w, q, k, attn_rows, scale, s);
  if (e != hipSuccess) return e;

  launch_begin("score_finalize", s);
  hipLaunchKernelGGL(k_score_finalize, dim3((unsigned)p.S_total), dim3(kThreads), 0, s, w.vlog,
                     w.stats, b->cu_vis, w.chunk_off, w.slice_off, w.slice_req, b->G * b->Hq,
                     p.C_total, p.N_total, p.slice_tokens, scores);
  e = launch_end(s);
  if (e != hipSuccess || !attn_rows) return e;

  launch_begin("score_rows", s);
  hipLaunchKernelGGL(k_rows_finalize, dim3((unsigned)(b->G * b->Hq * b->R)), dim3(kThreads), 0, s,
                     w.stats, b->cu_seqlens, w.chunk_off, b->R, p.C_total, p.T_total, attn_rows);
  return launch_end(s);
}

}  // namespace last
