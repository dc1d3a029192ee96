// Scores from several causal query rows per request (arXiv 2607.27952,
// Sec. 4.3, Table 4: "All Mean" averages the attention rows of every query
// token) for gfx950:
//
//   s_i = sum_l sum_h sum_{m in rows(r)} A^(l,h)[p_m, v_r + i],  w = s / sum s
//
// where the row at position p attends to keys 0 .. p (causal mask of Eq. 6).
// With M rows per request the logits of a (layer, KV head) form an
// (Hq/Hkv * M) x P product Q K^T, which runs on the matrix cores
// (v_mfma_f32_32x32x16_bf16 for bf16, v_mfma_f32_32x32x2f32 for fp32; bf16
// products are exact and accumulate in fp32). A row's softmax needs its max
// and normaliser over all its keys before any probability is final, and
// keeping every visual logit of every row would cost far more traffic than the
// keys themselves, so the keys are read twice:
//
//   k_rows_plan      one block: per request the row groups, key chunks and
//                    visual chunks, the work-item lists and their prefixes.
//   k_rows_stats     one block per (layer, KV head, request, row group, key
//                    chunk): 32 query rows per wave against the chunk's keys,
//                    staged through LDS 64 keys at a time. Each lane keeps, for
//                    the 16 rows of its accumulator, a running max and the sums
//                    of exp(l - max) over all keys and over the visual ones
//                    (one exponential per logit), merged over the wave's lanes
//                    at the end of the chunk.
//   k_rows_merge     one block per request: every row's chunks merged into its
//                    max M and 1/Z, and the visual mass S = sum V / Z over the
//                    request's rows (= sum_i s_i).
//   k_rows_visual    one block per (layer, KV head, request, row group, visual
//                    chunk): the visual logits again, exp(l - M) / Z summed over
//                    the block's rows per key, written per row group.
//   k_rows_finalize  one thread per visual token: the row-group sums over
//                    layers and KV heads in a fixed order, divided by S.
//
// Every reduction has a fixed order, so results are bitwise reproducible.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 64 * last::kRowWaves;
constexpr int kSub = 64;                      // keys per LDS stage: two 32-key tiles
constexpr int kCH = last::kRowChunk;
static_assert(kCH % kSub == 0, "whole stages per chunk");

// A key (or query) row of DH elements as 16-byte pieces. One matrix-core step
// takes one piece from each half of the wave: lanes 0-31 piece 2s, lanes
// 32-63 piece 2s + 1 (8 bf16 -> one 32x32x16 MFMA; 4 fp32 -> four 32x32x2).
template <typename T, int DH>
struct KeyRow {
  static constexpr int kPieces = DH * (int)sizeof(T) / 16;
  static constexpr int kSteps = kPieces / 2;
  static constexpr int kStage = kSub * kPieces;           // pieces per LDS stage
  static constexpr int kPer = kStage / kThreads;          // pieces each thread stages
  static_assert(kPieces >= 8 && kStage % kThreads == 0, "row shape");
};

// LDS slot of piece p of stage row j: the 16 rows a fragment read serves
// together fall in 16 distinct 16-byte bank groups.
template <int NP>
__device__ __forceinline__ int slot(int j, int p) {
  return j * NP + (p ^ (NP >= 16 ? (j & 15) : ((j >> 1) & 7)));
}

__device__ __forceinline__ void mma_piece(f32x16_t &acc, const uint4 &a, const uint4 &b, uint16_t) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma_piece(f32x16_t &acc, const uint4 &a, const uint4 &b, float) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// In a 32 x 32 accumulator lane l holds column l % 32 and, at element v, row
// 4 * (l / 32) + (v % 4) + 8 * (v / 4).
__device__ __forceinline__ int acc_row(int lane, int v) { return 4 * (lane >> 5) + (v & 3) + 8 * (v >> 2); }

// What a block works on: its request's rows split into the (head, row) pairs
// of one KV head, 32 per wave.
struct RowSet {
  int r, m0, M, nrows, tile0;
  bool active;   // the wave has at least one real row
};

__device__ __forceinline__ RowSet row_set(const int32_t *cu_rows, int r, int rg, int g) {
  RowSet s;
  s.r = r;
  s.m0 = cu_rows[r];
  s.M = cu_rows[r + 1] - s.m0;
  s.nrows = g * s.M;
  s.tile0 = (rg * last::kRowWaves + (int)(threadIdx.x >> 6)) * 32;
  s.active = s.tile0 < s.nrows;
  return s;
}

// Row rho of a KV head's set is query head kv * g + rho / M, row rho % M.
template <typename T, int DH>
__device__ __forceinline__ void load_query_frags(const T *q, const RowSet &s, int l, int kv, int g,
                                                 int Hq, int64_t M_total,
                                                 uint4 (&a)[KeyRow<T, DH>::kSteps]) {
  const int lane = threadIdx.x & 63;
  const int rho = s.tile0 + (lane & 31);
  if (rho < s.nrows) {
    const int hh = rho / s.M, m = rho - hh * s.M;
    const char *qp = reinterpret_cast<const char *>(q + (((int64_t)l * M_total + s.m0 + m) * Hq + kv * g + hh) * DH);
#pragma unroll
    for (int st = 0; st < KeyRow<T, DH>::kSteps; ++st)
      a[st] = *reinterpret_cast<const uint4 *>(qp + (2 * st + (lane >> 5)) * 16);
  } else {
#pragma unroll
    for (int st = 0; st < KeyRow<T, DH>::kSteps; ++st) a[st] = make_uint4(0, 0, 0, 0);
  }
}

// Keys [j0, j0 + nk) of one KV head staged in registers, then in LDS.
template <typename T, int DH>
struct Stager {
  using KR = KeyRow<T, DH>;
  uint4 v[KR::kPer];
  __device__ __forceinline__ void load(const char *kbase, int64_t kstride, int j0, int nk) {
#pragma unroll
    for (int i = 0; i < KR::kPer; ++i) {
      const int e = (int)threadIdx.x + kThreads * i, j = e / KR::kPieces, p = e - j * KR::kPieces;
      v[i] = j < nk ? *reinterpret_cast<const uint4 *>(kbase + (int64_t)(j0 + j) * kstride + p * 16)
                    : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(uint4 *buf) const {
#pragma unroll
    for (int i = 0; i < KR::kPer; ++i) {
      const int e = (int)threadIdx.x + kThreads * i, j = e / KR::kPieces, p = e - j * KR::kPieces;
      buf[slot<KR::kPieces>(j, p)] = v[i];
    }
  }
};

// Logits of the wave's 32 rows against the stage's 64 keys (unscaled):
// c0 for keys 0-31, c1 for keys 32-63.
template <typename T, int DH>
__device__ __forceinline__ void stage_dots(const uint4 *buf, const uint4 (&a)[KeyRow<T, DH>::kSteps],
                                           f32x16_t &c0, f32x16_t &c1) {
  using KR = KeyRow<T, DH>;
  const int lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  c0 = f32x16_t{};
  c1 = f32x16_t{};
#pragma unroll
  for (int st = 0; st < KR::kSteps; ++st) {
    const uint4 b0 = buf[slot<KR::kPieces>(col, 2 * st + half)];
    const uint4 b1 = buf[slot<KR::kPieces>(32 + col, 2 * st + half)];
    mma_piece(c0, a[st], b0, T());
    mma_piece(c1, a[st], b1, T());
  }
}

// Running (max, sum exp, visual sum exp) with one exponential per logit: the
// smaller of the new logit and the running max is scaled against the larger.
__device__ __forceinline__ void online_add(float x, bool vis, float &m, float &z, float &vz) {
  const float d = x - m;
  const float e = expf(-fabsf(d));
  const bool up = d > 0.f;
  const float nz = up ? fmaf(z, e, 1.f) : z + e;
  const float nv = up ? fmaf(vz, e, vis ? 1.f : 0.f) : vz + (vis ? e : 0.f);
  const bool live = x != -INFINITY;
  z = live ? nz : z;
  vz = live ? nv : vz;
  m = live ? fmaxf(m, x) : m;
}

__device__ __forceinline__ void online_merge(float &m, float &z, float &vz, float m2, float z2, float v2) {
  const float M = fmaxf(m, m2);
  const float f1 = m == -INFINITY ? 0.f : expf(m - M);
  const float f2 = m2 == -INFINITY ? 0.f : expf(m2 - M);
  z = z * f1 + z2 * f2;
  vz = vz * f1 + v2 * f2;
  m = M;
}

// ---------------------------------------------------------------- plan
__global__ __launch_bounds__(256) void k_rows_plan(
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ vis_start,
    const int32_t *__restrict__ cu_vis, const int32_t *__restrict__ cu_rows,
    const int32_t *__restrict__ row_pos, int R, int Hq, int g, int64_t cap1, int64_t cap2,
    int32_t *__restrict__ off1, int32_t *__restrict__ off2, int64_t *__restrict__ sc_off,
    int4 *__restrict__ rinfo, int4 *__restrict__ items1, int4 *__restrict__ items2) {
  __shared__ int sh[4];
  int carry1 = 0, carry2 = 0;
  int64_t carry_sc = 0;
  __shared__ long long s_sc[256];
  for (int base = 0; base < R; base += 256) {
    const int r = base + (int)threadIdx.x;
    int n1 = 0, n2 = 0, KC = 0, VC = 0, RG = 0, pmax = 0;
    long long nsc = 0;
    if (r < R) {
      const int m0 = cu_rows[r], M = cu_rows[r + 1] - m0;
      pmax = 0;
      for (int m = 0; m < M; ++m) pmax = max(pmax, row_pos[m0 + m]);
      const int tiles = (g * M + 31) / 32;
      RG = (tiles + last::kRowWaves - 1) / last::kRowWaves;
      KC = (pmax + 1 + kCH - 1) / kCH;
      const int N = cu_vis[r + 1] - cu_vis[r];
      const int seen = min(N, pmax - vis_start[r] + 1);
      VC = (seen + kCH - 1) / kCH;
      n1 = RG * KC;
      n2 = RG * VC;
      nsc = (long long)Hq * M * KC;
      rinfo[r] = make_int4(KC, VC, RG, pmax);
    }
    int t1, t2;
    const int p1 = block_exclusive_scan(n1, sh, &t1) + carry1;
    const int p2 = block_exclusive_scan(n2, sh, &t2) + carry2;
    // statistics prefix in 64 bits: a plain sequential scan of this pass's 256 counts
    s_sc[threadIdx.x] = nsc;
    __syncthreads();
    long long psc = carry_sc, tsc = 0;
    for (int i = 0; i < 256; ++i) {
      if (i < (int)threadIdx.x) psc += s_sc[i];
      tsc += s_sc[i];
    }
    __syncthreads();
    if (r < R) {
      off1[r] = p1;
      off2[r] = p2;
      sc_off[r] = psc;
      for (int c = 0; c < KC; ++c)
        for (int rg = 0; rg < RG; ++rg)
          if (p1 + c * RG + rg < cap1) items1[p1 + c * RG + rg] = make_int4(r, rg, c, 0);
      for (int c = 0; c < VC; ++c)
        for (int rg = 0; rg < RG; ++rg)
          if (p2 + c * RG + rg < cap2) items2[p2 + c * RG + rg] = make_int4(r, rg, c, 0);
    }
    carry1 += t1;
    carry2 += t2;
    carry_sc += tsc;
  }
  if (threadIdx.x == 0) {
    off1[R] = carry1;
    off2[R] = carry2;
    sc_off[R] = carry_sc;
  }
}

// ---------------------------------------------------------------- pass 1
template <typename T, int DH>
__global__ __launch_bounds__(kThreads) void k_rows_stats(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ cu_rows, const int32_t *__restrict__ row_pos,
    const int4 *__restrict__ items, const int4 *__restrict__ rinfo,
    const int64_t *__restrict__ sc_off, int64_t n_items, int Hq, int Hkv, int64_t T_total,
    int64_t M_total, int64_t SC_total, float scale, float4 *__restrict__ stats) {
  using KR = KeyRow<T, DH>;
  __shared__ uint4 s_k[2][KR::kStage];
  const int64_t item = blockIdx.x % n_items;
  const int lk = (int)(blockIdx.x / n_items);
  const int kv = lk % Hkv, l = lk / Hkv;
  const int4 it = items[item];
  const int r = it.x, rg = it.y, c = it.z;
  const int4 info = rinfo[r];
  const int KC = info.x, pmax = info.w;
  const int g = Hq / Hkv;
  const RowSet rs = row_set(cu_rows, r, rg, g);
  const int lane = threadIdx.x & 63, col = lane & 31;

  uint4 a[KR::kSteps];
  load_query_frags<T, DH>(q, rs, l, kv, g, Hq, M_total, a);
  int prow[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int rho = rs.tile0 + acc_row(lane, v);
    prow[v] = rho < rs.nrows ? row_pos[rs.m0 + rho % rs.M] : -1;
  }

  const int64_t tok0 = cu_seqlens[r];
  const int kb = c * kCH;
  const int ke = min(kb + kCH, pmax + 1);
  const int nk = ke - kb;
  const int vlo = vis_start[r], vhi = vlo + (cu_vis[r + 1] - cu_vis[r]);
  const int64_t kstride = (int64_t)Hkv * DH * sizeof(T);
  const char *kbase = reinterpret_cast<const char *>(k + (((int64_t)l * T_total + tok0 + kb) * Hkv + kv) * DH);

  float mx[16], z[16], vz[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    mx[v] = -INFINITY;
    z[v] = 0.f;
    vz[v] = 0.f;
  }

  Stager<T, DH> stg;
  stg.load(kbase, kstride, 0, nk);
  stg.store(s_k[0]);
  __syncthreads();
  const int nst = (nk + kSub - 1) / kSub;
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) stg.load(kbase, kstride, (st + 1) * kSub, nk - (st + 1) * kSub);
    if (rs.active) {
      f32x16_t c0, c1;
      stage_dots<T, DH>(s_k[st & 1], a, c0, c1);
      const int j0 = kb + st * kSub + col, j1 = j0 + 32;
      const bool v0 = j0 >= vlo && j0 < vhi, v1 = j1 >= vlo && j1 < vhi;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float x0 = (j0 <= prow[v] && j0 < ke) ? c0[v] * scale : -INFINITY;
        const float x1 = (j1 <= prow[v] && j1 < ke) ? c1[v] * scale : -INFINITY;
        online_add(x0, v0, mx[v], z[v], vz[v]);
        online_add(x1, v1, mx[v], z[v], vz[v]);
      }
    }
    if (st + 1 < nst) stg.store(s_k[(st + 1) & 1]);
    __syncthreads();
  }
  if (!rs.active) return;

  // merge the 32 lanes of each half (they hold the same rows, other keys)
#pragma unroll
  for (int v = 0; v < 16; ++v) {
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
      const float m2 = __shfl_xor(mx[v], o), z2 = __shfl_xor(z[v], o), v2 = __shfl_xor(vz[v], o);
      online_merge(mx[v], z[v], vz[v], m2, z2, v2);
    }
  }
  if (col == 0) {
    float4 *st_base = stats + (int64_t)l * SC_total + sc_off[r];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int rho = rs.tile0 + acc_row(lane, v);
      if (rho < rs.nrows) {
        const int hh = rho / rs.M, m = rho - hh * rs.M;
        st_base[((int64_t)(kv * g + hh) * rs.M + m) * KC + c] = make_float4(mx[v], z[v], vz[v], 0.f);
      }
    }
  }
}

// ---------------------------------------------------------------- merge
__global__ __launch_bounds__(256) void k_rows_merge(
    const float4 *__restrict__ stats, const int32_t *__restrict__ cu_rows,
    const int4 *__restrict__ rinfo, const int64_t *__restrict__ sc_off, int G, int Hq,
    int64_t M_total, int64_t SC_total, float2 *__restrict__ rowstat, float *__restrict__ mass) {
  __shared__ float s_red[4];
  const int r = blockIdx.x;
  const int m0 = cu_rows[r], M = cu_rows[r + 1] - m0;
  const int KC = rinfo[r].x;
  const int per_layer = Hq * M;
  float part = 0.f;
  for (int e = threadIdx.x; e < G * per_layer; e += 256) {
    const int l = e / per_layer, rem = e - l * per_layer;
    const int h = rem / M, m = rem - h * M;
    const float4 *st = stats + (int64_t)l * SC_total + sc_off[r] + (int64_t)rem * KC;
    float mx = -INFINITY, z = 0.f, vz = 0.f;
    for (int c = 0; c < KC; ++c) {
      const float4 x = st[c];
      online_merge(mx, z, vz, x.x, x.y, x.z);
    }
    rowstat[((int64_t)l * Hq + h) * M_total + m0 + m] = make_float2(mx, 1.0f / z);
    part += vz / z;
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = part;
  __syncthreads();
  if (threadIdx.x == 0) mass[r] = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
}

// ---------------------------------------------------------------- pass 2
template <typename T, int DH>
__global__ __launch_bounds__(kThreads) void k_rows_visual(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ cu_rows, const int32_t *__restrict__ row_pos,
    const int4 *__restrict__ items, const int4 *__restrict__ rinfo, int64_t n_items, int Hq,
    int Hkv, int64_t T_total, int64_t M_total, int64_t N_total, int RG_max, float scale,
    const float2 *__restrict__ rowstat, float *__restrict__ part) {
  using KR = KeyRow<T, DH>;
  __shared__ uint4 s_k[2][KR::kStage];
  __shared__ float s_col[last::kRowWaves][kCH];
  const int64_t item = blockIdx.x % n_items;
  const int lk = (int)(blockIdx.x / n_items);
  const int kv = lk % Hkv, l = lk / Hkv;
  const int4 it = items[item];
  const int r = it.x, rg = it.y, c = it.z;
  const int pmax = rinfo[r].w;
  const int g = Hq / Hkv;
  const RowSet rs = row_set(cu_rows, r, rg, g);
  const int lane = threadIdx.x & 63, col = lane & 31, wave = threadIdx.x >> 6;

  uint4 a[KR::kSteps];
  load_query_frags<T, DH>(q, rs, l, kv, g, Hq, M_total, a);
  int prow[16];
  float rm[16], riz[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int rho = rs.tile0 + acc_row(lane, v);
    prow[v] = -1;
    rm[v] = 0.f;
    riz[v] = 0.f;
    if (rho < rs.nrows) {
      const int hh = rho / rs.M, m = rho - hh * rs.M;
      prow[v] = row_pos[rs.m0 + m];
      const float2 x = rowstat[((int64_t)l * Hq + kv * g + hh) * M_total + rs.m0 + m];
      rm[v] = x.x;
      riz[v] = x.y;
    }
  }

  const int vlo = vis_start[r];
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int seen = min(N, pmax - vlo + 1);
  const int ib = c * kCH;                        // first visual token of the chunk
  const int nk = min(kCH, seen - ib);
  const int64_t tok0 = cu_seqlens[r];
  const int64_t kstride = (int64_t)Hkv * DH * sizeof(T);
  const char *kbase =
      reinterpret_cast<const char *>(k + (((int64_t)l * T_total + tok0 + vlo + ib) * Hkv + kv) * DH);

  Stager<T, DH> stg;
  stg.load(kbase, kstride, 0, nk);
  stg.store(s_k[0]);
  __syncthreads();
  const int nst = (nk + kSub - 1) / kSub;
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) stg.load(kbase, kstride, (st + 1) * kSub, nk - (st + 1) * kSub);
    float s0 = 0.f, s1 = 0.f;
    if (rs.active) {
      f32x16_t c0, c1;
      stage_dots<T, DH>(s_k[st & 1], a, c0, c1);
      const int j0 = vlo + ib + st * kSub + col, j1 = j0 + 32;   // key positions
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s0 += j0 <= prow[v] ? expf(c0[v] * scale - rm[v]) * riz[v] : 0.f;
        s1 += j1 <= prow[v] ? expf(c1[v] * scale - rm[v]) * riz[v] : 0.f;
      }
      // the other half of the wave holds the other 16 rows of the same keys
      s0 += __shfl_xor(s0, 32);
      s1 += __shfl_xor(s1, 32);
    }
    s_col[wave][st * kSub + lane] = (lane < 32) ? s0 : s1;
    if (st + 1 < nst) stg.store(s_k[(st + 1) & 1]);
    __syncthreads();
  }
  float *out = part + (((int64_t)l * Hkv + kv) * RG_max + rg) * N_total + n0 + ib;
  for (int t = threadIdx.x; t < nk; t += kThreads) {
    float x = s_col[0][t];
#pragma unroll
    for (int w = 1; w < last::kRowWaves; ++w) x += s_col[w][t];
    out[t] = x;
  }
}

// ---------------------------------------------------------------- finalize
__global__ __launch_bounds__(256) void k_rows_finalize(
    const float *__restrict__ part, const float *__restrict__ mass, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ vis_start, const int4 *__restrict__ rinfo, int R, int G, int Hkv,
    int RG_max, int64_t N_total, float *__restrict__ scores) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n >= N_total) return;
  int lo = 0, hi = R - 1;                        // request holding visual token n
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_vis[mid] <= n) lo = mid;
    else hi = mid - 1;
  }
  const int r = lo;
  const int4 info = rinfo[r];
  const int i = (int)(n - cu_vis[r]);
  const int N = cu_vis[r + 1] - cu_vis[r];
  const int seen = min(N, info.w - vis_start[r] + 1);
  if (i >= seen) {
    scores[n] = 0.f;
    return;
  }
  float s = 0.f;
  for (int l = 0; l < G; ++l)
    for (int kv = 0; kv < Hkv; ++kv)
      for (int rg = 0; rg < info.z; ++rg) s += part[(((int64_t)l * Hkv + kv) * RG_max + rg) * N_total + n];
  scores[n] = s / mass[r];
}

template <typename T, int DH>
hipError_t launch_passes(const last_batch *b, const last::RowsPlan &p, const last::RowsWs &w,
                         const int32_t *cu_rows, const int32_t *row_pos, const void *q,
                         const void *k, float scale, hipStream_t s) {
  const int64_t blocks1 = (int64_t)b->G * b->Hkv * p.items1;
  const int64_t blocks2 = (int64_t)b->G * b->Hkv * p.items2;
  last::launch_begin("rows_stats", s);
  hipLaunchKernelGGL((k_rows_stats<T, DH>), dim3((unsigned)blocks1), dim3(kThreads), 0, s,
                     (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis, cu_rows,
                     row_pos, w.items1, w.rinfo, w.sc_off, p.items1, b->Hq, b->Hkv, p.T_total,
                     p.M_total, p.SC_total, scale, w.stats);
  hipError_t e = last::launch_end(s);
  if (e != hipSuccess) return e;

  last::launch_begin("rows_merge", s);
  hipLaunchKernelGGL(k_rows_merge, dim3((unsigned)b->R), dim3(256), 0, s, w.stats, cu_rows, w.rinfo,
                     w.sc_off, b->G, b->Hq, p.M_total, p.SC_total, w.rowstat, w.mass);
  e = last::launch_end(s);
  if (e != hipSuccess) return e;

  last::launch_begin("rows_visual", s);
  hipLaunchKernelGGL((k_rows_visual<T, DH>), dim3((unsigned)blocks2), dim3(kThreads), 0, s,
                     (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis, cu_rows,
                     row_pos, w.items2, w.rinfo, p.items2, b->Hq, b->Hkv, p.T_total, p.M_total,
                     p.N_total, p.RG_max, scale, w.rowstat, w.part);
  return last::launch_end(s);
}

}  // namespace

namespace last {

RowsPlan make_rows_plan(const last_batch *b, const int32_t *cu_rows_h, const int32_t *row_pos_h) {
  RowsPlan p{};
  const int g = b->Hq / b->Hkv;
  p.M_total = cu_rows_h[b->R];
  p.N_total = b->cu_vis_h[b->R];
  p.T_total = b->cu_seqlens_h[b->R];
  for (int r = 0; r < b->R; ++r) {
    const int M = cu_rows_h[r + 1] - cu_rows_h[r];
    int pmax = 0;
    for (int m = 0; m < M; ++m) pmax = std::max(pmax, row_pos_h[cu_rows_h[r] + m]);
    const int tiles = (g * M + 31) / 32;
    const int RG = (tiles + kRowWaves - 1) / kRowWaves;
    const int KC = (pmax + 1 + kRowChunk - 1) / kRowChunk;
    const int N = b->cu_vis_h[r + 1] - b->cu_vis_h[r];
    const int seen = std::min(N, pmax - b->vis_start_h[r] + 1);
    const int VC = (seen + kRowChunk - 1) / kRowChunk;
    p.items1 += (int64_t)RG * KC;
    p.items2 += (int64_t)RG * VC;
    p.SC_total += (int64_t)b->Hq * M * KC;
    p.RG_max = std::max(p.RG_max, RG);
  }
  return p;
}

RowsWs carve_rows_ws(void *ws, const last_batch *b, const RowsPlan &p, size_t *bytes) {
  Carver cv(ws);
  RowsWs w{};
  w.off1 = cv.take<int32_t>(b->R + 1);
  w.off2 = cv.take<int32_t>(b->R + 1);
  w.sc_off = cv.take<int64_t>(b->R + 1);
  w.rinfo = cv.take<int4>(b->R);
  w.items1 = cv.take<int4>(p.items1);
  w.items2 = cv.take<int4>(p.items2);
  w.stats = cv.take<float4>((size_t)b->G * p.SC_total);
  w.rowstat = cv.take<float2>((size_t)b->G * b->Hq * p.M_total);
  w.mass = cv.take<float>(b->R);
  w.part = cv.take<float>((size_t)b->G * b->Hkv * p.RG_max * p.N_total);
  *bytes = cv.size();
  return w;
}

hipError_t launch_rows(const last_batch *b, const RowsPlan &p, const RowsWs &w,
                       const int32_t *cu_rows, const int32_t *row_pos, const void *q,
                       const void *k, float *scores, float scale, hipStream_t s) {
  const int g = b->Hq / b->Hkv;
  launch_begin("rows_plan", s);
  hipLaunchKernelGGL(k_rows_plan, dim3(1), dim3(256), 0, s, b->cu_seqlens, b->vis_start, b->cu_vis,
                     cu_rows, row_pos, b->R, b->Hq, g, p.items1, p.items2, w.off1, w.off2, w.sc_off,
                     w.rinfo, w.items1, w.items2);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;

  const bool bf = b->qk_dtype == LAST_BF16;
  e = bf ? (b->Dh == 64 ? launch_passes<uint16_t, 64>(b, p, w, cu_rows, row_pos, q, k, scale, s)
                        : launch_passes<uint16_t, 128>(b, p, w, cu_rows, row_pos, q, k, scale, s))
         : (b->Dh == 64 ? launch_passes<float, 64>(b, p, w, cu_rows, row_pos, q, k, scale, s)
                        : launch_passes<float, 128>(b, p, w, cu_rows, row_pos, q, k, scale, s));
  if (e != hipSuccess) return e;

  launch_begin("rows_finalize", s);
  hipLaunchKernelGGL(k_rows_finalize, dim3((unsigned)((p.N_total + 255) / 256)), dim3(256), 0, s,
                     w.part, w.mass, b->cu_vis, b->vis_start, w.rinfo, b->R, b->G, b->Hkv, p.RG_max,
                     p.N_total, scores);
  return launch_end(s);
}

}  // namespace last
