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
//                    chunk): the chunk's keys staged into LDS 128 at a time by
//                    LDS DMA, one stage in flight while the other is used;
//                    each wave multiplies one 32-row query tile by its share of
//                    every stage. Each lane keeps, for the 16 rows of its
//                    accumulator, a reference r and the sums of 2^(x - r) over
//                    all keys and over the visual ones, x being the logit in
//                    base-2 units (the softmax scale times log2 e folded into
//                    one multiply). The reference only moves when a logit
//                    exceeds it by 64 (sums stay far from overflow), so a logit
//                    costs one exponential and no rescaling.
//   k_rows_merge     one thread per row, 256 rows a block: every row's chunks
//                    merged into one reference and 1/Z, and the block's share
//                    of the visual mass S = sum V / Z over the request's rows
//                    (= sum_i s_i); k_rows_mass adds the shares per request.
//   k_rows_visual    one block per (layer, KV head, request, row group, visual
//                    chunk): the visual logits again, 2^(x - r) / Z summed over
//                    the block's rows per key, written per row group.
//   k_rows_finalize  one thread per visual token: the row-group sums over
//                    layers and KV heads in a fixed order, divided by S.
//
// Stages whose keys every row of a wave sees (all of them except near the
// rows themselves) skip the causal mask; stages wholly inside or outside the
// visual span skip the per-key visual test. Every reduction has a fixed
// order, so results are bitwise reproducible.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kW = last::kRowWaves;
constexpr int kThreads = 64 * kW;
constexpr int kSub = 128;                     // keys per LDS stage: four 32-key tiles
constexpr int kCH = last::kRowChunk;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSlack = 64.f;                // a reference may trail its row's max by this much
constexpr float kNoRef = -1e30f;              // the reference of a row that has seen no key yet
static_assert(kCH % kSub == 0, "whole stages per chunk");

// A key (or query) row of DH elements as 16-byte pieces. One matrix-core step
// takes one piece from each half of the wave: lanes 0-31 piece 2s, lanes
// 32-63 piece 2s + 1 (8 bf16 -> one 32x32x16 MFMA; 4 fp32 -> four 32x32x2).
template <typename T, int DH>
struct KeyRow {
  static constexpr int kPieces = DH * (int)sizeof(T) / 16;
  static constexpr int kSteps = kPieces / 2;
  static constexpr int kStage = kSub * kPieces;           // pieces per LDS stage
  static_assert(kPieces >= 8 && kStage % (64 * kW) == 0, "row shape");
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

// 2^x on the transcendental unit (results below 2^-126 flush to zero).
__device__ __forceinline__ float pow2(float x) { return __builtin_amdgcn_exp2f(x); }

// In a 32 x 32 accumulator lane l holds column l % 32 and, at element v, row
// 4 * (l / 32) + (v % 4) + 8 * (v / 4).
__device__ __forceinline__ int acc_row(int lane, int v) { return 4 * (lane >> 5) + (v & 3) + 8 * (v >> 2); }

// The block's place in its request: wave w multiplies row tile w % RT of the
// row group and key tiles w / RT, w / RT + KS, ... of every stage
// (KS = kW / RT waves share a row tile). Row rho of a KV head's set is query
// head kv * g + rho / M, query row rho % M.
template <int RT>
struct Place {
  static constexpr int KS = kW / RT;
  int m0, M, nrows, rt, ks, tile0;
  bool active;   // the wave's row tile has at least one real row
  __device__ Place(const int32_t *cu_rows, int r, int rg, int g) {
    m0 = cu_rows[r];
    M = cu_rows[r + 1] - m0;
    nrows = g * M;
    const int w = (int)(threadIdx.x >> 6);
    rt = w % RT;
    ks = w / RT;
    tile0 = (rg * RT + rt) * 32;
    active = tile0 < nrows;
  }
};

template <typename T, int DH, int RT>
__device__ __forceinline__ void load_query_frags(const T *q, const Place<RT> &pl, int l, int kv, int g,
                                                 int Hq, int64_t M_total,
                                                 uint4 (&a)[KeyRow<T, DH>::kSteps]) {
  const int lane = threadIdx.x & 63;
  const int rho = pl.tile0 + (lane & 31);
  if (rho < pl.nrows) {
    const int hh = rho / pl.M, m = rho - hh * pl.M;
    const char *qp = reinterpret_cast<const char *>(q + (((int64_t)l * M_total + pl.m0 + m) * Hq + kv * g + hh) * DH);
#pragma unroll
    for (int st = 0; st < KeyRow<T, DH>::kSteps; ++st)
      a[st] = *reinterpret_cast<const uint4 *>(qp + (2 * st + (lane >> 5)) * 16);
  } else {
#pragma unroll
    for (int st = 0; st < KeyRow<T, DH>::kSteps; ++st) a[st] = make_uint4(0, 0, 0, 0);
  }
}

// Keys of one KV head into the LDS stages by LDS DMA (no registers hold
// them): wave w issues instructions w, w + kW, ... of a stage, each filling
// 64 consecutive 16-byte slots; a slot's lane fetches the piece the swizzle
// puts there. Instruction n + kPat covers the rows of instruction n moved by
// a multiple of the swizzle's period, so a lane's offsets within a stage take
// kPat registers, worked out once; the rest is wave-uniform.
template <typename T, int DH>
struct KeyStager {
  static constexpr int NP = KeyRow<T, DH>::kPieces;
  static constexpr int kN = KeyRow<T, DH>::kStage / 64 / kW;
  static constexpr int kRowsPer = 64 * kW / NP;              // stage rows one instruction covers
  static constexpr int kPat = NP >= 16 ? NP / 16 : 1;        // swizzle period 16 rows
  static_assert(kN % kPat == 0 && (kPat * kRowsPer) % 16 == 0, "swizzle period");
  uint32_t roff[kPat];   // byte offsets of this lane's piece from the stage's first key
  uint32_t dst0;         // LDS address of this wave's first slot in stage buffer 0
  __device__ static void place(int n, int &j, int &p) {
    const int sl = ((int)(threadIdx.x >> 6) + kW * n) * 64 + (int)(threadIdx.x & 63);
    j = sl / NP;
    p = (sl % NP) ^ (NP >= 16 ? (j & 15) : ((j >> 1) & 7));
  }
  // kstride * kSub < 2^32: a batch has at most 4096 (layer, head) pairs, so
  // a token's keys take at most 4096 x 128 x 4 bytes
  __device__ KeyStager(const uint4 *buf0, int64_t kstride) {
#pragma unroll
    for (int n = 0; n < kPat; ++n) {
      int j, p;
      place(n, j, p);
      roff[n] = (uint32_t)(j * kstride + p * 16);
    }
    dst0 = __builtin_amdgcn_readfirstlane(lds_u32(buf0 + (threadIdx.x >> 6) * 64));
  }
  // Keys [j0, j0 + kSub) of the chunk at kbase (nk keys) into stage buffer
  // b; slots at or past key nk repeat key nk - 1 (callers never use them).
  // kbase must be wave-uniform.
  __device__ void issue(int b, const char *kbase, int64_t kstride, int j0, int nk) const {
    const uint32_t d = dst0 + (uint32_t)b * (KeyRow<T, DH>::kStage * 16);
    if (j0 + kSub <= nk) {
#pragma unroll
      for (int n = 0; n < kN; ++n) {
        const char *base = (const char *)uniform_ptr(kbase + (int64_t)(j0 + n / kPat * kPat * kRowsPer) * kstride);
        dma16(d + n * (kW * 64 * 16), base, roff[n % kPat]);
      }
    } else {
      const char *base = (const char *)uniform_ptr(kbase + (int64_t)j0 * kstride);
      const int last = nk - 1 - j0;
#pragma unroll
      for (int n = 0; n < kN; ++n) {
        int j, p;
        place(n, j, p);
        dma16(d + n * (kW * 64 * 16), base, (uint32_t)(min(j, last) * kstride + p * 16));
      }
    }
  }
};

// Dots (unscaled logits) of the wave's 32 query rows with the 32 keys of
// stage key tile kt.
template <typename T, int DH>
__device__ __forceinline__ void tile_dots(const uint4 *buf, const uint4 (&a)[KeyRow<T, DH>::kSteps], int kt,
                                          f32x16_t &c) {
  using KR = KeyRow<T, DH>;
  const int lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  c = f32x16_t{};
#pragma unroll
  for (int st = 0; st < KR::kSteps; ++st) mma_piece(c, a[st], buf[slot<KR::kPieces>(kt * 32 + col, 2 * st + half)], T());
}

// Scheduling of one pipelined tile: the next tile's fragment reads and
// matrix-core steps spread through this tile's vector work (NV vector
// instructions per step), so that the two overlap.
template <typename T, int DH, int NV>
__device__ __forceinline__ void interleave_hint() {
  constexpr int kMfma = KeyRow<T, DH>::kSteps * (sizeof(T) == 2 ? 1 : 4);
  constexpr int kDs = KeyRow<T, DH>::kSteps;
  __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
  for (int i = 0; i < kMfma; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i * kDs / kMfma + 2 < kDs && (i * kDs) % kMfma == 0) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, NV, 0);
  }
}

// Combine two (reference, sum, visual sum) triples in base 2. References are
// finite (kNoRef for a row that has seen no key: its sums are 0).
__device__ __forceinline__ void merge2(float &m, float &z, float &vz, float m2, float z2, float v2) {
  const float M = fmaxf(m, m2);
  const float f1 = pow2(m - M), f2 = pow2(m2 - M);
  z = z * f1 + z2 * f2;
  vz = vz * f1 + v2 * f2;
  m = M;
}

// Wave-uniform minimum of the real row positions in this lane's accumulator
// rows (positions are < 2^24, exact in fp32).
__device__ __forceinline__ int wave_min_pos(const int (&prow)[16]) {
  int mn = 1 << 24;
#pragma unroll
  for (int v = 0; v < 16; ++v)
    if (prow[v] >= 0) mn = min(mn, prow[v]);
  return (int)(-wave_max(-(float)mn));
}

// ---------------------------------------------------------------- plan
__global__ __launch_bounds__(256) void k_rows_plan(
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ vis_start,
    const int32_t *__restrict__ cu_vis, const int32_t *__restrict__ cu_rows,
    const int32_t *__restrict__ row_pos, int R, int Hq, int g, int RT, int64_t cap1, int64_t cap2,
    int32_t *__restrict__ off1, int32_t *__restrict__ off2, int64_t *__restrict__ sc_off,
    int4 *__restrict__ rinfo, int4 *__restrict__ items1, int4 *__restrict__ items2) {
  __shared__ int sh[4];
  __shared__ long long s_sc[256];
  __shared__ int s_p1[256], s_p2[256], s_kc[256], s_vc[256], s_rg[256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int carry1 = 0, carry2 = 0;
  long long carry_sc = 0;
  for (int base = 0; base < R; base += 256) {
    const int r = base + (int)threadIdx.x;
    int n1 = 0, n2 = 0, KC = 0, VC = 0, RG = 0, pmax = 0;
    long long nsc = 0;
    // each request's last row position: a wave per request, lanes over its rows
    for (int j = wave; j < min(256, R - base); j += 4) {
      const int m0 = cu_rows[base + j], M = cu_rows[base + j + 1] - m0;
      int pm = 0;
      for (int m = lane; m < M; m += 64) pm = max(pm, row_pos[m0 + m]);
      pm = (int)wave_max_u32((uint32_t)pm);
      if (lane == 0) s_kc[j] = pm;
    }
    __syncthreads();
    if (r < R) {
      const int m0 = cu_rows[r], M = cu_rows[r + 1] - m0;
      pmax = s_kc[threadIdx.x];
      const int tiles = (g * M + 31) / 32;
      RG = (tiles + RT - 1) / RT;
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
    }
    s_p1[threadIdx.x] = p1;
    s_p2[threadIdx.x] = p2;
    s_kc[threadIdx.x] = KC;
    s_vc[threadIdx.x] = VC;
    s_rg[threadIdx.x] = RG;
    __syncthreads();
    // the work items, chunk-major then row group: a wave per request
    for (int j = wave; j < min(256, R - base); j += 4) {
      const int rg_n = s_rg[j], q1 = s_p1[j], q2 = s_p2[j];
      for (int x = lane; x < s_kc[j] * rg_n; x += 64)
        if (q1 + x < cap1) items1[q1 + x] = make_int4(base + j, x % rg_n, x / rg_n, 0);
      for (int x = lane; x < s_vc[j] * rg_n; x += 64)
        if (q2 + x < cap2) items2[q2 + x] = make_int4(base + j, x % rg_n, x / rg_n, 0);
    }
    __syncthreads();
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
// two blocks a CU for bf16 keys; fp32 keys need the registers of one
template <typename T, int DH, int RT>
__global__ __launch_bounds__(kThreads, sizeof(T) == 2 ? 2 : 1) void k_rows_stats(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ cu_rows, const int32_t *__restrict__ row_pos,
    const int4 *__restrict__ items, const int4 *__restrict__ rinfo,
    const int64_t *__restrict__ sc_off, int64_t n_items, int Hq, int Hkv, int64_t T_total,
    int64_t M_total, int64_t SC_total, float scale2, float4 *__restrict__ stats) {
  using KR = KeyRow<T, DH>;
  constexpr int KS = kW / RT;
  __shared__ uint4 s_k[2][KR::kStage];
  __shared__ float4 s_st[kW][32];
  __shared__ int s_pos[kW][32];     // position of each row of a wave's tile (-1: none)
  // the row groups of one key chunk are neighbouring items: XCD-contiguous
  // numbering runs them on one XCD, where they share the chunk in L2
  const int64_t bid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int64_t item = bid % n_items;
  const int lk = (int)(bid / n_items);
  const int kv = lk % Hkv, l = lk / Hkv;
  const int4 it = items[item];
  const int r = it.x, rg = it.y, c = it.z;
  const int4 info = rinfo[r];
  const int KC = info.x, pmax = info.w;
  const int g = Hq / Hkv;
  const Place<RT> pl(cu_rows, r, rg, g);
  const int lane = threadIdx.x & 63, col = lane & 31, wave = threadIdx.x >> 6;

  uint4 a[KR::kSteps];
  load_query_frags<T, DH, RT>(q, pl, l, kv, g, Hq, M_total, a);
  int pmin;
  {
    int prow[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int rho = pl.tile0 + acc_row(lane, v);
      prow[v] = rho < pl.nrows ? row_pos[pl.m0 + rho % pl.M] : -1;
    }
    pmin = wave_min_pos(prow);
    if (lane < 32) {
      const int rho = pl.tile0 + lane;
      s_pos[wave][lane] = rho < pl.nrows ? row_pos[pl.m0 + rho % pl.M] : -1;
    }
  }

  const int64_t tok0 = cu_seqlens[r];
  const int kb = c * kCH;
  const int ke = min(kb + kCH, pmax + 1);
  const int nk = ke - kb;
  const int vlo = vis_start[r], vhi = vlo + (cu_vis[r + 1] - cu_vis[r]);
  const int64_t kstride = (int64_t)Hkv * DH * sizeof(T);
  const char *kbase = (const char *)uniform_ptr(k + (((int64_t)l * T_total + tok0 + kb) * Hkv + kv) * DH);

  float mr[16], z[16], vz[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    mr[v] = kNoRef;
    z[v] = 0.f;
    vz[v] = 0.f;
  }

  const KeyStager<T, DH> stager(s_k[0], kstride);
  stager.issue(0, kbase, kstride, 0, nk);
  vm_wait<0>();
  __syncthreads();
  const int nst = (nk + kSub - 1) / kSub;
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) stager.issue((st + 1) & 1, kbase, kstride, (st + 1) * kSub, nk);
    if (pl.active) {
      const int s0 = kb + st * kSub;                         // first key position of the stage
      const int s1 = s0 + kSub - 1;                          // last
      // every row of the wave sees every key of the stage, all keys exist
      const bool full = s1 <= pmin && s1 < ke;
      const bool allvis = s0 >= vlo && s1 < vhi, novis = s1 < vlo || s0 >= vhi;
      const uint4 *buf = s_k[st & 1];
      f32x16_t cur, nxt;
      tile_dots<T, DH>(buf, a, pl.ks, cur);
      // Per tile: the next tile's matrix-core steps run under this tile's
      // exponentials. A term whose logit passes its row's reference by more
      // than the slack is held back and folded in afterwards with a new
      // reference (rare: the first key a row sees, or a jump of 2^64). The
      // masked and unmasked loops are separate, so that neither branches.
      auto fold_big = [&](int j, float vis) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const bool live = full || (j <= s_pos[wave][acc_row(lane, v)] && j < ke);
          const float x = cur[v] * scale2;
          const bool b = live && x - mr[v] > kSlack;
          const float f = pow2(mr[v] - x);
          z[v] = b ? fmaf(z[v], f, 1.f) : z[v];
          vz[v] = b ? fmaf(vz[v], f, vis) : vz[v];
          mr[v] = b ? x : mr[v];
        }
      };
      if (full) {
#pragma unroll
        for (int i = 0; i < RT; ++i) {
          const int j = s0 + (pl.ks + KS * i) * 32 + col;
          const float vis = allvis ? 1.f : (novis ? 0.f : ((j >= vlo && j < vhi) ? 1.f : 0.f));
          if (i + 1 < RT) tile_dots<T, DH>(buf, a, pl.ks + KS * (i + 1), nxt);
          bool big = false;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float d = fmaf(cur[v], scale2, -mr[v]);
            const bool b = d > kSlack;
            const float e = pow2(b ? -INFINITY : d);
            z[v] += e;
            vz[v] = fmaf(e, vis, vz[v]);
            big |= b;
          }
          if (i + 1 < RT) interleave_hint<T, DH, 8>();
          if (__any(big)) fold_big(j, vis);
          if (i + 1 < RT) cur = nxt;
        }
      } else {
#pragma unroll
        for (int i = 0; i < RT; ++i) {
          const int j = s0 + (pl.ks + KS * i) * 32 + col;
          const float vis = (j >= vlo && j < vhi) ? 1.f : 0.f;
          if (i + 1 < RT) tile_dots<T, DH>(buf, a, pl.ks + KS * (i + 1), nxt);
          bool big = false;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const bool live = j <= s_pos[wave][acc_row(lane, v)] && j < ke;
            const float d = live ? fmaf(cur[v], scale2, -mr[v]) : -INFINITY;
            const bool b = d > kSlack;
            const float e = pow2(b ? -INFINITY : d);
            z[v] += e;
            vz[v] = fmaf(e, vis, vz[v]);
            big |= b;
          }
          if (i + 1 < RT) interleave_hint<T, DH, 10>();
          if (__any(big)) fold_big(j, vis);
          if (i + 1 < RT) cur = nxt;
        }
      }
    }
    vm_wait<0>();
    __syncthreads();
  }

  // merge the 32 lanes of each half (same rows, other keys), then the KS
  // waves that share a row tile, in a fixed order
  if (pl.active) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) {
        const float m2 = __shfl_xor(mr[v], o), z2 = __shfl_xor(z[v], o), v2 = __shfl_xor(vz[v], o);
        merge2(mr[v], z[v], vz[v], m2, z2, v2);
      }
    }
    if (col == 0)
#pragma unroll
      for (int v = 0; v < 16; ++v) s_st[wave][acc_row(lane, v)] = make_float4(mr[v], z[v], vz[v], 0.f);
  }
  __syncthreads();
  if ((int)threadIdx.x < RT * 32) {
    const int rt = threadIdx.x / 32, x = threadIdx.x % 32;
    const int rho = (rg * RT + rt) * 32 + x;
    if (rho < pl.nrows) {
      float4 acc = s_st[rt][x];
#pragma unroll
      for (int s = 1; s < KS; ++s) {
        const float4 e = s_st[rt + RT * s][x];
        merge2(acc.x, acc.y, acc.z, e.x, e.y, e.z);
      }
      const int hh = rho / pl.M, m = rho - hh * pl.M;
      stats[(int64_t)l * SC_total + sc_off[r] + ((int64_t)(kv * g + hh) * pl.M + m) * KC + c] = acc;
    }
  }
}

// ---------------------------------------------------------------- merge
// Grid (MB, R): block (x, r) merges rows x * 256 .. x * 256 + 255 of request
// r, one row a thread, and writes their visual mass V / Z summed in a fixed
// order as part x of the request's mass; k_rows_mass adds the parts.
__global__ __launch_bounds__(256) void k_rows_merge(
    const float4 *__restrict__ stats, const int32_t *__restrict__ cu_rows,
    const int4 *__restrict__ rinfo, const int64_t *__restrict__ sc_off, int G, int Hq,
    int64_t M_total, int64_t SC_total, float2 *__restrict__ rowstat, float *__restrict__ mass_part) {
  __shared__ float s_red[4];
  const int r = blockIdx.y;
  const int m0 = cu_rows[r], M = cu_rows[r + 1] - m0;
  const int KC = rinfo[r].x;
  const int per_layer = Hq * M;
  float part = 0.f;
  const int e = blockIdx.x * 256 + (int)threadIdx.x;
  if (e < G * per_layer) {
    const int l = e / per_layer, rem = e - l * per_layer;
    const int h = rem / M, m = rem - h * M;
    const float4 *st = stats + (int64_t)l * SC_total + sc_off[r] + (int64_t)rem * KC;
    float mx = kNoRef, z = 0.f, vz = 0.f;
    for (int c = 0; c < KC; ++c) {
      const float4 x = st[c];
      merge2(mx, z, vz, x.x, x.y, x.z);
    }
    rowstat[((int64_t)l * Hq + h) * M_total + m0 + m] = make_float2(mx, 1.0f / z);
    part = vz / z;
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = part;
  __syncthreads();
  if (threadIdx.x == 0) mass_part[(int64_t)r * gridDim.x + blockIdx.x] = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
}

// A request's visual mass: its MB merge parts, lane-strided and then across
// the wave, in a fixed order.
__global__ __launch_bounds__(64) void k_rows_mass(const float *__restrict__ mass_part, int MB,
                                                  float *__restrict__ mass) {
  const int r = blockIdx.x;
  float s = 0.f;
  for (int x = threadIdx.x; x < MB; x += 64) s += mass_part[(int64_t)r * MB + x];
  s = wave_sum(s);
  if (threadIdx.x == 0) mass[r] = s;
}

// ---------------------------------------------------------------- pass 2
// two blocks a CU for bf16 keys; fp32 keys need the registers of one
template <typename T, int DH, int RT>
__global__ __launch_bounds__(kThreads, sizeof(T) == 2 ? 2 : 1) void k_rows_visual(
    const T *__restrict__ q, const T *__restrict__ k, const int32_t *__restrict__ cu_seqlens,
    const int32_t *__restrict__ vis_start, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ cu_rows, const int32_t *__restrict__ row_pos,
    const int4 *__restrict__ items, const int4 *__restrict__ rinfo, int64_t n_items, int Hq,
    int Hkv, int64_t T_total, int64_t M_total, int64_t N_total, int RG_max, float scale2,
    const float2 *__restrict__ rowstat, float *__restrict__ part) {
  using KR = KeyRow<T, DH>;
  constexpr int KS = kW / RT;
  __shared__ uint4 s_k[2][KR::kStage];
  __shared__ float s_col[RT][kCH];
  // the row groups of one key chunk are neighbouring items: XCD-contiguous
  // numbering runs them on one XCD, where they share the chunk in L2
  const int64_t bid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int64_t item = bid % n_items;
  const int lk = (int)(bid / n_items);
  const int kv = lk % Hkv, l = lk / Hkv;
  const int4 it = items[item];
  const int r = it.x, rg = it.y, c = it.z;
  const int pmax = rinfo[r].w;
  const int g = Hq / Hkv;
  const Place<RT> pl(cu_rows, r, rg, g);
  const int lane = threadIdx.x & 63, col = lane & 31;

  uint4 a[KR::kSteps];
  load_query_frags<T, DH, RT>(q, pl, l, kv, g, Hq, M_total, a);
  // per accumulator row: position, reference and 1/Z; a missing row gets an
  // infinite reference, so its terms are exactly 0
  int prow[16];
  float rm[16], riz[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int rho = pl.tile0 + acc_row(lane, v);
    prow[v] = -1;
    rm[v] = INFINITY;
    riz[v] = 0.f;
    if (rho < pl.nrows) {
      const int hh = rho / pl.M, m = rho - hh * pl.M;
      prow[v] = row_pos[pl.m0 + m];
      const float2 x = rowstat[((int64_t)l * Hq + kv * g + hh) * M_total + pl.m0 + m];
      rm[v] = x.x;
      riz[v] = x.y;
    }
  }
  const int pmin = wave_min_pos(prow);

  const int vlo = vis_start[r];
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int seen = min(N, pmax - vlo + 1);
  const int ib = c * kCH;                        // first visual token of the chunk
  const int nk = min(kCH, seen - ib);
  const int64_t tok0 = cu_seqlens[r];
  const int64_t kstride = (int64_t)Hkv * DH * sizeof(T);
  const char *kbase = (const char *)uniform_ptr(k + (((int64_t)l * T_total + tok0 + vlo + ib) * Hkv + kv) * DH);

  const KeyStager<T, DH> stager(s_k[0], kstride);
  stager.issue(0, kbase, kstride, 0, nk);
  vm_wait<0>();
  __syncthreads();
  const int nst = (nk + kSub - 1) / kSub;
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) stager.issue((st + 1) & 1, kbase, kstride, (st + 1) * kSub, nk);
    float sum[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) sum[i] = 0.f;
    if (pl.active) {
      const int s0 = vlo + ib + st * kSub;                   // key position of the stage's first key
      const bool full = s0 + kSub - 1 <= pmin;               // every row of the wave sees every key
      const uint4 *buf = s_k[st & 1];
      f32x16_t cur, nxt;
      tile_dots<T, DH>(buf, a, pl.ks, cur);
      // the next tile's matrix-core steps run under this tile's exponentials;
      // the two loops differ only in the causal mask, so that neither branches
      if (full) {
#pragma unroll
        for (int i = 0; i < RT; ++i) {
          if (i + 1 < RT) tile_dots<T, DH>(buf, a, pl.ks + KS * (i + 1), nxt);
#pragma unroll
          for (int v = 0; v < 16; ++v) sum[i] = fmaf(pow2(fmaf(cur[v], scale2, -rm[v])), riz[v], sum[i]);
          if (i + 1 < RT) {
            interleave_hint<T, DH, 6>();
            cur = nxt;
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < RT; ++i) {
          const int j = s0 + (pl.ks + KS * i) * 32 + col;
          if (i + 1 < RT) tile_dots<T, DH>(buf, a, pl.ks + KS * (i + 1), nxt);
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float x = j <= prow[v] ? fmaf(cur[v], scale2, -rm[v]) : -INFINITY;
            sum[i] = fmaf(pow2(x), riz[v], sum[i]);
          }
          if (i + 1 < RT) {
            interleave_hint<T, DH, 8>();
            cur = nxt;
          }
        }
      }
      // the other half of the wave holds the other 16 rows of the same keys
#pragma unroll
      for (int i = 0; i < RT; ++i) sum[i] += __shfl_xor(sum[i], 32);
    }
    if (lane < 32)
#pragma unroll
      for (int i = 0; i < RT; ++i) s_col[pl.rt][st * kSub + (pl.ks + KS * i) * 32 + col] = sum[i];
    vm_wait<0>();
    __syncthreads();
  }
  float *out = part + (((int64_t)l * Hkv + kv) * RG_max + rg) * N_total + n0 + ib;
  for (int t = threadIdx.x; t < nk; t += kThreads) {
    float x = s_col[0][t];
#pragma unroll
    for (int w = 1; w < RT; ++w) x += s_col[w][t];
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

template <typename T, int DH, int RT>
hipError_t launch_passes(const last_batch *b, const last::RowsPlan &p, const last::RowsWs &w,
                         const int32_t *cu_rows, const int32_t *row_pos, const void *q,
                         const void *k, float scale2, hipStream_t s) {
  const int64_t blocks1 = (int64_t)b->G * b->Hkv * p.items1;
  const int64_t blocks2 = (int64_t)b->G * b->Hkv * p.items2;
  last::launch_begin("rows_stats", s);
  hipLaunchKernelGGL((k_rows_stats<T, DH, RT>), dim3((unsigned)blocks1), dim3(kThreads), 0, s,
                     (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis, cu_rows,
                     row_pos, w.items1, w.rinfo, w.sc_off, p.items1, b->Hq, b->Hkv, p.T_total,
                     p.M_total, p.SC_total, scale2, w.stats);
  hipError_t e = last::launch_end(s);
  if (e != hipSuccess) return e;

  last::launch_begin("rows_merge", s);
  hipLaunchKernelGGL(k_rows_merge, dim3((unsigned)p.MB, (unsigned)b->R), dim3(256), 0, s, w.stats, cu_rows,
                     w.rinfo, w.sc_off, b->G, b->Hq, p.M_total, p.SC_total, w.rowstat, w.mass_part);
  hipLaunchKernelGGL(k_rows_mass, dim3((unsigned)b->R), dim3(64), 0, s, w.mass_part, p.MB, w.mass);
  e = last::launch_end(s);
  if (e != hipSuccess) return e;

  last::launch_begin("rows_visual", s);
  hipLaunchKernelGGL((k_rows_visual<T, DH, RT>), dim3((unsigned)blocks2), dim3(kThreads), 0, s,
                     (const T *)q, (const T *)k, b->cu_seqlens, b->vis_start, b->cu_vis, cu_rows,
                     row_pos, w.items2, w.rinfo, p.items2, b->Hq, b->Hkv, p.T_total, p.M_total,
                     p.N_total, p.RG_max, scale2, w.rowstat, w.part);
  return last::launch_end(s);
}

template <typename T, int DH>
hipError_t launch_rt(const last_batch *b, const last::RowsPlan &p, const last::RowsWs &w,
                     const int32_t *cu_rows, const int32_t *row_pos, const void *q, const void *k,
                     float scale2, hipStream_t s) {
  switch (p.RT) {
    case 1: return launch_passes<T, DH, 1>(b, p, w, cu_rows, row_pos, q, k, scale2, s);
    case 2: return launch_passes<T, DH, 2>(b, p, w, cu_rows, row_pos, q, k, scale2, s);
    default: return launch_passes<T, DH, 4>(b, p, w, cu_rows, row_pos, q, k, scale2, s);
  }
}

}  // namespace

namespace last {

RowsPlan make_rows_plan(const last_batch *b, const int32_t *cu_rows_h, const int32_t *row_pos_h) {
  RowsPlan p{};
  const int g = b->Hq / b->Hkv;
  p.M_total = cu_rows_h[b->R];
  p.N_total = b->cu_vis_h[b->R];
  p.T_total = b->cu_seqlens_h[b->R];
  int max_tiles = 1;
  for (int r = 0; r < b->R; ++r)
    max_tiles = std::max(max_tiles, (g * (cu_rows_h[r + 1] - cu_rows_h[r]) + 31) / 32);
  p.RT = max_tiles >= 3 ? 4 : max_tiles;
  for (int r = 0; r < b->R; ++r) {
    const int M = cu_rows_h[r + 1] - cu_rows_h[r];
    int pmax = 0;
    for (int m = 0; m < M; ++m) pmax = std::max(pmax, row_pos_h[cu_rows_h[r] + m]);
    const int tiles = (g * M + 31) / 32;
    const int RG = (tiles + p.RT - 1) / p.RT;
    const int KC = (pmax + 1 + kRowChunk - 1) / kRowChunk;
    const int N = b->cu_vis_h[r + 1] - b->cu_vis_h[r];
    const int seen = std::min(N, pmax - b->vis_start_h[r] + 1);
    const int VC = (seen + kRowChunk - 1) / kRowChunk;
    p.items1 += (int64_t)RG * KC;
    p.items2 += (int64_t)RG * VC;
    p.SC_total += (int64_t)b->Hq * M * KC;
    p.RG_max = std::max(p.RG_max, RG);
    p.MB = std::max<int32_t>(p.MB, (int32_t)(((int64_t)b->G * b->Hq * M + 255) / 256));
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
  w.mass_part = cv.take<float>((size_t)b->R * p.MB);
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
                     cu_rows, row_pos, b->R, b->Hq, g, p.RT, p.items1, p.items2, w.off1, w.off2,
                     w.sc_off, w.rinfo, w.items1, w.items2);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;

  // logits in base-2 units: sigma * log2(e) * q.k
  const float scale2 = scale * kLog2e;
  const bool bf = b->qk_dtype == LAST_BF16;
  e = bf ? (b->Dh == 64 ? launch_rt<uint16_t, 64>(b, p, w, cu_rows, row_pos, q, k, scale2, s)
                        : launch_rt<uint16_t, 128>(b, p, w, cu_rows, row_pos, q, k, scale2, s))
         : (b->Dh == 64 ? launch_rt<float, 64>(b, p, w, cu_rows, row_pos, q, k, scale2, s)
                        : launch_rt<float, 128>(b, p, w, cu_rows, row_pos, q, k, scale2, s));
  if (e != hipSuccess) return e;

  launch_begin("rows_finalize", s);
  hipLaunchKernelGGL(k_rows_finalize, dim3((unsigned)((p.N_total + 255) / 256)), dim3(256), 0, s,
                     w.part, w.mass, b->cu_vis, b->vis_start, w.rinfo, b->R, b->G, b->Hkv, p.RG_max,
                     p.N_total, scores);
  return launch_end(s);
}

}  // namespace last
