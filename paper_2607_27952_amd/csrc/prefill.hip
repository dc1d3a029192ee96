// Causal prefill attention of the guidance model with the LAST statistics
// of each request's last row as a by-product (arXiv 2607.27952, Sec. 3.3:
// the relevance is read from the attention of the same prefill pass), for
// gfx950, bf16 inputs:
//
//   out_p = sum_{j <= p} softmax_j(sigma q_p . k_j) v_j      for every position p
//
// and, for the last position p* = P_r - 1, the scaled logits of the visual
// keys and the row's (max, sum exp, visual sum exp), in the layout the
// last-token score pass uses, so that its merge and finalize kernels turn
// them into w~ (Eq. 7-8) without another pass over the keys.
//
// One block per (layer, request, query head, 128 query positions); each of
// its four waves owns 32 positions. Keys and values go through LDS 64 at a
// time, both row-major with XOR-swizzled 16-byte pieces, copied straight from
// memory by LDS DMA (global_load_lds_dwordx4: no registers, no transposing
// stores) one stage ahead of their use. The value fragments are read with the
// LDS transpose load (ds_read_b64_tr_b16): in each group of 16 lanes, lane i's
// element j comes from element i % 4 of the 8 bytes lane 4 j + i / 4 points
// at, so lanes pointing at 4 keys x 4 four-dimension chunks receive 4 keys of
// one dimension each.
//
// The product runs transposed so that every lane owns one query:
//   S^T = K Q^T   (v_mfma_f32_32x32x16_bf16, A = 32 keys, B = the wave's 32
//                  queries, kept in registers): lane l holds query l % 32 and
//                  16 of the 32 keys of a tile, the other 16 being in lane
//                  l ^ 32. The tile's keys are loaded into the MFMA rows in a
//                  permuted order, so that lane half h holds keys
//                  8h .. 8h + 7 and 16 + 8h .. 16 + 8h + 7 of the tile.
//   O^T = V^T P^T (A = 32 value dimensions x 16 keys from the transposed
//                  LDS stage, B = 8 probabilities of the lane, packed to bf16):
//                  the permutation above makes each lane's probabilities
//                  exactly the keys its half of the B operand needs.
// The softmax runs online per lane in base-2 units (the scale times log2 e
// folded into the exponent's fma): the stage's row max and sum take one
// exchange with the partner lane, and the lane's O^T column is rescaled in
// place when some lane's max has moved.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kQB = 32 * kWaves;              // query positions per block
constexpr int kKS = 64;                       // keys per LDS stage
constexpr float kLog2e = 1.4426950408889634f;

template <int DH>
struct Shape {
  static constexpr int kPieces = DH * 2 / 16;            // 16-byte pieces per key row
  static constexpr int kSteps = kPieces / 2;             // S^T MFMA steps per key tile
  static constexpr int kDT = DH / 32;                    // value-dimension tiles of O^T
  static constexpr int kDma = kKS * kPieces / 64;        // DMA instructions per operand stage
  static constexpr int kDmaPerWave = kDma / kWaves;      // ... per wave
  static_assert(kDmaPerWave >= 1 && kDma % kWaves == 0, "stage split");
};

template <int NP>
__device__ __forceinline__ int kslot(int j, int p) {
  return j * NP + (p ^ (NP >= 16 ? (j & 15) : ((j >> 1) & 7)));
}

// Physical 16-byte piece of logical piece p in row j of a stage (keys and
// values alike).
template <int NP>
__device__ __forceinline__ int pswz(int j, int p) {
  return p ^ (NP >= 16 ? (j & 15) : ((j >> 1) & 7));
}

typedef short s16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ s16x4_t read_tr(const uint16_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t *)p);
}

// Key of a 32-key tile that MFMA row i carries: lane half h, element v of the
// accumulator (row 4h + v % 4 + 8 (v / 4)) then holds key 8h + v (v < 8) or
// 16 + 8h + v - 8 (v >= 8).
__device__ __forceinline__ int perm_key(int i) {
  const int h = (i >> 2) & 1, v = (i & 3) + 4 * (i >> 3);
  return 8 * h + v + (v >= 8 ? 8 : 0);
}
__device__ __forceinline__ int acc_key(int half, int v) { return 8 * half + v + (v >= 8 ? 8 : 0); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// two floats to bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const f32x2_t x = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2_t));
}

// One (layer, request, head, 128-position block) per block.
template <int DH>
__global__ __launch_bounds__(kThreads, 2) void k_prefill(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k, const uint16_t *__restrict__ v,
    const int32_t *__restrict__ cu_seqlens, const int32_t *__restrict__ vis_start,
    const int32_t *__restrict__ cu_vis, const int32_t *__restrict__ qb_off,
    const int32_t *__restrict__ qb_req, int R, int Hq, int Hkv, int64_t QB_total,
    int64_t T_total, int64_t N_total, float scale, uint16_t *__restrict__ out,
    float *__restrict__ vlog, float4 *__restrict__ stats) {
  using SH = Shape<DH>;
  __shared__ uint4 s_k[2][kKS * SH::kPieces];
  __shared__ uint4 s_v[2][kKS * SH::kPieces];

  // The query blocks of one (layer, head, request) are neighbours in this
  // order; XCD-contiguous numbering runs them together on one XCD, so they
  // re-read the request's keys and values from its L2 rather than from HBM.
  int64_t bid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int64_t qbi = bid % QB_total;
  bid /= QB_total;
  const int h = (int)(bid % Hq);
  const int l = (int)(bid / Hq);
  const int r = qb_req[qbi];
  const int qb = (int)(qbi - qb_off[r]);
  const int g = Hq / Hkv, kv = h / g;
  const int64_t tok0 = cu_seqlens[r];
  const int P = cu_seqlens[r + 1] - (int)tok0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 31, half = lane >> 5;
  const int q0 = qb * kQB + wave * 32;           // the wave's first query position
  const int qpos = q0 + col;                     // this lane's query
  const bool qreal = qpos < P;
  const int kend = min(P, qb * kQB + kQB);       // keys the block needs: 0 .. kend - 1
  const int wave_last = min(P, q0 + 32) - 1;     // the wave's last real query (-1: none)
  const float s2 = scale * kLog2e;
  const int vlo = vis_start[r], vhi = vlo + (cu_vis[r + 1] - cu_vis[r]);
  const bool has_last = q0 <= P - 1 && P - 1 < q0 + 32;   // the wave holds the request's last row

  // B operand of S^T: the lane's query row, pieces 2st + half
  uint4 bq[SH::kSteps];
  {
    const char *qp = reinterpret_cast<const char *>(q + (((int64_t)l * T_total + tok0 + min(qpos, P - 1)) * Hq + h) * DH);
#pragma unroll
    for (int st = 0; st < SH::kSteps; ++st) bq[st] = *reinterpret_cast<const uint4 *>(qp + (2 * st + half) * 16);
  }

  const int64_t kvstride = (int64_t)Hkv * DH;    // elements between consecutive tokens
  const uint16_t *kbase = k + ((int64_t)l * T_total + tok0) * kvstride + (int64_t)kv * DH;
  const uint16_t *vbase = v + ((int64_t)l * T_total + tok0) * kvstride + (int64_t)kv * DH;

  // One stage: keys j0 .. j0 + 63 (clamped to the block's last needed key) of
  // both operands. DMA instruction x of this wave covers 16-byte slots
  // 64 q + lane, q = wave + kWaves x, of the stage: row (slot / kPieces),
  // physical piece (slot % kPieces), which holds logical piece
  // pswz(row, physical) (an XOR, its own inverse).
  auto issue_stage = [&](int j0, int buf) {
#pragma unroll
    for (int x = 0; x < SH::kDmaPerWave; ++x) {
      const int q = wave + kWaves * x, slot = q * 64 + lane;
      const int j = slot / SH::kPieces, pp = slot % SH::kPieces;
      const int jj = min(j0 + j, kend - 1);
      const uint32_t voff = (uint32_t)(((int64_t)jj * kvstride + pswz<SH::kPieces>(j, pp) * 8) * 2);
      dma16(__builtin_amdgcn_readfirstlane(lds_u32(&s_k[buf][q * 64])), uniform_ptr(kbase), voff);
      dma16(__builtin_amdgcn_readfirstlane(lds_u32(&s_v[buf][q * 64])), uniform_ptr(vbase), voff);
    }
  };

  float m = -INFINITY, lsum = 0.f, vsum = 0.f;   // per lane (= per query), base-2 units
  f32x16_t o[SH::kDT];
#pragma unroll
  for (int dt = 0; dt < SH::kDT; ++dt) o[dt] = f32x16_t{};

  const int nst = (kend + kKS - 1) / kKS;
  issue_stage(0, 0);
  vm_wait<0>();
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    // the other buffer was last read in stage st - 1, which every wave has left
    if (st + 1 < nst) issue_stage((st + 1) * kKS, (st + 1) & 1);
    const int k0 = st * kKS;
    if (k0 <= wave_last) {
      const uint4 *kb = s_k[st & 1];
      const uint16_t *vs = reinterpret_cast<const uint16_t *>(s_v[st & 1]);
      // The fragment addresses derive from the lane index anew in every stage
      // (opaque to the compiler), instead of two dozen of them being hoisted
      // out of the loop and held in registers.
      int ln = (int)threadIdx.x & 63;
      asm volatile("" : "+v"(ln));
      const int lcol = ln & 31, lhalf = ln >> 5;
      // S^T for the stage's two 32-key tiles
      f32x16_t sc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sc[t] = f32x16_t{};
        const int krow = t * 32 + perm_key(lcol);
#pragma unroll
        for (int s = 0; s < SH::kSteps; ++s)
          sc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, kb[kslot<SH::kPieces>(krow, 2 * s + lhalf)]),
              __builtin_bit_cast(bf16x8_t, bq[s]), sc[t], 0, 0, 0);
      }
      // base-2 logits: the raw dots stay in place and the scale goes into the
      // exponent (s2 > 0, so the largest dot gives the largest logit); keys a
      // query does not see (causal mask, past the block's end) are -inf
      const bool full = k0 + kKS - 1 <= q0;   // every query of the wave sees every key
      if (!full) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = k0 + t * 32 + acc_key(half, e);
            sc[t][e] = (key <= qpos && key < kend) ? sc[t][e] : -INFINITY;
          }
      }
      float mx = sc[0][0];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[t][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * s2;
      const float mnew = fmaxf(m, mx);
      // a query with no key seen yet keeps -inf; its terms are 0 and its
      // factor 1 (its sums are still 0)
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(m - mref);
      float ps = 0.f, pv = 0.f;
      uint32_t pb[2][8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[t][e], s2, -mref));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[t][e + 1], s2, -mref));
          ps += p0 + p1;
          if (has_last) {
            const int key = k0 + t * 32 + acc_key(half, e);
            pv += (key >= vlo && key < vhi ? p0 : 0.f) + (key + 1 >= vlo && key + 1 < vhi ? p1 : 0.f);
          }
          pb[t][e / 2] = pack_bf16(p0, p1);
        }
      ps += __shfl_xor(ps, 32);
      lsum = lsum * alpha + ps;
      if (has_last) {
        pv += __shfl_xor(pv, 32);
        vsum = vsum * alpha + pv;
      }
      // the running max moves rarely after the first stages: rescale only then
      if (__any(mnew != m)) {
#pragma unroll
        for (int dt = 0; dt < SH::kDT; ++dt) o[dt] *= alpha;
      }
      m = mnew;
      // O^T += V^T P^T: four 16-key steps, each lane's B operand being 8 of
      // its own probabilities (keys 16s + 8 half .. + 7 of the stage)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const uint32_t *pw = &pb[s >> 1][(s & 1) * 4];
        const uint4 bp = make_uint4(pw[0], pw[1], pw[2], pw[3]);
#pragma unroll
        for (int dt = 0; dt < SH::kDT; ++dt) {
          // A = V^T: lane l needs dimension dt 32 + l % 32 of keys 16 s + 8 half
          // .. + 7, as two transpose reads of 4 keys; lane p of its 16-lane
          // group points at key (p / 4) of the four and dimensions
          // 4 (p % 4) .. + 3 of the group's 16
          const int g = ln >> 4, pl = ln & 15;
          const int d = dt * 32 + 16 * (g & 1) + 4 * (pl & 3);   // first dimension of the chunk
          s16x4_t tv[2];
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int key = 16 * s + 8 * (g >> 1) + 4 * c + (pl >> 2);
            tv[c] = read_tr(vs + key * DH + pswz<SH::kPieces>(key, d >> 3) * 8 + (d & 7));
          }
          const s16x4_t a0 = tv[0], a1 = tv[1];
          typedef short s16x8_t __attribute__((ext_vector_type(8)));
          const s16x8_t av = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                          __builtin_bit_cast(bf16x8_t, bp), o[dt], 0, 0, 0);
        }
      }
      // the request's last row: its visual logits, in the score pass's base-2
      // units
      if (has_last && qpos == P - 1) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = k0 + t * 32 + acc_key(half, e);
            if (key >= vlo && key < vhi && key < kend)
              vlog[((int64_t)l * N_total + cu_vis[r] + key - vlo) * Hq + h] = sc[t][e] * s2;
          }
      }
    }
    // the next stage has landed (this wave's copies), and every wave's after
    // the barrier
    vm_wait<0>();
    __syncthreads();
  }

  // out_p = O^T column / sum; lane half h holds dimensions 4h + e % 4 + 8 (e / 4)
  if (qreal) {
    const float inv = 1.0f / lsum;
    uint16_t *op = out + (((int64_t)l * T_total + tok0 + qpos) * Hq + h) * DH;
#pragma unroll
    for (int dt = 0; dt < SH::kDT; ++dt)
#pragma unroll
      for (int e = 0; e < 16; e += 4) {
        const int d = dt * 32 + 4 * half + 8 * (e / 4);
        uint2 w;
        w.x = pack_bf16(o[dt][e] * inv, o[dt][e + 1] * inv);
        w.y = pack_bf16(o[dt][e + 2] * inv, o[dt][e + 3] * inv);
        *reinterpret_cast<uint2 *>(op + d) = w;
      }
  }
  // the last row's statistics as one chunk of the score pass: (max, sum, visual sum)
  if (has_last && qpos == P - 1 && half == 0)
    stats[((int64_t)l * Hq + h) * R + r] = make_float4(m, lsum, vsum, 0.f);
}

// Per request: the number of 128-position query blocks, their prefix and the
// block -> request map.
__global__ __launch_bounds__(256) void k_prefill_plan(const int32_t *__restrict__ cu_seqlens, int R,
                                                      int64_t cap, int32_t *__restrict__ qb_off,
                                                      int32_t *__restrict__ qb_req) {
  __shared__ int sh[4];
  int carry = 0;
  for (int base = 0; base < R; base += 256) {
    const int r = base + (int)threadIdx.x;
    int n = 0;
    if (r < R) n = (cu_seqlens[r + 1] - cu_seqlens[r] + kQB - 1) / kQB;
    int tot;
    const int pre = block_exclusive_scan(n, sh, &tot) + carry;
    if (r < R) {
      qb_off[r] = pre;
      for (int i = 0; i < n; ++i)
        if (pre + i < cap) qb_req[pre + i] = r;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) qb_off[R] = carry;
}

}  // namespace

namespace last {

int64_t prefill_query_blocks(const last_batch *b) {
  int64_t n = 0;
  for (int r = 0; r < b->R; ++r) n += (b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r] + kQB - 1) / kQB;
  return n;
}

hipError_t launch_prefill(const last_batch *b, int64_t QB_total, int32_t *qb_off, int32_t *qb_req,
                          const void *q, const void *k, const void *v, void *out, float *vlog,
                          float4 *stats, float scale, hipStream_t s) {
  launch_begin("prefill_plan", s);
  hipLaunchKernelGGL(k_prefill_plan, dim3(1), dim3(256), 0, s, b->cu_seqlens, b->R, QB_total, qb_off, qb_req);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;
  const int64_t blocks = (int64_t)b->G * b->Hq * QB_total;
  const int64_t T_total = b->cu_seqlens_h[b->R], N_total = b->cu_vis_h[b->R];
  launch_begin("prefill", s);
  if (b->Dh == 64)
    hipLaunchKernelGGL(k_prefill<64>, dim3((unsigned)blocks), dim3(kThreads), 0, s, (const uint16_t *)q,
                       (const uint16_t *)k, (const uint16_t *)v, b->cu_seqlens, b->vis_start, b->cu_vis,
                       qb_off, qb_req, b->R, b->Hq, b->Hkv, QB_total, T_total, N_total, scale,
                       (uint16_t *)out, vlog, stats);
  else
    hipLaunchKernelGGL(k_prefill<128>, dim3((unsigned)blocks), dim3(kThreads), 0, s, (const uint16_t *)q,
                       (const uint16_t *)k, (const uint16_t *)v, b->cu_seqlens, b->vis_start, b->cu_vis,
                       qb_off, qb_req, b->R, b->Hq, b->Hkv, QB_total, T_total, N_total, scale,
                       (uint16_t *)out, vlog, stats);
  return launch_end(s);
}

}  // namespace last
