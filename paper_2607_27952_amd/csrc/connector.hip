// The cloud's token-wise connector on the transmitted rows (arXiv
// 2607.27952: Sec. 3.4 applies phi_c to the rows of Eq. 12, H_S = phi_c(X_S);
// Sec. 3.2 defines phi_c as a token-wise connector) for gfx950, bf16:
//
//   xhat = LayerNorm(x) = (x - mean) / sqrt(var + eps) * gamma + beta
//   h    = GELU(W1 xhat + b1)        (GELU with erf)
//   y    = W2 h + b2
//
// for every kept row x. The paper gives no formula for phi_c; this is the
// token-wise connector structure of the model family it uses.
//
//   k_layernorm   one wave per row, fp32 statistics in a fixed order; xhat
//                 rounded to bf16 (the matrix cores' input type).
//   k_gemm_nt     C[m][n] = sum_k A[n][k] B[m][k] (both operands row-major
//                 with k contiguous: weights one output feature per row,
//                 tokens one row each) plus bias, optionally GELU, rounded to
//                 bf16. Block tile 256 features x 256 tokens, four waves of
//                 128 x 128 (4 x 4 v_mfma_f32_32x32x16_bf16 tiles); the
//                 weights are the MFMA's A operand. Operands stream through a
//                 2-stage LDS ring by LDS DMA, 64 columns a stage, one barrier
//                 per stage; the output tile leaves through the same LDS, so
//                 that its stores cover whole rows.
#include <algorithm>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const f32x2_t x = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2_t));
}

// ---------------------------------------------------------------- LayerNorm
// One wave per row, 16-byte pieces (8 values): lane l takes pieces l, l + 64,
// ... Rows of up to 64 NP pieces are loaded once into registers (all loads
// in flight together); longer rows stream, reading the row again from cache
// for the deviations and the output. Sums are fp32, each lane's in piece
// order, then across the wave in a fixed order.
constexpr int kLnWaves = 4;

__device__ __forceinline__ void unpack8(const uint4 &w, float *v) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_lo(u[i]);
    v[2 * i + 1] = bf16_hi(u[i]);
  }
}

__device__ __forceinline__ uint4 norm8(const uint4 &w, float mean, float rstd, const float *__restrict__ gamma,
                                       const float *__restrict__ beta, int p) {
  float v[8];
  unpack8(w, v);
  const float4 *g4 = reinterpret_cast<const float4 *>(gamma);
  const float4 *b4 = reinterpret_cast<const float4 *>(beta);
  const float4 ga = g4[2 * p], gb = g4[2 * p + 1], ba = b4[2 * p], bb = b4[2 * p + 1];
  const float g[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
  const float b[8] = {ba.x, ba.y, ba.z, ba.w, bb.x, bb.y, bb.z, bb.w};
  float y[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = (v[i] - mean) * rstd * g[i] + b[i];
  return make_uint4(pack_bf16(y[0], y[1]), pack_bf16(y[2], y[3]), pack_bf16(y[4], y[5]), pack_bf16(y[6], y[7]));
}

// NP > 0: at most NP pieces per lane, held in registers; NP == 0: streaming.
template <int NP>
__global__ __launch_bounds__(64 * kLnWaves) void k_layernorm(const uint16_t *__restrict__ x,
                                                             const float *__restrict__ gamma,
                                                             const float *__restrict__ beta, int64_t K,
                                                             int Dv, float eps, uint16_t *__restrict__ xn) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * kLnWaves + (threadIdx.x >> 6);
  if (t >= K) return;
  const uint4 *row = reinterpret_cast<const uint4 *>(x + t * Dv);
  uint4 *out = reinterpret_cast<uint4 *>(xn + t * Dv);
  const int np = Dv / 8;
  float v[8];
  if constexpr (NP > 0) {
    uint4 w[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) w[i] = lane + 64 * i < np ? row[lane + 64 * i] : make_uint4(0, 0, 0, 0);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      unpack8(w[i], v);
#pragma unroll
      for (int j = 0; j < 8; ++j) s += v[j];
    }
    const float mean = wave_sum(s) / (float)Dv;
    float c2 = 0.f;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if (lane + 64 * i >= np) break;
      unpack8(w[i], v);
#pragma unroll
      for (int j = 0; j < 8; ++j) c2 = fmaf(v[j] - mean, v[j] - mean, c2);
    }
    const float rstd = 1.0f / sqrtf(wave_sum(c2) / (float)Dv + eps);
#pragma unroll
    for (int i = 0; i < NP; ++i)
      if (lane + 64 * i < np) out[lane + 64 * i] = norm8(w[i], mean, rstd, gamma, beta, lane + 64 * i);
  } else {
    float s = 0.f;
    for (int p = lane; p < np; p += 64) {
      unpack8(row[p], v);
#pragma unroll
      for (int j = 0; j < 8; ++j) s += v[j];
    }
    const float mean = wave_sum(s) / (float)Dv;
    float c2 = 0.f;
    for (int p = lane; p < np; p += 64) {
      unpack8(row[p], v);
#pragma unroll
      for (int j = 0; j < 8; ++j) c2 = fmaf(v[j] - mean, v[j] - mean, c2);
    }
    const float rstd = 1.0f / sqrtf(wave_sum(c2) / (float)Dv + eps);
    for (int p = lane; p < np; p += 64) out[p] = norm8(row[p], mean, rstd, gamma, beta, p);
  }
}

// ---------------------------------------------------------------- GEMM
// Block tile kGN features x kGM tokens, four waves of 128 x 128 (4 x 4
// v_mfma_f32_32x32x16_bf16 tiles). A stage holds kGK columns of both
// operands; kRing stages live in LDS, filled by LDS DMA one stage ahead of
// use (kRing - 1 stages in flight). Each 16-column step's fragments are read
// from LDS while the previous step's 16 products run, and the stage's last
// step is multiplied after the barrier that publishes the next stage, so the
// matrix cores keep busy across it.
constexpr int kGN = 256, kGM = 256;          // block tile: features x tokens
constexpr int kGWaves = 4, kGThreads = 64 * kGWaves;
constexpr int kGK = 64;                      // columns per stage
constexpr int kRing = 2;
constexpr int kRowPieces = kGK * 2 / 16;     // 16-byte pieces of one row of a stage
constexpr int kAPieces = kGN * kRowPieces;   // weights
constexpr int kBPieces = kGM * kRowPieces;   // tokens
constexpr int kStagePieces = kAPieces + kBPieces;
constexpr int kInstr = kStagePieces / 64;    // DMA wave instructions per stage
constexpr int kPerWave = kInstr / kGWaves;
constexpr int kSteps = kGK / 16;             // MFMA k-steps per stage
static_assert(kInstr % kGWaves == 0 && (kAPieces / 64) % kGWaves == 0, "even DMA split");
static_assert(kRowPieces == 8 || kRowPieces == 4, "swizzle assumes 4 or 8 pieces a row");
static_assert(kGN == 256 && kGM * kGN * 2 <= kRing * kStagePieces * 16, "the output tile is staged in the ring");

// A row's pieces are permuted so that 16 consecutive rows read at one piece
// index hit 16 distinct 16-byte bank groups.
__device__ __forceinline__ int gslot(int row, int piece) {
  return row * kRowPieces + (piece ^ ((row / (16 / kRowPieces)) % kRowPieces));
}

// GELU(u) = u (1 + erf(u / sqrt 2)) / 2 with erf from Abramowitz and Stegun,
// Handbook of Mathematical Functions, formula 7.1.26: for x >= 0,
// erfc(x) = (a1 t + ... + a5 t^5) e^(-x^2), t = 1 / (1 + p x), within
// 1.5e-7. With q = erfc(|u| / sqrt 2), GELU is u (1 - q / 2) for u >= 0 and
// u q / 2 below; in fp32 the result stays within 1e-6 (1 + |u|), far under
// the bf16 rounding that follows. One reciprocal and one exponential, where
// a full-precision erf costs several times more in this one-wave-per-SIMD
// epilogue.
__device__ __forceinline__ float gelu(float u) {
  const float x = fabsf(u) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  float poly = fmaf(1.061405429f, t, -1.453152027f);
  poly = fmaf(poly, t, 1.421413741f);
  poly = fmaf(poly, t, -0.284496736f);
  poly = fmaf(poly, t, 0.254829592f);
  poly *= t;
  const float q = poly * __builtin_amdgcn_exp2f(-(x * x) * 1.4426950408889634f);
  return u >= 0.0f ? u * fmaf(-0.5f, q, 1.0f) : 0.5f * u * q;
}

struct Frags {
  bf16x8_t a[4], b[4];
};

template <bool GELU>
__global__ __launch_bounds__(kGThreads, 1) void k_gemm_nt(const uint16_t *__restrict__ A,   // [N][Kd]
                                                          const uint16_t *__restrict__ B,   // [M][Kd]
                                                          const float *__restrict__ bias,   // [N]
                                                          int64_t M, int N, int Kd, int n_tiles,
                                                          int blocks_xcd,
                                                          uint16_t *__restrict__ C) {       // [M][N]
  __shared__ uint4 ring[kRing][kStagePieces];
  // Blocks are dealt to the 8 XCDs in turn; renumber them so that each XCD
  // runs a contiguous range of tiles, taken 8 token tiles at a time across
  // the feature tiles, which keeps the operands it shares in its own L2.
  const int64_t b = blockIdx.x;
  const int64_t l = b < (int64_t)blocks_xcd * 8 ? (b % 8) * blocks_xcd + b / 8 : b;
  const int64_t band = l / (8 * (int64_t)n_tiles), in_band = l % (8 * (int64_t)n_tiles);
  const int64_t m_tiles = (M + kGM - 1) / kGM;
  const int64_t band_rows = std::min<int64_t>(8, m_tiles - band * 8);
  const int64_t mt = band * 8 + in_band % band_rows;
  const int nt = (int)(in_band / band_rows);
  const int n0 = nt * kGN;
  const int64_t m0 = mt * kGM;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int wn = wave >> 1, wm = wave & 1;   // 2 x 2 waves of 128 x 128

  // This wave's DMA instructions q = wave + 4 x: the first kAPieces / 64 fill
  // the weight rows of a stage, the rest the token rows. The base is the
  // block's first row of the operand (64-bit, wave-uniform), a lane's byte
  // offset from it (under 256 rows) is fixed for the block, and each stage
  // moves the base by kGK columns. Rows past the end repeat the last row.
  const char *baseA = (const char *)uniform_ptr((const char *)A + (int64_t)n0 * Kd * 2);
  const char *baseB = (const char *)uniform_ptr((const char *)B + m0 * Kd * 2);
  uint32_t voff[kPerWave], dst[kPerWave];
#pragma unroll
  for (int x = 0; x < kPerWave; ++x) {
    const int q = wave + kGWaves * x;
    const bool isA = x < kAPieces / 64 / kGWaves;   // q < kAPieces / 64
    const int sl = (isA ? q : q - kAPieces / 64) * 64 + lane;
    const int row = sl / kRowPieces, slot = sl % kRowPieces;
    const int p = slot ^ ((row / (16 / kRowPieces)) % kRowPieces);
    const int64_t first = isA ? n0 : m0, last_row = (isA ? (int64_t)N : M) - 1;
    const int64_t grow = std::min<int64_t>(first + row, last_row);
    voff[x] = (uint32_t)((grow - first) * Kd * 2 + p * 16);
    dst[x] = __builtin_amdgcn_readfirstlane(lds_u32(&ring[0][(isA ? 0 : kAPieces) + (sl - lane)]));
  }
  constexpr uint32_t kStageBytes = kStagePieces * 16;
  // Instructions x in [x0, x1) of stage st's DMA.
  auto issue = [&](int st, int x0, int x1) {
    const int64_t col = (int64_t)st * kGK * 2;
    const uint32_t so = (uint32_t)(st % kRing) * kStageBytes;
#pragma unroll
    for (int x = 0; x < kPerWave; ++x)
      if (x >= x0 && x < x1) dma16(dst[x] + so, (x < kAPieces / 64 / kGWaves ? baseA : baseB) + col, voff[x]);
  };

  // Fragment addresses: lane row lane % 32 of every 32-row tile; the piece
  // for k-step ks is 2 ks + lane / 32.
  const int r32 = lane & 31, half = lane >> 5;
  auto load = [&](Frags &f, int st, int ks) {
    const uint4 *sa = ring[st % kRing];
    const uint4 *sb = sa + kAPieces;
    const int piece = 2 * ks + half;
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = __builtin_bit_cast(bf16x8_t, sa[gslot(128 * wn + 32 * i + r32, piece)]);
#pragma unroll
    for (int j = 0; j < 4; ++j) f.b[j] = __builtin_bit_cast(bf16x8_t, sb[gslot(128 * wm + 32 * j + r32, piece)]);
  };

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};
  auto mma = [&](const Frags &f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  };

  // The look-ahead stage's DMA goes out a k-step at a time, kChunk
  // instructions after each step's fragment reads: one burst at the top of
  // the stage backs up the memory queue and stalls the products (measured:
  // a 4096-cube product takes 141 us with one burst, 130 us over two steps,
  // 125 us over four).
  constexpr int kChunk = kPerWave / kSteps;
  static_assert(kPerWave % kSteps == 0, "DMA chunks per k-step");
  const int nst = Kd / kGK;
#pragma unroll
  for (int st = 0; st < kRing - 1; ++st)
    if (st < nst) issue(st, 0, kPerWave);
  Frags cur, nxt;
  for (int st = 0; st < nst; ++st) {
    // stage st has landed for this wave once at most the later stages' loads
    // are outstanding; the barrier publishes it and retires every read of
    // the slot the look-ahead DMA overwrites
    if (st + kRing - 2 < nst && kRing > 2) vm_wait<(kRing - 2) * kPerWave>();
    else vm_wait<0>();
    __syncthreads();
    const bool ahead = st + kRing - 1 < nst;
    load(nxt, st, 0);
    if (ahead) issue(st + kRing - 1, 0, kChunk);
    if (st > 0) mma(cur);
#pragma unroll
    for (int ks = 1; ks < kSteps; ++ks) {
      cur = nxt;
      load(nxt, st, ks);
      if (ahead) issue(st + kRing - 1, ks * kChunk, (ks + 1) * kChunk);
      mma(cur);
    }
    cur = nxt;
  }
  mma(cur);

  // Epilogue, in two passes through the ring (free once every wave is past
  // its last fragment read). A lane's accumulators hold one token and
  // scattered groups of four features (token m0 + 128 wm + 32 j + lane % 32,
  // features n0 + 128 wn + 32 i + 8 g + 4 (lane / 32) + 0..3 at elements
  // 4 g .. 4 g + 3); stored as they are, every 8-byte piece would land in a
  // different cache line. So the block's 256 x 256 tile goes to LDS as bf16
  // (rows of 32 16-byte pieces, piece index XOR token % 32 so that the 32
  // tokens of a write spread over the banks), then leaves row by row, 32
  // lanes covering a row's 512 bytes.
  __syncthreads();
  uint2 *ot2 = reinterpret_cast<uint2 *>(&ring[0][0]);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int t = 128 * wm + 32 * j + r32;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = 128 * wn + 32 * i + 8 * g;
        const int n = n0 + nl + 4 * half;
        const float4 bb = n < N ? *reinterpret_cast<const float4 *>(bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
        float y0 = acc[i][j][4 * g + 0] + bb.x, y1 = acc[i][j][4 * g + 1] + bb.y;
        float y2 = acc[i][j][4 * g + 2] + bb.z, y3 = acc[i][j][4 * g + 3] + bb.w;
        if (GELU) {
          y0 = gelu(y0);
          y1 = gelu(y1);
          y2 = gelu(y2);
          y3 = gelu(y3);
        }
        ot2[(t * 32 + ((nl >> 3) ^ (t & 31))) * 2 + half] = make_uint2(pack_bf16(y0, y1), pack_bf16(y2, y3));
      }
  }
  __syncthreads();
  const uint4 *ot = &ring[0][0];
  const int piece = threadIdx.x & 31;
  const int n = n0 + 8 * piece;
  // N is a multiple of 4: a piece is whole, half (8-byte aligned rows when
  // N % 8 == 4) or past the end.
  const bool whole = N % 8 == 0;
#pragma unroll 4
  for (int k = 0; k < kGM / (kGThreads / 32); ++k) {
    const int t = k * (kGThreads / 32) + ((int)threadIdx.x >> 5);
    const int64_t m = m0 + t;
    if (m >= M || n >= N) continue;
    const uint4 v = ot[t * 32 + (piece ^ (t & 31))];
    uint16_t *dst = C + m * N + n;
    if (whole) {
      *reinterpret_cast<uint4 *>(dst) = v;
    } else {
      *reinterpret_cast<uint2 *>(dst) = make_uint2(v.x, v.y);
      if (n + 4 < N) *reinterpret_cast<uint2 *>(dst + 4) = make_uint2(v.z, v.w);
    }
  }
}

template <bool GELU>
hipError_t launch_gemm(const void *A, const void *B, const float *bias, int64_t M, int N, int Kd, void *C,
                       hipStream_t s) {
  const int n_tiles = (N + kGN - 1) / kGN;
  const int64_t blocks = (int64_t)n_tiles * ((M + kGM - 1) / kGM);
  last::launch_begin(GELU ? "connector_gemm1" : "connector_gemm2", s);
  hipLaunchKernelGGL(k_gemm_nt<GELU>, dim3((unsigned)blocks), dim3(kGThreads), 0, s, (const uint16_t *)A,
                     (const uint16_t *)B, bias, M, N, Kd, n_tiles, (int)(blocks / 8), (uint16_t *)C);
  return last::launch_end(s);
}

}  // namespace

namespace last {

bool connector_shape_ok(int64_t K, int32_t Dv, int32_t Dh, int32_t Do) {
  const int64_t blocks = (K + kGM - 1) / kGM * ((std::max(Dh, Do) + kGN - 1) / kGN);
  return Dv % kGK == 0 && Dh % kGK == 0 && Do % 4 == 0 && blocks <= INT32_MAX;
}

hipError_t launch_connector(int64_t K, int32_t Dv, int32_t Dh, int32_t Do, float eps, const void *x,
                            const float *gamma, const float *beta, const void *w1, const float *b1,
                            const void *w2, const float *b2, void *out, void *xn, void *hid,
                            hipStream_t s) {
  if (K == 0) return hipSuccess;
  launch_begin("connector_layernorm", s);
  const dim3 grid((unsigned)((K + kLnWaves - 1) / kLnWaves)), block(64 * kLnWaves);
  const int per_lane = (Dv / 8 + 63) / 64;
  if (per_lane <= 4)
    hipLaunchKernelGGL(k_layernorm<4>, grid, block, 0, s, (const uint16_t *)x, gamma, beta, K, Dv, eps,
                       (uint16_t *)xn);
  else if (per_lane <= 8)
    hipLaunchKernelGGL(k_layernorm<8>, grid, block, 0, s, (const uint16_t *)x, gamma, beta, K, Dv, eps,
                       (uint16_t *)xn);
  else
    hipLaunchKernelGGL(k_layernorm<0>, grid, block, 0, s, (const uint16_t *)x, gamma, beta, K, Dv, eps,
                       (uint16_t *)xn);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;
  e = launch_gemm<true>(w1, xn, b1, K, Dh, Dv, hid, s);
  if (e != hipSuccess) return e;
  return launch_gemm<false>(w2, hid, b2, K, Do, Dh, out, s);
}

}  // namespace last
