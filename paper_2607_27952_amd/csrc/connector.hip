// The cloud's token-wise connector on the transmitted rows (arXiv
// 2607.27952, Sec. 3.4, Eq. 12: H_S = phi_c(X_S)) for gfx950, bf16:
//
//   xhat = LayerNorm(x) = (x - mean) / sqrt(var + eps) * gamma + beta
//   h    = GELU(W1 xhat + b1)        (GELU with erf)
//   y    = W2 h + b2
//
// for every kept row x. The paper gives no formula for phi_c; this is the
// token-wise connector structure of the model family it uses.
//
//   k_layernorm   one block per row, fp32 statistics in a fixed order; xhat
//                 rounded to bf16 (the matrix cores' input type).
//   k_gemm_nt     C[m][n] = sum_k A[n][k] B[m][k] (both operands row-major
//                 with k contiguous: weights one output feature per row,
//                 tokens one row each) plus bias, optionally GELU, rounded to
//                 bf16. Block tile 256 features x 128 tokens, eight waves of
//                 64 x 64 (2 x 2 v_mfma_f32_32x32x16_bf16 tiles); the weights
//                 are the MFMA's A operand, so a lane's accumulator holds one
//                 token and four consecutive features per group, stored as
//                 8-byte pieces. Operands stream through a 3-stage LDS ring by
//                 LDS DMA, 64 columns a stage, one barrier per stage.
#include <algorithm>
#include <math.h>

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
constexpr int kLnThreads = 256;

__device__ float block_sum(float v, float *sh) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[wave] = v;
  __syncthreads();
  float s = 0.f;
  for (int w = 0; w < kLnThreads / 64; ++w) s += sh[w];
  return s;
}

__global__ __launch_bounds__(kLnThreads) void k_layernorm(const uint16_t *__restrict__ x,
                                                          const float *__restrict__ gamma,
                                                          const float *__restrict__ beta, int Dv, float eps,
                                                          uint16_t *__restrict__ xn) {
  __shared__ float sh[kLnThreads / 64];
  const int64_t t = blockIdx.x;
  const uint16_t *row = x + t * Dv;
  float s = 0.f;
  for (int d = threadIdx.x; d < Dv; d += kLnThreads) s += __uint_as_float((uint32_t)row[d] << 16);
  const float mean = block_sum(s, sh) / (float)Dv;
  float c2 = 0.f;
  for (int d = threadIdx.x; d < Dv; d += kLnThreads) {
    const float c = __uint_as_float((uint32_t)row[d] << 16) - mean;
    c2 = fmaf(c, c, c2);
  }
  const float rstd = 1.0f / sqrtf(block_sum(c2, sh) / (float)Dv + eps);
  uint32_t *out = reinterpret_cast<uint32_t *>(xn + t * Dv);
  for (int d = 2 * threadIdx.x; d < Dv; d += 2 * kLnThreads) {
    const float a = (__uint_as_float((uint32_t)row[d] << 16) - mean) * rstd * gamma[d] + beta[d];
    const float b = (__uint_as_float((uint32_t)row[d + 1] << 16) - mean) * rstd * gamma[d + 1] + beta[d + 1];
    out[d / 2] = pack_bf16(a, b);
  }
}

// ---------------------------------------------------------------- GEMM
constexpr int kGN = 256, kGM = 128;          // block tile: features x tokens
constexpr int kGWaves = 8, kGThreads = 64 * kGWaves;
constexpr int kGK = 64;                      // columns per stage
constexpr int kRing = 3;
constexpr int kAPieces = kGN * kGK * 2 / 16;  // 16-byte pieces of a stage: weights (2048)
constexpr int kBPieces = kGM * kGK * 2 / 16;  // tokens (1024)
constexpr int kInstr = (kAPieces + kBPieces) / 64;   // DMA wave instructions per stage (48)
constexpr int kPerWave = kInstr / kGWaves;           // 6
static_assert(kInstr % kGWaves == 0, "even DMA split");

__device__ __forceinline__ int gslot(int row, int piece) { return row * 8 + (piece ^ ((row >> 1) & 7)); }

__device__ __forceinline__ float gelu(float u) { return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f)); }

template <bool GELU>
__global__ __launch_bounds__(kGThreads) void k_gemm_nt(const uint16_t *__restrict__ A,   // [N][Kd]
                                                       const uint16_t *__restrict__ B,   // [M][Kd]
                                                       const float *__restrict__ bias,   // [N]
                                                       int64_t M, int N, int Kd, int n_tiles,
                                                       uint16_t *__restrict__ C) {       // [M][N]
  __shared__ uint4 ring[kRing][kAPieces + kBPieces];
  const int nt = blockIdx.x % n_tiles;
  const int64_t mt = blockIdx.x / n_tiles;
  const int n0 = nt * kGN;
  const int64_t m0 = mt * kGM;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int wn = wave >> 1, wm = wave & 1;   // 4 x 2 waves of 64 x 64

  // This wave's DMA instructions: q = wave + 8 x; the first 32 fill the
  // weight rows of the stage, the other 16 the token rows. The wave-uniform
  // base is the block's first row of the operand (64-bit), a lane's byte
  // offset from it (under 128 rows) is fixed for the block, and the stage
  // moves the base by 64 columns. Rows past the end repeat the last row.
  const char *gbase[kPerWave];
  uint32_t voff[kPerWave], dst[kPerWave];
#pragma unroll
  for (int x = 0; x < kPerWave; ++x) {
    const int q = wave + kGWaves * x;
    const bool isA = q < kAPieces / 64;
    const int sl = (isA ? q : q - kAPieces / 64) * 64 + lane;
    const int row = sl / 8, p = (sl % 8) ^ ((row >> 1) & 7);
    const int64_t first = isA ? n0 : m0, last_row = (isA ? (int64_t)N : M) - 1;
    const int64_t grow = std::min<int64_t>(first + row, last_row);
    gbase[x] = (const char *)uniform_ptr((const char *)(isA ? (const void *)A : (const void *)B) +
                                         first * Kd * 2);
    voff[x] = (uint32_t)((grow - first) * Kd * 2 + p * 16);
    dst[x] = __builtin_amdgcn_readfirstlane(lds_u32(&ring[0][(isA ? 0 : kAPieces) + (sl - lane)]));
  }
  constexpr uint32_t kStageBytes = (kAPieces + kBPieces) * 16;
  auto issue = [&](int st) {
#pragma unroll
    for (int x = 0; x < kPerWave; ++x)
      dma16(dst[x] + (uint32_t)(st % kRing) * kStageBytes, gbase[x] + (int64_t)st * kGK * 2, voff[x]);
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  const int nst = Kd / kGK;
  issue(0);
  if (nst > 1) issue(1);
  if (nst > 1) vm_wait<kPerWave>();
  else vm_wait<0>();
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    if (st + 2 < nst) issue(st + 2);
    const uint4 *sa = ring[st % kRing];
    const uint4 *sb = sa + kAPieces;
#pragma unroll
    for (int ks = 0; ks < kGK / 16; ++ks) {
      const int piece = 2 * ks + (lane >> 5);
      bf16x8_t a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = __builtin_bit_cast(bf16x8_t, sa[gslot(64 * wn + 32 * i + (lane & 31), piece)]);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = __builtin_bit_cast(bf16x8_t, sb[gslot(64 * wm + 32 * j + (lane & 31), piece)]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    // the next stage must have landed before the barrier that publishes it
    if (st + 2 < nst) vm_wait<kPerWave>();
    else vm_wait<0>();
    __syncthreads();
  }

  // Epilogue: lane holds token m0 + 64 wm + 32 j + lane % 32 and features
  // n0 + 64 wn + 32 i + 8 g + 4 (lane / 32) + 0..3 at elements 4 g .. 4 g + 3.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t m = m0 + 64 * wm + 32 * j + (lane & 31);
    if (m >= M) continue;
    uint16_t *crow = C + m * N;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + 64 * wn + 32 * i + 8 * g + 4 * (lane >> 5);
        if (n >= N) continue;
        const float4 bb = *reinterpret_cast<const float4 *>(bias + n);
        float y0 = acc[i][j][4 * g + 0] + bb.x, y1 = acc[i][j][4 * g + 1] + bb.y;
        float y2 = acc[i][j][4 * g + 2] + bb.z, y3 = acc[i][j][4 * g + 3] + bb.w;
        if (GELU) {
          y0 = gelu(y0);
          y1 = gelu(y1);
          y2 = gelu(y2);
          y3 = gelu(y3);
        }
        uint2 w;
        w.x = pack_bf16(y0, y1);
        w.y = pack_bf16(y2, y3);
        *reinterpret_cast<uint2 *>(crow + n) = w;
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
                     (const uint16_t *)B, bias, M, N, Kd, n_tiles, (uint16_t *)C);
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
  hipLaunchKernelGGL(k_layernorm, dim3((unsigned)K), dim3(kLnThreads), 0, s, (const uint16_t *)x, gamma, beta,
                     Dv, eps, (uint16_t *)xn);
  hipError_t e = launch_end(s);
  if (e != hipSuccess) return e;
  e = launch_gemm<true>(w1, xn, b1, K, Dh, Dv, hid, s);
  if (e != hipSuccess) return e;
  return launch_gemm<false>(w2, hid, b2, K, Do, Dh, out, s);
}

}  // namespace last
