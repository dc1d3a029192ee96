// Selection of LAST (arXiv 2607.27952, Sec. 3.4, Eq. 9-12; Sec. 4.3 Table 5)
// for gfx950.
//
// k-center mode. The greedy of Eq. 9-11 needs, at each of its K sequential
// steps, the coverage distance of every token to the newest pick. Instead of
// re-reading the request's features every step (a GEMV per step, K full
// passes over X), the distances are formed once as a matrix on the matrix
// cores and each step reads one row of it:
//
//   k_select_plan   per-request Gram tile prefix, tile -> request map and the
//                   element offset of each request's N_r x N_r block.
//   k_sqnorm_bf16   |x_i|^2 with the very arithmetic the Gram uses for its
//                   diagonal (32x32x16 bf16 MFMA, fp32 partial sums over
//                   64-element chunks folded into fp64), so that a row and
//                   its bitwise duplicate get coverage distance exactly 0.
//   k_gram_bf16     upper-triangular 128x128 tiles of X_r X_r^T on MFMA
//                   (v_mfma_f32_32x32x16_bf16; bf16 products are exact, the
//                   fp32 accumulator is folded into fp64 every 64 elements),
//                   then delta_ij = max(0, 1 - dot_ij / (|x_i| |x_j|)) in fp64,
//                   stored as fp32 in both (i, j) and (j, i).
//   k_sqnorm_f32 / k_gram_f32   the same for fp32 features, in fp64 VALU FMAs.
//   k_greedy        one block per request; w and delta live in registers.
//                   Step t loads row j_{t-1} of the distance block, folds it
//                   into delta with min, and takes the block-wide argmax of
//                   w * delta over unselected tokens (ties -> lowest index,
//                   via a 64-bit key of (value bits, ~index)). The kept set is
//                   compacted in ascending order at the end (Eq. 12).
//
// Top-k mode (Table 5): k_topk, one block per request, radix-selects the K
// largest scores on their fp32 bit patterns (non-negative floats order like
// their bits), breaks ties at the threshold towards the lowest index, and
// ranks the kept tokens for the pick order.
#include <algorithm>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kTile = last::kGramTile;   // 128
constexpr int kKS = 64;                  // elements per k stage = one fp64 fold chunk
constexpr int kLdsPitch = kKS + 8;       // bf16 per LDS row (pad against bank conflicts)
constexpr int kGramThreads = 256;

// ------------------------------------------------------------------ plan
__device__ int block_excl_scan_i64(int64_t v, int64_t *sh, int64_t *total, int64_t *out) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int64_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int64_t before = 0, tot = 0;
  for (int w = 0; w < nw; ++w) {
    if (w < wave) before += sh[w];
    tot += sh[w];
  }
  __syncthreads();
  *total = tot;
  *out = before + x - v;
  return 0;
}

__global__ __launch_bounds__(256) void k_select_plan(const int32_t *__restrict__ cu_vis, int R,
                                                     int64_t tiles_cap,
                                                     int32_t *__restrict__ tile_off,
                                                     int32_t *__restrict__ tile_req,
                                                     int64_t *__restrict__ d_off) {
  __shared__ int64_t sh[4];
  int64_t carry_t = 0, carry_d = 0;
  for (int base = 0; base < R; base += 256) {
    const int r = base + (int)threadIdx.x;
    int64_t nt = 0, nd = 0;
    if (r < R) {
      const int64_t N = cu_vis[r + 1] - cu_vis[r];
      const int64_t tb = (N + kTile - 1) / kTile;
      nt = tb * (tb + 1) / 2;
      nd = N * N;
    }
    int64_t tt, td, pt, pd;
    block_excl_scan_i64(nt, sh, &tt, &pt);
    block_excl_scan_i64(nd, sh, &td, &pd);
    pt += carry_t;
    pd += carry_d;
    if (r < R) {
      tile_off[r] = (int32_t)pt;
      d_off[r] = pd;
      for (int64_t c = 0; c < nt; ++c)
        if (pt + c < tiles_cap) tile_req[pt + c] = r;
    }
    carry_t += tt;
    carry_d += td;
  }
  if (threadIdx.x == 0) {
    tile_off[R] = (int32_t)carry_t;
    d_off[R] = carry_d;
  }
}

// ------------------------------------------------- shared MFMA arithmetic
// One fold chunk: four 16-deep MFMA steps accumulated in fp32 from zero.
// a[s], b[s] hold this lane's operands for step s (row l%32, elements
// chunk*64 + s*16 + (l/32)*8 .. +8). Both the Gram tiles and the norm pass
// go through this function, so equal operands give bitwise-equal sums.
__device__ __forceinline__ f32x16 mfma_chunk(const bf16x8 (&a)[4], const bf16x8 (&b)[4]) {
  f32x16 acc = {};
#pragma unroll
  for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[s], acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
  const uint4 v = *reinterpret_cast<const uint4 *>(p);
  return __builtin_bit_cast(bf16x8, v);
}

// |x_i|^2 for bf16 features: one wave per 32 consecutive rows (rows past
// N_total use zeros; every row's norm only involves itself).
__global__ __launch_bounds__(256) void k_sqnorm_bf16(const uint16_t *__restrict__ X, int64_t N_total,
                                                     int Dv, double *__restrict__ nn) {
  const int lane = threadIdx.x & 63;
  const int64_t row0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 32;
  if (row0 >= N_total) return;
  const int64_t row = row0 + (lane & 31);
  const bool valid = row < N_total;
  const uint16_t *xp = X + (valid ? row : 0) * Dv + (lane >> 5) * 8;
  f32x16 zero = {};
  double acc64[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) acc64[v] = 0.0;
  const int nchunks = (Dv + kKS - 1) / kKS;
  for (int ch = 0; ch < nchunks; ++ch) {
    bf16x8 a[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int kk = ch * kKS + s * 16 + (lane >> 5) * 8;
      if (valid && kk < Dv)
        a[s] = load_bf16x8(xp + ch * kKS + s * 16);
      else
        a[s] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
    }
    const f32x16 acc = mfma_chunk(a, a);
#pragma unroll
    for (int v = 0; v < 16; ++v) acc64[v] += (double)acc[v];
  }
  (void)zero;
  // lane l holds column c = l%32, rows (l/32)*4 + (v%4) + 8*(v/4); the diagonal
  // element of column c sits in the half hi = (c%8)/4 at v = 4*(c/8) + (c%8) - 4*hi.
  const int c = lane & 31, hi = lane >> 5;
  if (((c & 7) >> 2) == hi) {
    const int vsel = 4 * (c >> 3) + (c & 7) - 4 * hi;
    double d = 0.0;
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (v == vsel) d = acc64[v];
    if (row0 + c < N_total) nn[row0 + c] = d;
  }
}

__device__ __forceinline__ float coverage(double dot, double nni, double nnj) {
  // Eq. 10 term: 1 - cos, clamped at 0. Zero-norm rows have cosine 0.
  // Bitwise-identical rows give dot == nni == nnj exactly, hence distance 0.
  if (nni <= 0.0 || nnj <= 0.0) return 1.0f;
  if (dot == nni && nni == nnj) return 0.0f;
  const double t = 1.0 - dot / sqrt(nni * nnj);
  return t > 0.0 ? (float)t : 0.0f;
}

// Map a request-local upper-triangular tile index to (I, J), I <= J.
__device__ __forceinline__ void tile_ij(int t, int nb, int &I, int &J) {
  int i = 0, rem = t;
  while (rem >= nb - i) {
    rem -= nb - i;
    ++i;
  }
  I = i;
  J = i + rem;
}

__global__ __launch_bounds__(kGramThreads) void k_gram_bf16(
    const uint16_t *__restrict__ X, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ tile_off, const int32_t *__restrict__ tile_req,
    const int64_t *__restrict__ d_off, const double *__restrict__ nn, int Dv, int64_t tiles_total,
    int64_t d_cap, float *__restrict__ dmat) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[kTile * kLdsPitch];
  __shared__ __attribute__((aligned(16))) uint16_t sB[kTile * kLdsPitch];

  // XCD-aware order: consecutive logical tiles (same request, shared row
  // blocks) go to the same XCD, which receives every 8th block.
  const int64_t nb_grid = gridDim.x;
  const int64_t per_xcd = nb_grid / 8;
  const int64_t t_glob = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t_glob >= tiles_total) return;
  const int r = tile_req[t_glob];
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int nb = (N + kTile - 1) / kTile;
  int I, J;
  tile_ij((int)(t_glob - tile_off[r]), nb, I, J);
  const int rowA0 = I * kTile, rowB0 = J * kTile;
  const uint16_t *XA = X + (n0 + rowA0) * Dv;
  const uint16_t *XB = X + (n0 + rowB0) * Dv;
  const int nA = min(kTile, N - rowA0), nB = min(kTile, N - rowB0);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wy = wave >> 1, wx = wave & 1;

  double acc64[2][2][16];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc64[mi][ni][v] = 0.0;

  // global -> LDS staging: thread covers rows tid/8 + 32*j, 16-byte piece tid%8
  const int lrow = tid >> 3, lpiece = tid & 7;
  const int nchunks = (Dv + kKS - 1) / kKS;
  uint4 ra[4], rb[4];
  auto gload = [&](int ch) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = lrow + 32 * j;
      const int kk = ch * kKS + lpiece * 8;
      ra[j] = (row < nA && kk < Dv) ? *reinterpret_cast<const uint4 *>(XA + (int64_t)row * Dv + kk)
                                    : make_uint4(0, 0, 0, 0);
      rb[j] = (row < nB && kk < Dv) ? *reinterpret_cast<const uint4 *>(XB + (int64_t)row * Dv + kk)
                                    : make_uint4(0, 0, 0, 0);
    }
  };
  gload(0);
  for (int ch = 0; ch < nchunks; ++ch) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = lrow + 32 * j;
      *reinterpret_cast<uint4 *>(&sA[row * kLdsPitch + lpiece * 8]) = ra[j];
      *reinterpret_cast<uint4 *>(&sB[row * kLdsPitch + lpiece * 8]) = rb[j];
    }
    __syncthreads();
    if (ch + 1 < nchunks) gload(ch + 1);
    bf16x8 a[2][4], b[2][4];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int row = wy * 64 + mi * 32 + (lane & 31);
        a[mi][s] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const uint4 *>(&sA[row * kLdsPitch + s * 16 + (lane >> 5) * 8]));
      }
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int row = wx * 64 + ni * 32 + (lane & 31);
        b[ni][s] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const uint4 *>(&sB[row * kLdsPitch + s * 16 + (lane >> 5) * 8]));
      }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const f32x16 acc = mfma_chunk(a[mi], b[ni]);
#pragma unroll
        for (int v = 0; v < 16; ++v) acc64[mi][ni][v] += (double)acc[v];
      }
  }

  // Epilogue: coverage distances, written to (i, j) and mirrored to (j, i).
  float *D = dmat + d_off[r];
  const double *nnr = nn + n0;
  const int64_t dlim = d_cap - d_off[r];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int j = rowB0 + wx * 64 + ni * 32 + (lane & 31);
      const double nnj = j < N ? nnr[j] : 0.0;
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int ibase = rowA0 + wy * 64 + mi * 32 + (lane >> 5) * 4 + 8 * vq;
        float dv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = ibase + u;
          dv[u] = (i < N && j < N) ? coverage(acc64[mi][ni][4 * vq + u], nnr[i], nnj) : 0.f;
          if (i < N && j < N && (int64_t)i * N + j < dlim) D[(int64_t)i * N + j] = dv[u];
        }
        if (I != J && j < N) {
          const int64_t o = (int64_t)j * N + ibase;
          if (ibase + 3 < N && ((d_off[r] + o) & 3) == 0 && o + 3 < dlim) {
            *reinterpret_cast<float4 *>(D + o) = make_float4(dv[0], dv[1], dv[2], dv[3]);
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (ibase + u < N && o + u < dlim) D[o + u] = dv[u];
          }
        }
      }
    }
}

// fp32 features: squared norms and dots in fp64 FMAs over d = 0..Dv-1 in
// order, the same loop for both, so duplicates again give distance 0.
__global__ __launch_bounds__(256) void k_sqnorm_f32(const float *__restrict__ X, int64_t N_total,
                                                    int Dv, double *__restrict__ nn) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N_total) return;
  const float *x = X + i * Dv;
  double s = 0.0;
  for (int d = 0; d < Dv; ++d) s = fma((double)x[d], (double)x[d], s);
  nn[i] = s;
}

constexpr int kF32Tile = 64;
constexpr int kF32KS = 32;

__global__ __launch_bounds__(256) void k_gram_f32(
    const float *__restrict__ X, const int32_t *__restrict__ cu_vis,
    const int32_t *__restrict__ tile_off, const int32_t *__restrict__ tile_req,
    const int64_t *__restrict__ d_off, const double *__restrict__ nn, int Dv, int64_t tiles_total,
    int64_t d_cap, float *__restrict__ dmat) {
  // A 128x128 Gram tile is covered by 2x2 sub-tiles of 64x64, one pass each.
  __shared__ float sA[kF32KS][kF32Tile + 1];
  __shared__ float sB[kF32KS][kF32Tile + 1];
  const int64_t t_glob = blockIdx.x;
  if (t_glob >= tiles_total) return;
  const int r = tile_req[t_glob];
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int nb = (N + kTile - 1) / kTile;
  int I, J;
  tile_ij((int)(t_glob - tile_off[r]), nb, I, J);
  float *D = dmat + d_off[r];
  const int64_t dlim = d_cap - d_off[r];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  for (int sub = 0; sub < 4; ++sub) {
    const int rowA0 = I * kTile + (sub >> 1) * kF32Tile;
    const int rowB0 = J * kTile + (sub & 1) * kF32Tile;
    if (rowA0 >= N || rowB0 >= N) continue;
    double acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = 0.0;
    for (int k0 = 0; k0 < Dv; k0 += kF32KS) {
      __syncthreads();
      for (int e = threadIdx.x; e < kF32KS * kF32Tile; e += 256) {
        const int row = e / kF32KS, kk = e % kF32KS;
        const int ia = rowA0 + row, ib = rowB0 + row;
        sA[kk][row] = (ia < N && k0 + kk < Dv) ? X[(n0 + ia) * Dv + k0 + kk] : 0.f;
        sB[kk][row] = (ib < N && k0 + kk < Dv) ? X[(n0 + ib) * Dv + k0 + kk] : 0.f;
      }
      __syncthreads();
      const int kmax = min(kF32KS, Dv - k0);
      for (int kk = 0; kk < kmax; ++kk) {
        double av[4], bv[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) av[a] = sA[kk][ty + 16 * a];
#pragma unroll
        for (int b = 0; b < 4; ++b) bv[b] = sB[kk][tx + 16 * b];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = fma(av[a], bv[b], acc[a][b]);
      }
    }
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int i = rowA0 + ty + 16 * a, j = rowB0 + tx + 16 * b;
        if (i >= N || j >= N) continue;
        const float dv = coverage(acc[a][b], nn[n0 + i], nn[n0 + j]);
        if ((int64_t)i * N + j < dlim) D[(int64_t)i * N + j] = dv;
        if (I != J && (int64_t)j * N + i < dlim) D[(int64_t)j * N + i] = dv;
      }
  }
}

// ------------------------------------------------------------ greedy
__device__ __forceinline__ unsigned long long obj_key(float o, int i) {
  // o >= 0 here; its bit pattern orders like its value. Ties -> lowest index.
  return ((unsigned long long)__float_as_uint(o) << 32) | (unsigned long long)(0xFFFFFFFFu - (unsigned)i);
}

__device__ __forceinline__ float clean_score(float w) { return w > 0.f ? w : 0.f; }  // NaN -> 0

// Ascending compaction of flagged elements (element e of thread t is index
// t + e * blockDim). Writes dst[rank] = index.
template <int EPT>
__device__ void compact_ascending(const bool (&flag)[EPT], int32_t *dst, int *sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int base = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const unsigned long long m = __ballot(flag[e]);
    const int before_lane = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) sh[wave] = __popcll(m);
    __syncthreads();
    int before_wave = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
      if (w < wave) before_wave += sh[w];
      tot += sh[w];
    }
    if (flag[e]) dst[base + before_wave + before_lane] = (int32_t)(threadIdx.x + e * blockDim.x);
    base += tot;
    __syncthreads();
  }
}

template <int EPT>
__global__ __launch_bounds__(1024) void k_greedy(const float *__restrict__ scores,
                                                 const float *__restrict__ dmat,
                                                 const int64_t *__restrict__ d_off,
                                                 const int32_t *__restrict__ cu_vis,
                                                 const int32_t *__restrict__ cu_keep,
                                                 int32_t *__restrict__ kept,
                                                 int32_t *__restrict__ order,
                                                 float *__restrict__ gains) {
  __shared__ unsigned long long s_key[2][16];
  __shared__ int s_cnt[16];
  const int r = blockIdx.x;
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const float *D = dmat + d_off[r];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int nth = blockDim.x;

  float w[EPT], dl[EPT];
  bool sel[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = tid + e * nth;
    w[e] = i < N ? clean_score(scores[n0 + i]) : 0.f;
    dl[e] = INFINITY;
    sel[e] = false;
  }
  int j = -1;
  for (int t = 0; t < K; ++t) {
    if (t > 0) {
      const float *row = D + (int64_t)j * N;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int i = tid + e * nth;
        if (i < N) dl[e] = fminf(dl[e], row[i]);
      }
    }
    unsigned long long best = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int i = tid + e * nth;
      if (i < N && !sel[e]) {
        const float o = t == 0 ? w[e] : w[e] * dl[e];
        const unsigned long long kk = obj_key(o, i);
        best = kk > best ? kk : best;
      }
    }
    best = wave_max_u64(best);
    if (lane == 0) s_key[t & 1][wave] = best;
    __syncthreads();
    best = s_key[t & 1][0];
    for (int wv = 1; wv < nw; ++wv) {
      const unsigned long long o = s_key[t & 1][wv];
      best = o > best ? o : best;
    }
    if (best == 0ull) break;   // no unselected token left (budget beyond N): stop
    j = (int)(0xFFFFFFFFu - (unsigned)(best & 0xFFFFFFFFull));
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (tid + e * nth == j) sel[e] = true;
    if (tid == 0) {
      order[k0 + t] = j;
      gains[k0 + t] = __uint_as_float((unsigned)(best >> 32));
    }
  }
  __syncthreads();
  compact_ascending<EPT>(sel, kept + k0, s_cnt);
}

// ------------------------------------------------------------ top-k
template <int EPT>
__global__ __launch_bounds__(1024) void k_topk(const float *__restrict__ scores,
                                               const int32_t *__restrict__ cu_vis,
                                               const int32_t *__restrict__ cu_keep,
                                               int32_t *__restrict__ kept,
                                               int32_t *__restrict__ order,
                                               float *__restrict__ gains) {
  __shared__ int hist[256];
  __shared__ int s_cnt[16];
  __shared__ unsigned s_prefix;
  __shared__ int s_remaining;
  constexpr int kStage = 2048;
  __shared__ unsigned long long s_keys[kStage];
  const int r = blockIdx.x;
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const int tid = threadIdx.x, nth = blockDim.x;

  unsigned key[EPT];
  bool valid[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = tid + e * nth;
    valid[e] = i < N;
    key[e] = valid[e] ? __float_as_uint(clean_score(scores[n0 + i])) : 0u;
  }
  if (tid == 0) {
    s_prefix = 0u;
    s_remaining = K;
  }
  unsigned mask = 0u;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += nth) hist[b] = 0;
    __syncthreads();
    const unsigned prefix = s_prefix;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (valid[e] && (key[e] & mask) == prefix) atomicAdd(&hist[(key[e] >> shift) & 255u], 1);
    __syncthreads();
    if (tid == 0) {
      int cum = 0, rem = s_remaining, d = 255;
      for (; d > 0; --d) {
        if (cum + hist[d] >= rem) break;
        cum += hist[d];
      }
      s_remaining = rem - cum;
      s_prefix = prefix | ((unsigned)d << shift);
    }
    mask |= 255u << shift;
    __syncthreads();
  }
  const unsigned thr = s_prefix;
  const int need = s_remaining;   // how many keys equal to thr to take, lowest index first
  bool take[EPT];
  // rank the threshold-equal keys by index
  {
    const int lane = tid & 63, wave = tid >> 6, nw = nth >> 6;
    int base = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool eq = valid[e] && key[e] == thr;
      const unsigned long long m = __ballot(eq);
      if (lane == 0) s_cnt[wave] = __popcll(m);
      __syncthreads();
      int bw = 0, tot = 0;
      for (int w = 0; w < nw; ++w) {
        if (w < wave) bw += s_cnt[w];
        tot += s_cnt[w];
      }
      const int rank = base + bw + __popcll(m & ((1ull << lane) - 1ull));
      take[e] = valid[e] && (key[e] > thr || (eq && rank < need));
      base += tot;
      __syncthreads();
    }
  }
  compact_ascending<EPT>(take, kept + k0, s_cnt);
  __threadfence_block();
  __syncthreads();
  if (!order && !gains) return;
  // pick order: decreasing score, ties by index; rank = number of kept keys before it
  int rank[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) rank[e] = 0;
  for (int s0 = 0; s0 < K; s0 += kStage) {
    const int ns = min(kStage, K - s0);
    for (int x = tid; x < ns; x += nth) {
      const int i = kept[k0 + s0 + x];
      s_keys[x] = obj_key(__uint_as_float(__float_as_uint(clean_score(scores[n0 + i]))), i);
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (!take[e]) continue;
      const unsigned long long mine = obj_key(__uint_as_float(key[e]), tid + e * nth);
      int c = 0;
      for (int x = 0; x < ns; ++x) c += s_keys[x] > mine ? 1 : 0;
      rank[e] += c;
    }
    __syncthreads();
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    if (!take[e]) continue;
    if (order) order[k0 + rank[e]] = tid + e * nth;
    if (gains) gains[k0 + rank[e]] = __uint_as_float(key[e]);
  }
}

}  // namespace

namespace last {

SelectPlan make_select_plan(int32_t R, const int32_t *cu_vis_h, const int32_t *cu_keep_h,
                            last_sel_mode mode) {
  (void)mode;
  SelectPlan p{};
  p.N_total = cu_vis_h[R];
  p.K_total = cu_keep_h[R];
  for (int r = 0; r < R; ++r) {
    const int64_t N = cu_vis_h[r + 1] - cu_vis_h[r];
    const int64_t K = cu_keep_h[r + 1] - cu_keep_h[r];
    p.N_max = std::max<int32_t>(p.N_max, (int32_t)N);
    p.K_max = std::max<int32_t>(p.K_max, (int32_t)K);
    const int64_t tb = (N + kTile - 1) / kTile;
    p.tiles_total += tb * (tb + 1) / 2;
    p.d_elems += N * N;
  }
  p.threads = p.N_max > 1024 ? 1024 : std::max(64, (p.N_max + 63) / 64 * 64);
  const int ept = (p.N_max + p.threads - 1) / p.threads;
  p.ept = ept <= 1 ? 1 : ept <= 2 ? 2 : ept <= 4 ? 4 : ept <= 8 ? 8 : 16;
  return p;
}

SelectWs carve_select_ws(void *ws, int32_t R, const SelectPlan &p, last_sel_mode mode,
                         size_t *bytes) {
  Carver cv(ws);
  SelectWs w{};
  if (mode == LAST_SEL_KCENTER) {
    w.tile_off = cv.take<int32_t>(R + 1);
    w.tile_req = cv.take<int32_t>(p.tiles_total);
    w.d_off = cv.take<int64_t>(R + 1);
    w.nn = cv.take<double>(p.N_total);
    w.dmat = cv.take<float>(p.d_elems);
  }
  *bytes = cv.size();
  return w;
}

hipError_t launch_select(int32_t R, int32_t Dv, last_dtype fdtype, last_sel_mode mode,
                         const SelectPlan &p, const SelectWs &w, const float *scores,
                         const void *feats, const int32_t *cu_vis, const int32_t *cu_keep,
                         int32_t *kept, int32_t *order, float *gains, hipStream_t s) {
  hipError_t e;
  if (mode == LAST_SEL_TOPK) {
    launch_begin("topk", s);
#define LAST_TOPK(E) \
  hipLaunchKernelGGL(k_topk<E>, dim3(R), dim3(p.threads), 0, s, scores, cu_vis, cu_keep, kept, order, gains)
    switch (p.ept) {
      case 1: LAST_TOPK(1); break;
      case 2: LAST_TOPK(2); break;
      case 4: LAST_TOPK(4); break;
      case 8: LAST_TOPK(8); break;
      default: LAST_TOPK(16); break;
    }
#undef LAST_TOPK
    return launch_end(s);
  }

  launch_begin("select_plan", s);
  hipLaunchKernelGGL(k_select_plan, dim3(1), dim3(256), 0, s, cu_vis, R, p.tiles_total, w.tile_off,
                     w.tile_req, w.d_off);
  if ((e = launch_end(s)) != hipSuccess) return e;

  if (fdtype == LAST_BF16) {
    launch_begin("sqnorm", s);
    const int64_t nblk = (p.N_total + 127) / 128;
    hipLaunchKernelGGL(k_sqnorm_bf16, dim3((unsigned)nblk), dim3(256), 0, s,
                       (const uint16_t *)feats, p.N_total, Dv, w.nn);
    if ((e = launch_end(s)) != hipSuccess) return e;
    launch_begin("gram", s);
    const int64_t grid = (p.tiles_total + 7) / 8 * 8;
    hipLaunchKernelGGL(k_gram_bf16, dim3((unsigned)grid), dim3(kGramThreads), 0, s,
                       (const uint16_t *)feats, cu_vis, w.tile_off, w.tile_req, w.d_off, w.nn, Dv,
                       p.tiles_total, p.d_elems, w.dmat);
    if ((e = launch_end(s)) != hipSuccess) return e;
  } else {
    launch_begin("sqnorm", s);
    hipLaunchKernelGGL(k_sqnorm_f32, dim3((unsigned)((p.N_total + 255) / 256)), dim3(256), 0, s,
                       (const float *)feats, p.N_total, Dv, w.nn);
    if ((e = launch_end(s)) != hipSuccess) return e;
    launch_begin("gram", s);
    hipLaunchKernelGGL(k_gram_f32, dim3((unsigned)p.tiles_total), dim3(256), 0, s,
                       (const float *)feats, cu_vis, w.tile_off, w.tile_req, w.d_off, w.nn, Dv,
                       p.tiles_total, p.d_elems, w.dmat);
    if ((e = launch_end(s)) != hipSuccess) return e;
  }

  launch_begin("greedy", s);
#define LAST_GREEDY(E)                                                                       \
  hipLaunchKernelGGL(k_greedy<E>, dim3(R), dim3(p.threads), 0, s, scores, w.dmat, w.d_off, \
                     cu_vis, cu_keep, kept, order, gains)
  switch (p.ept) {
    case 1: LAST_GREEDY(1); break;
    case 2: LAST_GREEDY(2); break;
    case 4: LAST_GREEDY(4); break;
    case 8: LAST_GREEDY(8); break;
    default: LAST_GREEDY(16); break;
  }
#undef LAST_GREEDY
  return launch_end(s);
}

}  // namespace last
