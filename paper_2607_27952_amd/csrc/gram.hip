// Coverage distances of LAST's k-center (arXiv 2607.27952, Sec. 3.4, Eq. 10)
// for gfx950: per request, the matrix of delta_ij = max(0, 1 - cos(x_i, x_j))
// that the greedy of select.hip reads one row of per step.
//
// The greedy of Eq. 9-11 needs, at each of its K sequential steps, the
// coverage distance of every token to the newest pick. Instead of re-reading
// the request's features every step (a GEMV per step, K full passes over X),
// the distances are formed once as a matrix on the matrix cores:
//
//   k_select_plan   per-request prefixes of the diagonal and off-diagonal
//   k_tile_fill     Gram tiles, the element offset of each request's N_r x N_r
//                   block, and the tile -> request maps (one block a request).
//   k_gram_bf16     128x128 tiles of X_r X_r^T on MFMA
//                   (v_mfma_f32_32x32x16_bf16; bf16 products are exact, the
//                   fp32 accumulator is folded into fp64 every 128 elements),
//                   then delta_ij = max(0, 1 - dot_ij / (|x_i| |x_j|)) in fp64,
//                   stored as fp32, with -inf on the diagonal (a pick's mark,
//                   see k_greedy). A first launch over the diagonal tiles also
//                   yields |x_i|^2 from the same arithmetic (so a row and its
//                   bitwise duplicate get distance exactly 0); a second launch
//                   covers the tiles above the diagonal and mirrors them.
//   k_gram_f32      the same for fp32 features, in fp64 VALU FMAs over
//                   32 x 32 sub-tiles; the diagonal sub-tiles run first and
//                   yield the norms from the same FMA chains.
#include <algorithm>
#include <atomic>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

using last::TileMeta;
using last::cov_blocks;
using last::cov_elems;
using last::cov_index;
using last::kCovTileElems;

constexpr int kTile = last::kGramTile;   // 128
constexpr int kKS = 64;                  // elements per k stage = one fp64 fold chunk

// ------------------------------------------------------------------ plan
__device__ void block_excl_scan_i64(int64_t v, int64_t *sh, int64_t *total, int64_t *out) {
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
}

// Per request: nb = ceil(N / 128) row blocks give nb diagonal Gram tiles and
// nb (nb - 1) / 2 tiles above the diagonal; the coverage matrix (nb x nb
// tiles of 128 x 128) starts at d_off.
//
// ranked (R <= kRankMaxR): the off-diagonal tiles are listed request by request
// in decreasing size (ties: lower index first), rank k being request
// req_order[k], so that a ragged batch's largest requests finish their Gram
// first; otherwise in request order.
__global__ __launch_bounds__(256) void k_select_plan(const int32_t *__restrict__ cu_vis, int R, int ranked,
                                                     int32_t *__restrict__ dtile_off,
                                                     int32_t *__restrict__ otile_off,
                                                     int64_t *__restrict__ d_off,
                                                     int32_t *__restrict__ req_order) {
  __shared__ int64_t sh[4];
  __shared__ int32_t s_n[last::kRankMaxR], s_ord[last::kRankMaxR];
  int64_t carry_d = 0, carry_o = 0, carry_m = 0;
  for (int base = 0; base < R; base += 256) {
    const int r = base + (int)threadIdx.x;
    int64_t nd = 0, no = 0, nm = 0;
    if (r < R) {
      const int64_t N = cu_vis[r + 1] - cu_vis[r];
      nd = (N + kTile - 1) / kTile;
      no = nd * (nd - 1) / 2;
      nm = cov_elems(N);
    }
    int64_t td, to, tm, pd, po, pm;
    block_excl_scan_i64(nd, sh, &td, &pd);
    block_excl_scan_i64(no, sh, &to, &po);
    block_excl_scan_i64(nm, sh, &tm, &pm);
    pd += carry_d;
    po += carry_o;
    pm += carry_m;
    if (r < R) {
      dtile_off[r] = (int32_t)pd;
      if (!ranked) otile_off[r] = (int32_t)po;
      d_off[r] = pm;
    }
    carry_d += td;
    carry_o += to;
    carry_m += tm;
  }
  if (threadIdx.x == 0) {
    dtile_off[R] = (int32_t)carry_d;
    otile_off[R] = (int32_t)carry_o;
    d_off[R] = carry_m;
  }
  if (!ranked) return;
  // rank of r: the requests larger than r, and the equal ones before it
  for (int r = threadIdx.x; r < R; r += 256) s_n[r] = cu_vis[r + 1] - cu_vis[r];
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += 256) {
    const int n = s_n[r];
    int rank = 0;
    for (int q = 0; q < R; ++q) rank += (s_n[q] > n) || (s_n[q] == n && q < r);
    s_ord[rank] = r;
  }
  __syncthreads();
  carry_o = 0;
  for (int base = 0; base < R; base += 256) {
    const int k = base + (int)threadIdx.x;
    int64_t no = 0;
    if (k < R) {
      const int64_t nd = (s_n[s_ord[k]] + kTile - 1) / kTile;
      no = nd * (nd - 1) / 2;
    }
    int64_t to, po;
    block_excl_scan_i64(no, sh, &to, &po);
    if (k < R) {
      otile_off[s_ord[k]] = (int32_t)(po + carry_o);
      req_order[k] = s_ord[k];
    }
    carry_o += to;
  }
}

// Map a request-local index of the tiles strictly above the diagonal to (I, J).
__device__ __forceinline__ void tile_ij_upper(int t, int nb, int &I, int &J) {
  int i = 0, rem = t;
  while (rem >= nb - 1 - i) {
    rem -= nb - 1 - i;
    ++i;
  }
  I = i;
  J = i + 1 + rem;
}

// Tile descriptions, one block per request: every diagonal tile and every
// tile strictly above the diagonal, with its row blocks packed as I << 16 | J.
// Off-diagonal tiles are listed region by region (kRegion x kRegion row
// blocks, regions in upper-triangle order, tiles I-major inside), so the
// tiles that run together share few row blocks and re-read them from cache,
// not HBM. The caps bound every write.
constexpr int kRegion = 8;
// Request r's tiles, given its first diagonal tile pd (of td in all) and its
// first off-diagonal tile po.
__device__ void fill_request_tiles(const int32_t *__restrict__ cu_vis, int r, int R, int64_t pd, int64_t td,
                                   int64_t po, int64_t doff, int64_t diag_cap, int64_t off_cap,
                                   TileMeta *__restrict__ dtile, TileMeta *__restrict__ otile) {
  const int n0 = cu_vis[r], N = cu_vis[r + 1] - n0;
  auto meta = [&](int I, int J) {
    TileMeta m;
    m.n0 = n0;
    m.n = N;
    m.ij = (I << 16) | J;
    m.r = r;
    m.doff = doff;
    m.pad = 0;
    return m;
  };
  const int nb = (N + kTile - 1) / kTile;
  const int64_t o1 = min(po + (int64_t)nb * (nb - 1) / 2, off_cap);
  // Diagonal tiles: the first nb - 1 row blocks of every request in request
  // order, then the last row block of every request (it may be partial), so
  // that a grid-stride walk meets the full tiles first.
  {
    const int64_t head = pd - r, tail = td - R;
    for (int I = threadIdx.x; I < nb; I += 256) {
      const int64_t t = I + 1 < nb ? head + I : tail + r;
      if (t < diag_cap) dtile[t] = meta(I, I);
    }
  }
  const int nR = (nb + kRegion - 1) / kRegion;
  int64_t base = po;
  for (int P = 0; P < nR; ++P)
    for (int Q = P; Q < nR; ++Q) {
      const int i0 = P * kRegion, hI = min(i0 + kRegion, nb) - i0;
      const int j0 = Q * kRegion, hJ = min(j0 + kRegion, nb) - j0;
      const int cnt = P < Q ? hI * hJ : hI * (hI - 1) / 2;
      for (int k = threadIdx.x; k < cnt; k += 256) {
        int I, J;
        if (P < Q) {
          I = i0 + k / hJ;
          J = j0 + k % hJ;
        } else {
          tile_ij_upper(k, hI, I, J);
          I += i0;
          J += i0;
        }
        if (base + k < o1) otile[base + k] = meta(I, J);
      }
      base += cnt;
    }
}

// Tile descriptions, one block per request: every diagonal tile and every
// tile strictly above the diagonal, with its row blocks packed as I << 16 | J.
// Off-diagonal tiles are listed region by region (kRegion x kRegion row
// blocks, regions in upper-triangle order, tiles I-major inside), so the
// tiles that run together share few row blocks and re-read them from cache,
// not HBM. The caps bound every write.
__global__ __launch_bounds__(256) void k_tile_fill(const int32_t *__restrict__ cu_vis,
                                                   const int32_t *__restrict__ dtile_off,
                                                   const int32_t *__restrict__ otile_off,
                                                   const int64_t *__restrict__ d_off,
                                                   int64_t diag_cap, int64_t off_cap,
                                                   TileMeta *__restrict__ dtile,
                                                   TileMeta *__restrict__ otile) {
  const int r = blockIdx.x, R = gridDim.x;
  fill_request_tiles(cu_vis, r, R, dtile_off[r], dtile_off[R], otile_off[r], d_off[r], diag_cap, off_cap, dtile,
                     otile);
}

// The same for a batch in request order (no ranking): the plan and the tile
// lists in one launch, one block a request. A block sums the counts of the
// requests before it (and of all of them, for the totals) itself, in a fixed
// order, instead of reading k_select_plan's prefixes.
__global__ __launch_bounds__(256) void k_plan_fill(const int32_t *__restrict__ cu_vis, int64_t diag_cap,
                                                   int64_t off_cap, int32_t *__restrict__ dtile_off,
                                                   int32_t *__restrict__ otile_off, int64_t *__restrict__ d_off,
                                                   TileMeta *__restrict__ dtile, TileMeta *__restrict__ otile) {
  __shared__ int64_t sh[4][4];
  const int r = blockIdx.x, R = gridDim.x;
  int64_t v[4] = {0, 0, 0, 0};   // diagonal, off-diagonal and matrix elements before r; diagonal in all
  for (int q = threadIdx.x; q < R; q += 256) {
    const int64_t N = cu_vis[q + 1] - cu_vis[q];
    const int64_t nd = (N + kTile - 1) / kTile;
    if (q < r) {
      v[0] += nd;
      v[1] += nd * (nd - 1) / 2;
      v[2] += cov_elems(N);
    }
    v[3] += nd;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    for (int o = 32; o > 0; o >>= 1) v[x] += __shfl_xor(v[x], o);
    if (lane == 0) sh[x][wave] = v[x];
  }
  __syncthreads();
#pragma unroll
  for (int x = 0; x < 4; ++x) v[x] = sh[x][0] + sh[x][1] + sh[x][2] + sh[x][3];
  if (threadIdx.x == 0) {
    dtile_off[r] = (int32_t)v[0];
    otile_off[r] = (int32_t)v[1];
    d_off[r] = v[2];
    if (r == R - 1) {
      const int64_t N = cu_vis[r + 1] - cu_vis[r];
      const int64_t nd = (N + kTile - 1) / kTile;
      dtile_off[R] = (int32_t)(v[0] + nd);
      otile_off[R] = (int32_t)(v[1] + nd * (nd - 1) / 2);
      d_off[R] = v[2] + cov_elems(N);
    }
  }
  fill_request_tiles(cu_vis, r, R, v[0], v[3], v[1], v[2], diag_cap, off_cap, dtile, otile);
}

// The coverage matrix holds -inf on its diagonal instead of a token's distance
// to itself: the greedy folds a pick's own row into its running minimum at the
// next step, and -inf there makes the pick's objective -inf or NaN, which no
// comparison ever prefers -- the pick is marked selected at no extra cost.
constexpr float kSelfMark = -INFINITY;

__device__ __forceinline__ float coverage(double dot, double nni, double nnj, double invi, double invj) {
  // Eq. 10 term: 1 - cos, clamped at 0. Zero-norm rows have cosine 0 (distance
  // 1); bitwise-identical rows give dot == nni == nnj exactly, hence distance
  // 0. Written as selects, in that order of precedence, so that it compiles
  // without branches.
  const double t = 1.0 - dot * invi * invj;
  float c = t > 0.0 ? (float)t : 0.0f;
  c = (dot == nni && nni == nnj) ? 0.0f : c;
  c = (nni <= 0.0 || nnj <= 0.0) ? 1.0f : c;
  return c;
}

// ------------------------------------------------- Gram on the matrix cores
// Dot products accumulate in fp32 over stages of 64 columns (four 16-deep
// v_mfma_f32_32x32x16_bf16 steps starting from zero); each stage's partial
// sums are then added into fp64 totals. Diagonal tiles (which also yield the
// squared norms) and off-diagonal tiles run this same schedule, so equal
// operand rows give bitwise-equal sums.
//
// Block tile 128 x 128 (rows of X_r against rows of X_r), WM x WN waves, each
// wave TM x TN MFMA tiles of 32 x 32. A stage of each operand is 128 rows x
// 64 bf16 in LDS, the 16-byte piece p of row r at slot r*8 + (p ^ ((r>>1)&7))
// so that the fragment reads of 16 consecutive rows hit distinct banks. Two
// stages alternate; the next stage is fetched into registers while the
// current one feeds the matrix cores.
// Block tile 128 x 128: 4 x 2 waves, each 1 x 2 MFMA tiles of 32 x 32.
constexpr int kWM = 4, kWN = 2, kTM = 1, kTN = 2;
constexpr int kGramWaves = kWM * kWN;
constexpr int kGramThreads = 64 * kGramWaves;
constexpr int kPieces = kTile * 8;                     // 16-byte pieces per operand stage
constexpr int kLoadsPerThread = kPieces / kGramThreads;
static_assert(kWM * kTM == 4 && kWN * kTN == 4, "128 x 128 block tile");

__device__ __forceinline__ int lds_slot(int row, int piece) { return row * 8 + (piece ^ ((row >> 1) & 7)); }

template <bool DIAG>
__global__ __launch_bounds__(kGramThreads) void k_gram_bf16_staged(
    const uint16_t *__restrict__ X, const TileMeta *__restrict__ meta, double *__restrict__ nn,
    double *__restrict__ inv, int Dv, int64_t tiles, int64_t d_cap, float *__restrict__ dmat) {
  __shared__ uint4 sA[2][kPieces];
  __shared__ uint4 sB[DIAG ? 1 : 2][DIAG ? 1 : kPieces];
  __shared__ double s_nn[2][kTile], s_inv[2][kTile];   // [0]: rows of A, [1]: rows of B

  int64_t t = blockIdx.x;
  if (!DIAG) {
    // XCD-aware order: consecutive tiles (same request, shared row blocks)
    // go to the same XCD, which receives every 8th block.
    const int64_t per_xcd = gridDim.x / 8;
    t = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  }
  if (t >= tiles) return;
  const TileMeta m = meta[t];
  const int64_t n0 = m.n0;
  const int N = m.n, I = m.ij >> 16, J = m.ij & 0xFFFF;
  const int rowA0 = I * kTile, rowB0 = J * kTile;
  const int nA = min(kTile, N - rowA0), nB = min(kTile, N - rowB0);
  const uint16_t *XA = X + (n0 + rowA0) * Dv;
  const uint16_t *XB = X + (n0 + rowB0) * Dv;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / kWN, wn = wave % kWN;

  double acc64[kTM][kTN][16];
  f32x16 acc[kTM][kTN];
#pragma unroll
  for (int tm = 0; tm < kTM; ++tm)
#pragma unroll
    for (int tn = 0; tn < kTN; ++tn) {
      acc[tm][tn] = f32x16{};
#pragma unroll
      for (int v = 0; v < 16; ++v) acc64[tm][tn][v] = 0.0;
    }

  uint4 ra[kLoadsPerThread], rb[DIAG ? 1 : kLoadsPerThread];
  auto gload = [&](int ch) {
#pragma unroll
    for (int j = 0; j < kLoadsPerThread; ++j) {
      const int e = tid + kGramThreads * j, row = e >> 3, k = ch * kKS + (e & 7) * 8;
      ra[j] = (row < nA && k < Dv) ? *reinterpret_cast<const uint4 *>(XA + (int64_t)row * Dv + k)
                                   : make_uint4(0, 0, 0, 0);
      if (!DIAG)
        rb[DIAG ? 0 : j] = (row < nB && k < Dv) ? *reinterpret_cast<const uint4 *>(XB + (int64_t)row * Dv + k)
                                                : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < kLoadsPerThread; ++j) {
      const int e = tid + kGramThreads * j, slot = lds_slot(e >> 3, e & 7);
      sA[buf][slot] = ra[j];
      if (!DIAG) sB[DIAG ? 0 : buf][slot] = rb[DIAG ? 0 : j];
    }
  };

  const int nch = (Dv + kKS - 1) / kKS;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int ch = 0; ch < nch; ++ch) {
    const int buf = ch & 1;
    if (ch + 1 < nch) gload(ch + 1);
    const uint4 *pa = sA[buf];
    const uint4 *pb = DIAG ? sA[buf] : sB[DIAG ? 0 : buf];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int piece = s * 2 + (lane >> 5);
      bf16x8 a[kTM], b[kTN];
#pragma unroll
      for (int tm = 0; tm < kTM; ++tm)
        a[tm] = __builtin_bit_cast(bf16x8, pa[lds_slot((wm * kTM + tm) * 32 + (lane & 31), piece)]);
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn)
        b[tn] = __builtin_bit_cast(bf16x8, pb[lds_slot((wn * kTN + tn) * 32 + (lane & 31), piece)]);
#pragma unroll
      for (int tm = 0; tm < kTM; ++tm)
#pragma unroll
        for (int tn = 0; tn < kTN; ++tn)
          acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[tm], b[tn], acc[tm][tn], 0, 0, 0);
    }
#pragma unroll
    for (int tm = 0; tm < kTM; ++tm)
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn) {
#pragma unroll
        for (int v = 0; v < 16; ++v) acc64[tm][tn][v] += (double)acc[tm][tn][v];
        acc[tm][tn] = f32x16{};
      }
    if (ch + 1 < nch) sstore((ch + 1) & 1);
    __syncthreads();
  }

  // Squared norms (diagonal tiles) or the norms of both row blocks, into LDS.
  // In a 32 x 32 MFMA tile, lane l holds column l%32 and rows
  // (l/32)*4 + (v%4) + 8*(v/4); column c's diagonal element is in half
  // hi = (c%8)/4 at v = 4*(c/8) + (c%8) - 4*hi.
  if (DIAG) {
#pragma unroll
    for (int tm = 0; tm < kTM; ++tm)
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn) {
        if (wm * kTM + tm != wn * kTN + tn) continue;
        const int c = lane & 31, hi = lane >> 5;
        if (((c & 7) >> 2) != hi) continue;
        const int vsel = 4 * (c >> 3) + (c & 7) - 4 * hi;
        double d = 0.0;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (v == vsel) d = acc64[tm][tn][v];
        s_nn[0][(wm * kTM + tm) * 32 + c] = d;
      }
    __syncthreads();
    for (int i = tid; i < kTile; i += kGramThreads) {
      const double v = s_nn[0][i];
      const double iv = v > 0.0 ? 1.0 / sqrt(v) : 0.0;
      s_inv[0][i] = iv;
      s_nn[1][i] = v;
      s_inv[1][i] = iv;
      if (i < nA) {
        nn[n0 + rowA0 + i] = v;
        inv[n0 + rowA0 + i] = iv;
      }
    }
  } else {
    for (int i = tid; i < 2 * kTile; i += kGramThreads) {
      const int side = i / kTile, x = i % kTile;
      const int row = (side ? rowB0 : rowA0) + x;
      const bool ok = x < (side ? nB : nA);
      s_nn[side][x] = ok ? nn[n0 + row] : 0.0;
      s_inv[side][x] = ok ? inv[n0 + row] : 0.0;
    }
  }
  __syncthreads();

  // Coverage distances into the tile's 128 x 128 block and, off the diagonal,
  // the transposed values into the mirror block (J, I). Entries past N are
  // padding (written as 0). One uniform check guards the request's matrix.
  const int64_t nbr = cov_blocks(N);
  if (m.doff + nbr * nbr * kCovTileElems <= d_cap) {
    float *DA = dmat + m.doff + ((int64_t)I * nbr + J) * kCovTileElems;
    float *DB = dmat + m.doff + ((int64_t)J * nbr + I) * kCovTileElems;
#pragma unroll
    for (int tm = 0; tm < kTM; ++tm)
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn) {
        const int jl = (wn * kTN + tn) * 32 + (lane & 31), j = rowB0 + jl;
        const double nnj = s_nn[1][jl], invj = s_inv[1][jl];
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const int il0 = (wm * kTM + tm) * 32 + (lane >> 5) * 4 + 8 * vq, i0 = rowA0 + il0;
          float dv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int i = i0 + u;
            const float c = DIAG && i == j ? kSelfMark
                                           : coverage(acc64[tm][tn][4 * vq + u], s_nn[0][il0 + u], nnj,
                                                      s_inv[0][il0 + u], invj);
            dv[u] = (i < N && j < N) ? c : 0.f;
            DA[(il0 + u) * kTile + jl] = dv[u];
          }
          if (!DIAG)
            *reinterpret_cast<float4 *>(DB + jl * kTile + il0) = make_float4(dv[0], dv[1], dv[2], dv[3]);
        }
      }
  }
}

// The same tiles with the operands streamed straight into LDS by
// global_load_lds_dwordx4 (lane i's 16 bytes land at M0 + 16 i), through a
// ring of kRing stages of 64 columns (kRingOff for off-diagonal tiles,
// kRingDiag for diagonal ones): the loads for stage ch + kRing - 1 are
// in flight while stage ch feeds the matrix cores. The loads are issued from
// inline assembly so that the compiler does not serialise every LDS read
// behind them; this kernel waits for them itself (s_waitcnt vmcnt) before the
// block barrier that publishes a stage. A fold chunk is two stages (128
// columns); two accumulator sets alternate so that folding chunk c - 1 into
// fp64 can overlap the matrix-core work of chunk c. Needs Dv % 256 == 0 (a
// stage count divisible by 4).
// Diagonal tiles stage one operand (16 KB a stage) and read every row exactly
// once, straight from HBM, so they keep a deeper ring in flight.
//
// The blocks are persistent, one per CU, and walk a list of tiles. While a
// tile's stages run, the block also fetches (by the same LDS DMA, so no
// registers are held) the description of its next tile and, off the
// diagonal, the norms its epilogue needs; the first ring stages of the next
// tile are issued before the epilogue of the current one, so their latency
// hides behind the epilogue's arithmetic and stores.
constexpr int kRingOff = 4, kRingDiag = 8;
constexpr int kChunkTiles = 4;                              // off-diagonal tiles per block per list chunk (about)
static_assert((kRingOff & (kRingOff - 1)) == 0 && (kRingDiag & (kRingDiag - 1)) == 0, "power-of-two ring");
constexpr int kDmaCols = kKS;                               // columns per ring stage (64)
constexpr int kDmaPieces = kTile * kDmaCols * 2 / 16;       // 16-byte pieces per operand stage (1024)
constexpr int kDmaInstr = kDmaPieces / 64;                  // wave instructions per operand stage (16)


// Persistent grid for `tiles` tiles on `cus` compute units: a multiple of 8
// (one share per XCD), at most one block per CU.
inline int64_t persistent_grid(int64_t tiles, int cus) {
  const int64_t cap = std::max(8, cus / 8 * 8);
  return std::min(cap, (tiles + 7) / 8 * 8);
}

template <bool DIAG>
__global__ __launch_bounds__(kGramThreads) void k_gram_bf16(
    const uint16_t *__restrict__ X, const TileMeta *__restrict__ meta, double *__restrict__ nn,
    double *__restrict__ inv, int Dv, int64_t tiles, int64_t d_cap, float *__restrict__ dmat) {
  constexpr int kOps = DIAG ? 1 : 2;
  constexpr int kRing = DIAG ? kRingDiag : kRingOff;
  constexpr int kInstr = kOps * kDmaInstr;                  // per stage, all operands
  static_assert(kInstr % kGramWaves == 0, "even DMA split");
  constexpr int kPerWave = kInstr / kGramWaves;
  constexpr int kSteady = (kRing - 2) * kPerWave;           // loads allowed in flight at a stage boundary
  static_assert(kSteady <= 63, "vmcnt immediate");
  __shared__ uint4 sbuf[kRing][kOps][kDmaPieces];
  __shared__ __align__(16) double s_nn[2][kTile];   // [0]: rows of A, [1]: rows of B
  __shared__ __align__(16) double s_inv[2][kTile];
  __shared__ TileMeta s_next;                        // the next tile, fetched during this one

  // Off the diagonal, XCD x receives blocks x, x + 8, ... (gridDim.x is a
  // multiple of 8). The XCDs walk the region-ordered tile list together, a
  // chunk of 8 ch tiles at a time: XCD x takes the contiguous slice
  // [x ch, (x + 1) ch) of each chunk and its blocks every per-th tile of that
  // slice. So the tiles that run together on one XCD are neighbours and share
  // row blocks in that XCD's L2, and all XCDs stay in one stretch of the list
  // (mostly one request), whose features then stay in the last-level cache.
  // (Giving XCD x the x-th eighth of the whole list put the XCDs on eight
  // different requests at once.) Diagonal tiles share nothing: blocks take
  // them with a plain grid stride, and the list puts every request's last
  // (possibly partial) row block at its tail, so a block takes at most one
  // full tile and one last-block tile before a second full one.
  const int per = DIAG ? (int)gridDim.x : (int)(gridDim.x / 8), xcd = (int)(blockIdx.x % 8);
  const int k_in = DIAG ? (int)blockIdx.x : (int)(blockIdx.x / 8);
  // chunks of about 8 per kChunkTiles tiles, sized evenly so that the last
  // one does not leave most XCDs idle
  const int64_t nchunks = DIAG ? 1 : std::max<int64_t>(1, (tiles + 8LL * per * kChunkTiles - 1) / (8LL * per * kChunkTiles));
  const int64_t ch = DIAG ? 1 : (tiles + 8 * nchunks - 1) / (8 * nchunks);
  auto pos = [&](int64_t c, int j) -> int64_t {
    return DIAG ? k_in + (int64_t)j * per : c * 8 * ch + (int64_t)xcd * ch + k_in + (int64_t)j * per;
  };
  int64_t chunk = 0;
  int step = 0;
  if (!DIAG && k_in >= ch) return;
  int64_t t = pos(0, 0);
  if (t >= tiles) return;

  // the wave index is uniform: keep it (and all that derives from it) scalar
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int nst = Dv / kDmaCols;
  constexpr uint32_t kStageBytes = kOps * kDmaPieces * 16;

  // This wave's DMA instructions: q = wave + kGramWaves * x, operand q / 16,
  // LDS slots (q % 16) * 64 + lane of the stage. The operand's row-block base
  // and the LDS address are wave-uniform (scalar); each lane's byte offset
  // within the row block is fixed for a tile.
  const void *gbase[kPerWave];
  uint32_t voff[kPerWave], dst[kPerWave];
#pragma unroll
  for (int x = 0; x < kPerWave; ++x) {
    const int q = wave + kGramWaves * x, op = q / kDmaInstr, qi = q % kDmaInstr;
    dst[x] = __builtin_amdgcn_readfirstlane(lds_u32(&sbuf[0][op][qi * 64]));
  }
  auto aim = [&](int lane, int64_t n0_, int rowA0_, int rowB0_, int nA_, int nB_) {
#pragma unroll
    for (int x = 0; x < kPerWave; ++x) {
      const int q = wave + kGramWaves * x, op = q / kDmaInstr, qi = q % kDmaInstr;
      const int slot = qi * 64 + lane, row = slot >> 3, piece = (slot & 7) ^ ((row >> 1) & 7);
      const int rr = min(row, (op ? nB_ : nA_) - 1);
      gbase[x] = uniform_ptr(X + (n0_ + (op ? rowB0_ : rowA0_)) * (int64_t)Dv);
      voff[x] = (uint32_t)((rr * (int64_t)Dv + piece * 8) * 2);
    }
  };
  // diagonal tiles read every feature row exactly once (non-temporal: the
  // rows stream past the caches); off-diagonal tiles share row blocks in L2
  auto issue_one = [&](int st, int x) {
    const uint32_t to = dst[x] + (uint32_t)(st & (kRing - 1)) * kStageBytes;
    const char *from = (const char *)gbase[x] + (int64_t)st * kDmaCols * 2;
    if (DIAG) dma16_nt(to, from, voff[x]);
    else dma16(to, from, voff[x]);
  };
  auto issue = [&](int st) {
#pragma unroll
    for (int x = 0; x < kPerWave; ++x) issue_one(st, x);
  };
  auto prologue = [&]() {
    for (int st = 0; st < kRing && st < nst; ++st) issue(st);
  };

  // wait until at most n stages of this wave's loads are still in flight
  // (a literal n folds to one s_waitcnt). Other memory operations issued
  // after those loads (the prefetches, the previous tile's stores) only add
  // to the count, so every wait stays at least as strict.
  auto wait_pending = [&](int n) {
    static_assert(kRing - 1 <= 7, "cases below");
    switch (n) {
      case 7: vm_wait<7 * kPerWave>(); break;
      case 6: vm_wait<6 * kPerWave>(); break;
      case 5: vm_wait<5 * kPerWave>(); break;
      case 4: vm_wait<4 * kPerWave>(); break;
      case 3: vm_wait<3 * kPerWave>(); break;
      case 2: vm_wait<2 * kPerWave>(); break;
      case 1: vm_wait<kPerWave>(); break;
      default: vm_wait<0>(); break;
    }
  };

  // the first tile's description and ring stages
  int64_t n0, doff;
  int N, I, J;
  {
    const TileMeta m = meta[t];
    n0 = m.n0;
    doff = m.doff;
    N = m.n;
    I = m.ij >> 16;
    J = m.ij & 0xFFFF;
  }
  aim((int)threadIdx.x & 63, n0, I * kTile, J * kTile, min(kTile, N - I * kTile), min(kTile, N - J * kTile));
  prologue();

  for (;;) {
    // Lane-dependent values are rebuilt every tile instead of being hoisted
    // out of the tile loop and held (or spilled) across it.
    int tid = (int)threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int rowA0 = I * kTile, rowB0 = J * kTile;
    const int nA = min(kTile, N - rowA0), nB = min(kTile, N - rowB0);
    // (recomputed rather than kept alive through the previous epilogue)
    aim(lane, n0, rowA0, rowB0, nA, nB);
    int64_t chunk_next = chunk;
    int step_next = step + 1;
    if (!DIAG && k_in + (int64_t)step_next * per >= ch) {
      chunk_next = chunk + 1;
      step_next = 0;
    }
    const int64_t t_next = pos(chunk_next, step_next);
    const bool has_next = t_next < tiles;

    // This tile's work in pairs of 32 x 32 sub-tiles: A rows [32 a, 32 a + 32)
    // against B rows [64 c, 64 c + 64). Sub-tile (a, b) is needed iff A row
    // 32 a and B row 32 b exist (partial tiles at a request's end) and, on a
    // diagonal tile, b >= a (the lower triangle is the mirror). Pairs needing
    // both sub-tiles come first, then those needing one, and pair k goes to
    // wave k; waves k and k + 4 share a SIMD, so each SIMD gets an even share
    // of the MFMA work. Waves without a pair only issue their share of the loads.
    static_assert(kTM == 1 && kTN == 2 && kGramWaves == 8, "pair layout of the streamed kernel");
    int my_a = 0, my_b0 = 0, my_nt = 0;
    {
      auto need = [&](int sa, int sb) { return sa * 32 < nA && sb * 32 < nB && (!DIAG || sb >= sa); };
      int k = 0;
#pragma unroll
      for (int pass = 2; pass >= 1; --pass)
#pragma unroll
        for (int sa = 0; sa < 4; ++sa)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const bool n0c = need(sa, 2 * c), n1c = need(sa, 2 * c + 1);
            if ((int)n0c + (int)n1c != pass) continue;
            if (k == wave) {
              my_a = sa;
              my_b0 = n0c ? 2 * c : 2 * c + 1;   // first needed sub-tile column
              my_nt = pass;
            }
            ++k;
          }
    }

    // fragment slots: row (block row) * 8 + (piece ^ ((row >> 1) & 7)); the 16
    // lanes that the LDS serves together read 16 consecutive rows, whose 16-byte
    // slots then fall in 16 distinct bank groups (row parity x swizzled piece)
    int aslot[4], bslot[kTN][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int piece = s * 2 + (lane >> 5);
      const int row = my_a * 32 + (lane & 31);
      aslot[s] = row * 8 + (piece ^ ((row >> 1) & 7));
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn) {
        const int brow = min(my_b0 + tn, 3) * 32 + (lane & 31);
        bslot[tn][s] = brow * 8 + (piece ^ ((brow >> 1) & 7));
      }
    }

    double acc64[kTN][16];
#pragma unroll
    for (int tn = 0; tn < kTN; ++tn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc64[tn][v] = 0.0;

    // Fetches issued once the tile's first stage has landed (every wave has
    // then finished the previous epilogue, which read s_nn, s_inv and s_next):
    // wave 0 the next tile's 32-byte description, and off the diagonal waves
    // 1-4 this tile's norms (128 doubles a side; the arrays carry 128 entries
    // of slack, so a partial row block reads no further than that).
    auto prefetch = [&]() {
      if (wave == 0 && has_next && lane < 2)
        dma16(__builtin_amdgcn_readfirstlane(lds_u32(&s_next)), uniform_ptr(meta + t_next), (uint32_t)lane * 16);
      if (!DIAG && wave >= 1 && wave <= 4) {
        const int w = wave - 1, side = w >> 1;
        const double *src = ((w & 1) ? inv : nn) + n0 + (side ? rowB0 : rowA0);
        const double *to = (w & 1) ? s_inv[side] : s_nn[side];
        dma16(__builtin_amdgcn_readfirstlane(lds_u32(to)), uniform_ptr(src), (uint32_t)lane * 16);
      }
    };

    // The stage loop for a wave with NT sub-tiles (2, 1 or 0), software-
    // pipelined across the stage barrier. A stage's fragments are read in two
    // halves (k-steps 0-1 and 2-3). Stage ch reads its second half while its
    // first half feeds the MFMAs; then it waits for stage ch + 1's loads, meets
    // the other waves at the block barrier (whose fence also completes every
    // wave's reads of stage ch), refills stage ch's ring slot with stage
    // ch + kRing, and reads the first half of stage ch + 1 while its own second
    // half runs. A chunk is two stages (128 columns) accumulated in fp32; chunks
    // alternate between the P and Q sets and each is folded into fp64, a
    // quarter at a time, between the next chunk's MFMAs. nst is a multiple of 4
    // (Dv % 256 == 0); the first folds add zeros, exactly. The ring's first
    // stages were issued before the loop starts.
    auto run = [&](auto nt_const) {
      constexpr int NT = decltype(nt_const)::value;
      f32x16 accP[kTN], accQ[kTN];
      bf16x8 fa0[2], fb0[2][kTN], fa1[2], fb1[2][kTN];
      auto fold_q = [&](const f32x16 (&a)[kTN], int q) {   // elements [4 q, 4 q + 4)
#pragma unroll
        for (int tn = 0; tn < NT; ++tn)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc64[tn][4 * q + v] += (double)a[tn][4 * q + v];
      };
      auto read_half = [&](int ch, int half, bf16x8 (&fa)[2], bf16x8 (&fb)[2][kTN]) {
        if (NT == 0) return;
        const uint4 *pa = sbuf[ch & (kRing - 1)][0];
        const uint4 *pb = sbuf[ch & (kRing - 1)][kOps - 1];
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          fa[ss] = __builtin_bit_cast(bf16x8, pa[aslot[2 * half + ss]]);
#pragma unroll
          for (int tn = 0; tn < NT; ++tn) fb[ss][tn] = __builtin_bit_cast(bf16x8, pb[bslot[tn][2 * half + ss]]);
        }
      };
      auto mma_half = [&](f32x16 (&cur)[kTN], bool fresh, const bf16x8 (&fa)[2], const bf16x8 (&fb)[2][kTN]) {
#pragma unroll
        for (int ss = 0; ss < 2; ++ss)
#pragma unroll
          for (int tn = 0; tn < NT; ++tn)
            cur[tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ss], fb[ss][tn],
                                                              (fresh && ss == 0) ? f32x16{} : cur[tn], 0, 0, 0);
      };
      auto sched_half = [&]() {
        if (NT > 0) {
          constexpr int kMfmaHalf = 2 * (NT > 0 ? NT : 1);   // MFMAs per half stage
          constexpr int kFoldHalf = 8 * (NT > 0 ? NT : 1);   // fold instructions per half stage
          __builtin_amdgcn_sched_group_barrier(0x100, 2 * (1 + NT), 0);
#pragma unroll
          for (int i = 0; i < kMfmaHalf; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, kFoldHalf / kMfmaHalf, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      };
      // `pending`: later stages allowed in flight when stage ch + 1 is needed
      // (-1: ch is the last stage); `refill`: issue stage ch + kRing. Both are
      // literals in the steady loop, so its body has no branches.
      auto stage = [&](int ch, int pending, bool refill, f32x16 (&cur)[kTN], bool fresh,
                       const f32x16 (&prev)[kTN], int h) {
        read_half(ch, 1, fa1, fb1);
        mma_half(cur, fresh, fa0, fb0);
        fold_q(prev, 2 * h);
        sched_half();
        // second half: after the barrier, each MFMA is followed by a share of
        // this wave's loads of stage ch + kRing and two fold elements, in that
        // order, so the load issue does not hold the wave at the barrier
        if (pending >= 0) {
          wait_pending(pending);
          __syncthreads();
          read_half(ch + 1, 0, fa0, fb0);
        }
        if (NT == 0) {
          if (refill) issue(ch + kRing);
        } else {
          constexpr int kM = 2 * (NT > 0 ? NT : 1);
#pragma unroll
          for (int m = 0; m < kM; ++m) {
            const int ss = m / (NT > 0 ? NT : 1), tn = m % (NT > 0 ? NT : 1);
            cur[tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa1[ss], fb1[ss][tn], cur[tn], 0, 0, 0);
            if (refill)
#pragma unroll
              for (int x = m * kPerWave / kM; x < (m + 1) * kPerWave / kM; ++x) issue_one(ch + kRing, x);
#pragma unroll
            for (int e = 2 * m; e < 2 * m + 2; ++e) {
              const int et = e / 4, ev = 4 * (2 * h + 1) + e % 4;
              acc64[et][ev] += (double)prev[et][ev];
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      };
#pragma unroll
      for (int tn = 0; tn < kTN; ++tn) accQ[tn] = f32x16{};
      wait_pending(min(kRing, nst) - 1);   // stage 0 has landed
      __syncthreads();
      prefetch();
      read_half(0, 0, fa0, fb0);
      auto pend = [&](int c) { return c == nst - 1 ? -1 : min(kRing - 2, nst - 2 - c); };
      auto refills = [&](int c) { return c + kRing < nst; };
      int ch = 0;
      for (; ch + kRing + 3 < nst; ch += 4) {
        stage(ch, kRing - 2, true, accP, true, accQ, 0);
        stage(ch + 1, kRing - 2, true, accP, false, accQ, 1);
        stage(ch + 2, kRing - 2, true, accQ, true, accP, 0);
        stage(ch + 3, kRing - 2, true, accQ, false, accP, 1);
      }
      for (; ch < nst; ch += 4) {
        stage(ch, pend(ch), refills(ch), accP, true, accQ, 0);
        stage(ch + 1, pend(ch + 1), refills(ch + 1), accP, false, accQ, 1);
        stage(ch + 2, pend(ch + 2), refills(ch + 2), accQ, true, accP, 0);
        stage(ch + 3, pend(ch + 3), refills(ch + 3), accQ, false, accP, 1);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) fold_q(accQ, q);
    };
    static_assert(kRing <= 8, "waits cover up to 7 pending stages");
    if (my_nt == 2)
      run(std::integral_constant<int, 2>{});
    else if (my_nt == 1)
      run(std::integral_constant<int, 1>{});
    else
      run(std::integral_constant<int, 0>{});
    // Every wave is past its last ring read, and the wait before the last
    // stage covered the prefetches, so s_next, s_nn and s_inv are complete.
    __syncthreads();

    // The next tile: its description, its operand addresses and its first
    // ring stages, in flight during this tile's epilogue.
    int64_t n0_next = 0, doff_next = 0;
    int N_next = 0, I_next = 0, J_next = 0;
    if (has_next) {
      n0_next = __builtin_amdgcn_readfirstlane(s_next.n0);
      doff_next = uniform_i64(s_next.doff);
      N_next = __builtin_amdgcn_readfirstlane(s_next.n);
      const int ij = __builtin_amdgcn_readfirstlane(s_next.ij);
      I_next = ij >> 16;
      J_next = ij & 0xFFFF;
      aim(lane, n0_next, I_next * kTile, J_next * kTile, min(kTile, N_next - I_next * kTile),
          min(kTile, N_next - J_next * kTile));
      prologue();
    }

    // Squared norms of a diagonal tile's rows, from its own diagonal. In a
    // 32 x 32 MFMA tile, lane l holds column l%32 and rows
    // (l/32)*4 + (v%4) + 8*(v/4); column c's diagonal element is in half
    // hi = (c%8)/4 at v = 4*(c/8) + (c%8) - 4*hi.
    if (DIAG) {
      for (int tn = 0; tn < my_nt; ++tn) {
        if (my_b0 + tn != my_a) continue;
        const int c = lane & 31, hi2 = lane >> 5;
        if (((c & 7) >> 2) != hi2) continue;
        const int vsel = 4 * (c >> 3) + (c & 7) - 4 * hi2;
        double d = 0.0;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (v == vsel) d = tn ? acc64[1][v] : acc64[0][v];
        s_nn[0][my_a * 32 + c] = d;
      }
      __syncthreads();
      for (int i = tid; i < kTile; i += kGramThreads) {
        const double v = i < nA ? s_nn[0][i] : 0.0;
        const double iv = v > 0.0 ? 1.0 / sqrt(v) : 0.0;
        s_inv[0][i] = iv;
        s_nn[1][i] = v;
        s_inv[1][i] = iv;
        if (i < nA) {
          nn[n0 + rowA0 + i] = v;
          inv[n0 + rowA0 + i] = iv;
        }
      }
      __syncthreads();
    }

    // Coverage distances into the tile's 128 x 128 block (I, J) and, for
    // sub-tiles strictly above the diagonal, the transposed values into block
    // (J, I): two contiguous 64 KB blocks, every store inside them (entries
    // past N are padding, written as 0). One uniform check guards the
    // request's matrix.
    const int64_t nbr = cov_blocks(N);
    if (doff + nbr * nbr * kCovTileElems <= d_cap) {
      float *DA = dmat + doff + ((int64_t)I * nbr + J) * kCovTileElems;
      float *DB = dmat + doff + ((int64_t)J * nbr + I) * kCovTileElems;
      for (int tn = 0; tn < my_nt; ++tn) {
        const int sb = my_b0 + tn;
        const bool mirror = !DIAG || sb > my_a;
        const int jl = sb * 32 + (lane & 31), j = rowB0 + jl;
        const double nnj = s_nn[1][jl], invj = s_inv[1][jl];
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const int il0 = my_a * 32 + (lane >> 5) * 4 + 8 * vq, i0 = rowA0 + il0;
          float dv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int i = i0 + u;
            const double dot = tn ? acc64[1][4 * vq + u] : acc64[0][4 * vq + u];
            const float c = DIAG && i == j ? kSelfMark
                                           : coverage(dot, s_nn[0][il0 + u], nnj, s_inv[0][il0 + u], invj);
            dv[u] = (i < N && j < N) ? c : 0.f;
            DA[(il0 + u) * kTile + jl] = dv[u];
          }
          if (mirror)
            *reinterpret_cast<float4 *>(DB + jl * kTile + il0) = make_float4(dv[0], dv[1], dv[2], dv[3]);
        }
      }
    }

    if (!has_next) break;
    t = t_next;
    chunk = chunk_next;
    step = step_next;
    n0 = n0_next;
    doff = doff_next;
    N = N_next;
    I = I_next;
    J = J_next;
  }
}

// fp32 features: every dot product, squared norms included, is one fp64 FMA
// chain over d = 0..Dv-1 in order, so a row and its bitwise duplicate get
// distance exactly 0. One launch covers every 32 x 32 sub-tile that a
// request's coverage matrix needs: blocks [0, 16 tiles_diag) take sub-tile
// b % 16 of diagonal tile b / 16 (those below its diagonal return at once),
// the rest the sub-tiles of the off-diagonal tiles. 2 x 2 outputs a thread,
// over 64-column chunks staged through LDS, with four chunks of loads in
// flight. Wave 0 also runs the squared-norm chains of the block's 32 A rows
// and 32 B rows, the same FMAs in the same order as a dot product of a row
// with itself, so no block waits for another's norms. Sub-tiles on a
// diagonal write the norms out; those above it, and every off-diagonal
// sub-tile, also write the mirror.
constexpr int kF32Sub = 32, kF32KS = 64, kF32Subs = (kTile / kF32Sub) * (kTile / kF32Sub);
constexpr int kF32Per = kF32Sub * kF32KS / 256;   // staged elements per thread and operand
constexpr int kF32Ahead = 4;                      // chunks of loads in flight

__global__ __launch_bounds__(256) void k_gram_f32(
    const float *__restrict__ X, const TileMeta *__restrict__ dmeta, const TileMeta *__restrict__ ometa,
    double *__restrict__ nn, double *__restrict__ inv, int Dv, int64_t tiles_diag, int64_t tiles_off,
    int64_t d_cap, float *__restrict__ dmat) {
  __shared__ float sA[kF32KS][kF32Sub + 1];
  __shared__ float sB[kF32KS][kF32Sub + 1];
  __shared__ double s_nn[2][kF32Sub], s_inv[2][kF32Sub];   // [0]: A rows, [1]: B rows
  const int64_t t_glob = blockIdx.x / kF32Subs;
  const int sub = blockIdx.x % kF32Subs, sa = sub / (kTile / kF32Sub), sb = sub % (kTile / kF32Sub);
  const bool on_diag = t_glob < tiles_diag;
  if (t_glob >= tiles_diag + tiles_off) return;
  if (on_diag && sb < sa) return;
  const bool self = on_diag && sb == sa;
  const TileMeta m = on_diag ? dmeta[t_glob] : ometa[t_glob - tiles_diag];
  const int64_t n0 = m.n0;
  const int N = m.n, I = m.ij >> 16, J = m.ij & 0xFFFF;
  const int rowA0 = I * kTile + sa * kF32Sub, rowB0 = J * kTile + sb * kF32Sub;
  if (rowA0 >= N || rowB0 >= N) return;
  float *D = dmat + m.doff;
  const int64_t nbr = cov_blocks(N), dlim = d_cap - m.doff;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;

  // A block has one wave per SIMD, so a chunk's loads cannot hide behind
  // other waves: kF32Ahead chunks are in flight in a register ring while the
  // current one is multiplied.
  float pa[kF32Ahead][kF32Per], pb[kF32Ahead][kF32Per];
  auto fetch = [&](int k0, float (&fa)[kF32Per], float (&fb)[kF32Per]) {
#pragma unroll
    for (int q = 0; q < kF32Per; ++q) {
      const int e = tid + 256 * q, row = e / kF32KS, kk = e % kF32KS;
      const int ia = rowA0 + row, ib = rowB0 + row;
      fa[q] = (ia < N && k0 + kk < Dv) ? X[(n0 + ia) * Dv + k0 + kk] : 0.f;
      fb[q] = (ib < N && k0 + kk < Dv) ? X[(n0 + ib) * Dv + k0 + kk] : 0.f;
    }
  };
  double acc[2][2] = {{0.0, 0.0}, {0.0, 0.0}};
  double nacc = 0.0;   // wave 0: lane l < 32 row l of A, lane l >= 32 row l - 32 of B
  const int nch = (Dv + kF32KS - 1) / kF32KS;
#pragma unroll
  for (int b = 0; b < kF32Ahead; ++b)
    if (b < nch) fetch(b * kF32KS, pa[b], pb[b]);
  for (int c0 = 0; c0 < nch; c0 += kF32Ahead) {
#pragma unroll
    for (int b = 0; b < kF32Ahead; ++b) {
      const int c = c0 + b;
      if (c >= nch) break;
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kF32Per; ++q) {
        const int e = tid + 256 * q, row = e / kF32KS, kk = e % kF32KS;
        sA[kk][row] = pa[b][q];
        sB[kk][row] = pb[b][q];
      }
      __syncthreads();
      if (c + kF32Ahead < nch) fetch((c + kF32Ahead) * kF32KS, pa[b], pb[b]);
      // full chunks unrolled, so the LDS reads of later columns are issued
      // while earlier FMAs run; the FMA order along d is the same either way
      auto mac = [&](int kk) {
        const double a0 = sA[kk][ty], a1 = sA[kk][ty + 16];
        const double b0 = sB[kk][tx], b1 = sB[kk][tx + 16];
        acc[0][0] = fma(a0, b0, acc[0][0]);
        acc[0][1] = fma(a0, b1, acc[0][1]);
        acc[1][0] = fma(a1, b0, acc[1][0]);
        acc[1][1] = fma(a1, b1, acc[1][1]);
        if (tid < 64) {
          const double v = tid < 32 ? sA[kk][tid] : sB[kk][tid - 32];
          nacc = fma(v, v, nacc);
        }
      };
      const int kmax = min(kF32KS, Dv - c * kF32KS);
      if (kmax == kF32KS) {
#pragma unroll
        for (int kk = 0; kk < kF32KS; ++kk) mac(kk);
      } else {
        for (int kk = 0; kk < kmax; ++kk) mac(kk);
      }
    }
  }
  if (tid < 64) {
    const int side = tid >> 5, r = tid & 31;
    s_nn[side][r] = nacc;
    s_inv[side][r] = nacc > 0.0 ? 1.0 / sqrt(nacc) : 0.0;
    if (self && side == 0 && rowA0 + r < N) {
      nn[n0 + rowA0 + r] = nacc;
      inv[n0 + rowA0 + r] = s_inv[0][r];
    }
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int il = ty + 16 * a, jl = tx + 16 * b, i = rowA0 + il, j = rowB0 + jl;
      if (i >= N || j >= N) continue;
      const float dv = self && i == j ? kSelfMark
                                      : coverage(acc[a][b], s_nn[0][il], s_nn[1][jl], s_inv[0][il], s_inv[1][jl]);
      const int64_t oij = cov_index(i, j, nbr), oji = cov_index(j, i, nbr);
      if (oij < dlim) D[oij] = dv;
      if (!self && oji < dlim) D[oji] = dv;
    }
}

}  // namespace

namespace last {

hipError_t launch_gram_plan(int32_t R, const SelectPlan &p, const SelectWs &w, const int32_t *cu_vis,
                            hipStream_t s) {
  launch_begin("select_plan", s);
  if (!p.ranked) {
    hipLaunchKernelGGL(k_plan_fill, dim3(R), dim3(256), 0, s, cu_vis, p.tiles_diag, p.tiles_off, w.dtile_off,
                       w.otile_off, w.d_off, w.dtile, w.otile);
    return launch_end(s);
  }
  hipLaunchKernelGGL(k_select_plan, dim3(1), dim3(256), 0, s, cu_vis, R, 1, w.dtile_off, w.otile_off, w.d_off,
                     w.req_order);
  hipLaunchKernelGGL(k_tile_fill, dim3(R), dim3(256), 0, s, cu_vis, w.dtile_off, w.otile_off, w.d_off,
                     p.tiles_diag, p.tiles_off, w.dtile, w.otile);
  return launch_end(s);
}

bool gram_streamed(last_dtype fdtype, int32_t Dv) { return fdtype == LAST_BF16 && Dv % (4 * kDmaCols) == 0; }

hipError_t launch_gram_diag(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats, int cus,
                            hipStream_t s) {
  launch_begin("gram_diag", s);
  hipLaunchKernelGGL(k_gram_bf16<true>, dim3((unsigned)persistent_grid(p.tiles_diag, cus)), dim3(kGramThreads), 0,
                     s, (const uint16_t *)feats, w.dtile, w.nn, w.inv, Dv, p.tiles_diag, p.d_elems, w.dmat);
  return launch_end(s);
}

hipError_t launch_gram_off(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats, int64_t t0,
                           int64_t nt, int cus, hipStream_t s) {
  if (nt <= 0) return hipSuccess;
  launch_begin("gram", s);
  hipLaunchKernelGGL(k_gram_bf16<false>, dim3((unsigned)persistent_grid(nt, cus)), dim3(kGramThreads), 0, s,
                     (const uint16_t *)feats, w.otile + t0, w.nn, w.inv, Dv, nt, p.d_elems, w.dmat);
  return launch_end(s);
}

hipError_t launch_similarity(int32_t R, int32_t Dv, last_dtype fdtype, const SelectPlan &p,
                             const SelectWs &w, const void *feats, const int32_t *cu_vis,
                             hipStream_t s) {
  hipError_t e;
  if ((e = launch_gram_plan(R, p, w, cu_vis, s)) != hipSuccess) return e;

  if (fdtype == LAST_BF16) {
    // the streamed kernel needs a multiple of four 64-column stages; other widths use the staged one
    if (Dv % (4 * kDmaCols) == 0) {
      const int cus = device_cus();
      launch_begin("gram_diag", s);
      hipLaunchKernelGGL(k_gram_bf16<true>, dim3((unsigned)persistent_grid(p.tiles_diag, cus)), dim3(kGramThreads),
                         0, s, (const uint16_t *)feats, w.dtile, w.nn, w.inv, Dv, p.tiles_diag, p.d_elems, w.dmat);
      if ((e = launch_end(s)) != hipSuccess) return e;
      if (p.tiles_off > 0) {
        launch_begin("gram", s);
        hipLaunchKernelGGL(k_gram_bf16<false>, dim3((unsigned)persistent_grid(p.tiles_off, cus)),
                           dim3(kGramThreads), 0, s, (const uint16_t *)feats, w.otile, w.nn, w.inv, Dv,
                           p.tiles_off, p.d_elems, w.dmat);
        if ((e = launch_end(s)) != hipSuccess) return e;
      }
    } else {
      launch_begin("gram_diag", s);
      hipLaunchKernelGGL(k_gram_bf16_staged<true>, dim3((unsigned)p.tiles_diag), dim3(kGramThreads), 0, s,
                         (const uint16_t *)feats, w.dtile, w.nn, w.inv, Dv, p.tiles_diag, p.d_elems, w.dmat);
      if ((e = launch_end(s)) != hipSuccess) return e;
      if (p.tiles_off > 0) {
        launch_begin("gram", s);
        const int64_t grid = (p.tiles_off + 7) / 8 * 8;
        hipLaunchKernelGGL(k_gram_bf16_staged<false>, dim3((unsigned)grid), dim3(kGramThreads), 0, s,
                           (const uint16_t *)feats, w.otile, w.nn, w.inv, Dv, p.tiles_off, p.d_elems, w.dmat);
        if ((e = launch_end(s)) != hipSuccess) return e;
      }
    }
  } else {
    // one launch: every block computes its own rows' norms
    launch_begin("gram", s);
    hipLaunchKernelGGL(k_gram_f32, dim3((unsigned)((p.tiles_diag + p.tiles_off) * kF32Subs)), dim3(256), 0, s,
                       (const float *)feats, w.dtile, w.otile, w.nn, w.inv, Dv, p.tiles_diag, p.tiles_off,
                       p.d_elems, w.dmat);
    if ((e = launch_end(s)) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace last
