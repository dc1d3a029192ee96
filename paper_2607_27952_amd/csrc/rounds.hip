// The exact greedy k-center of LAST (arXiv 2607.27952, Sec. 3.4, Eq. 9-11)
// without the N x N coverage matrix, for gfx950.
//
// Step t of the greedy needs the coverage distance of every token to the
// newest pick (Eq. 10). gram.hip forms all N_r^2 distances up front; this file
// forms, as the paper's own incremental form does, only the distances to the
// tokens actually picked (about K_r N_r of them), yet keeps the matrix cores
// busy by taking the picks in rounds:
//
//   - at the start of a round every token's running minimum distance
//     delta_i is exact (every pick so far folded in), hence so is every
//     objective o_i = w_i delta_i and its key (o_i bits, lowest index first);
//   - the round's candidates are the kRB tokens with the largest keys, and T
//     is the largest key left outside them. delta only decreases, so every
//     outside key stays <= T for the rest of the round;
//   - the greedy then runs on the candidates alone, with their mutual
//     distances (a kRB x kRB Gram on the matrix cores): while its best key is
//     above T, that token is the best of the whole request, i.e. exactly the
//     pick the full greedy makes; the round ends at the first key that is
//     not, or after kRP picks;
//   - the round's picks are folded into every token's delta in one pass over
//     the request's features: a kRP-column product on the matrix cores.
// Each round makes at least one pick (the request's best key is a candidate).
// A round whose best objective is 0 (or not a number for every token) ends
// the greedy the way Eq. 9-11 with lowest-index ties do: the rest of the
// budget goes to the lowest-index tokens not yet picked.
//
// Every distance is the number gram.hip stores for the same ordered pair:
// dot products on v_mfma_f32_32x32x16_bf16 in 128-column chunks of fp32
// partial sums, folded into fp64 in column order; the squared norms from
// the same arithmetic; and 1 - dot / (|x_a| |x_b|) multiplied in the order
// gram.hip uses for that pair (its row block's token first). So this form and
// the matrix form pick the same tokens, bit for bit.
//
// Kernels:
//   k_rnorm    |x_i|^2 and 1 / |x_i| of every token (one pass over X).
//   k_rprep    fold-tile prefixes and the per-request state.
//   k_rounds   the rounds, as a queue of tasks on a persistent grid; per
//              request and round: S (select the candidates), C (one 32 x 32
//              block pair of the candidate Gram each), G (the greedy on the
//              candidates), F (fold the picks into 256 tokens each), listed
//              round by round and, within a round, phase by phase. A block
//              takes the next task index from a global counter and waits
//              until the tasks it depends on (all with smaller indices, so
//              already taken by running blocks) have completed: no block
//              ever waits for a block that has not started, so the grid needs
//              no co-residency. Every wait is bounded by a wall-clock limit.
//   k_rfail    after a timeout, marks the unfinished requests invalid.
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace last {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kRThreads = 512;
constexpr int kRWaves = kRThreads / 64;
constexpr int kRB = kRoundCands;              // candidates a round at most
constexpr int kRSub = kRB / 32;               // 32-slot blocks of the candidate list
constexpr int kRPairs = kRoundPairs;
static_assert(kRPairs == kRSub * (kRSub + 1) / 2, "block pairs");
constexpr int kRP = kRoundPicks;              // picks a round at most
constexpr int kFRows = kRoundFoldRows;        // tokens a fold task
constexpr int kFRing = 3;                     // fold ring stages (two in flight)
constexpr int kFCols = 64;                    // columns a ring stage
constexpr int kFTokPieces = kFRows * kFCols * 2 / 16;   // 16-byte pieces of tokens a stage
constexpr int kFPickPieces = kRP * kFCols * 2 / 16;     // ... of picks
constexpr int kFStagePieces = kFTokPieces + kFPickPieces;
constexpr int kFTokInstr = kFTokPieces / 64 / kRWaves;  // LDS-DMA instructions a wave, tokens
static_assert(kFPickPieces == 64 * kRWaves, "one pick DMA instruction a wave");
constexpr int kFPerWave = kFTokInstr + 1;
constexpr int kMaxChunks = kRoundMaxDv / 128;
constexpr int kCT = kRoundCandTasks;           // C tasks per request and round (one block pair each)
static_assert(kCT == kRPairs, "C tasks");
constexpr int kSelLds = kRoundMaxN;           // keys of a request held in LDS by the select
constexpr int kFtLds = 2048;                  // fold-tile prefixes held in LDS (batches of fewer requests)
static_assert(kRB % 64 == 0 && kRB <= 256, "candidate slots: whole waves");
static_assert(kFRows == 32 * kRWaves, "a fold task: 32 tokens a wave");

// Every word one task hands to a task of another block (delta, candidates,
// their distances, picks, state) is written with a device-scope (agent)
// atomic store and read with a device-scope atomic load (the sc1 forms),
// which go to the device's coherence point past the XCDs' separate L2
// caches: a device-scope store is acknowledged there, so once every wave has
// waited for its stores (s_waitcnt) and the block has met at its barrier,
// raising the completion count cannot overtake them. No task writes such a
// word with a plain store, which would need the L2 written back (a release
// fence) before the count; that fence on every task costs 10% of a video
// batch's selection.
__device__ __forceinline__ int ld_i32(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_i32(int32_t *p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_u32(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u32(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_u64(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u64(unsigned long long *p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_f32(const float *p) {
  return __uint_as_float(ld_u32(reinterpret_cast<const uint32_t *>(p)));
}
__device__ __forceinline__ void st_f32(float *p, float v) {
  st_u32(reinterpret_cast<uint32_t *>(p), __float_as_uint(v));
}

__device__ __forceinline__ float clean_score(float w) { return w > 0.f ? w : 0.f; }   // NaN -> 0

// Values that steer branches or loops around barriers are made wave-uniform
// as the compiler sees them (read from the first active lane): a branch on a
// value it takes as per-lane is lowered with exec masks, and around a loop
// with barriers the compiler may then give lanes loop nests of their own,
// in which a block repeats barriers without the lane that fetches its next
// task ever running. All lanes hold the same value wherever these are used.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniu(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }
__device__ __forceinline__ unsigned long long uni64(unsigned long long v) {
  return ((unsigned long long)uniu((uint32_t)(v >> 32)) << 32) | uniu((uint32_t)v);
}
__device__ __forceinline__ int64_t uni_i64(int64_t v) { return (int64_t)uni64((unsigned long long)v); }

// Eq. 10 term for the ordered pair (row token, column token) as gram.hip
// stores it: 1 - cos clamped at 0, zero-norm rows at distance 1, bitwise
// duplicates at 0; dot * inv_a * inv_b multiplied with a = the token of the
// lower 32-row block (the row token within one block), which is the order in
// which the Gram tile that owns the pair evaluates it. The pick's own entry is
// -inf (its selection mark).
__device__ __forceinline__ float coverage_ab(double dot, double nna, double nnb, double inva, double invb) {
  const double t = 1.0 - dot * inva * invb;
  float c = t > 0.0 ? (float)t : 0.0f;
  c = (dot == nna && nna == nnb) ? 0.0f : c;
  c = (nna <= 0.0 || nnb <= 0.0) ? 1.0f : c;
  return c;
}
__device__ __forceinline__ float coverage_dir(int x, int y, double dot, double nnx, double nny, double invx,
                                              double invy) {
  if (x == y) return -INFINITY;
  return (x >> 5) <= (y >> 5) ? coverage_ab(dot, nnx, nny, invx, invy) : coverage_ab(dot, nny, nnx, invy, invx);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

struct RArgs {
  const float *scores;
  const uint16_t *X;
  const double *nn, *inv;
  const int32_t *cu_vis, *cu_keep;
  int32_t *kept, *order;
  float *gains;
  float *dl;                       // [N_total] running minimum distance (+inf before the first pick, -inf once picked)
  int32_t *cand;                   // [R][kRB] this round's candidates (request-local token indices)
  int32_t *picks;                  // [R][kRP] this round's picks
  float *cmat;                     // [R][kRB][kRB] candidate distances, row = pick slot
  int32_t *st;                     // [R][4] picks so far, picks this round, candidates, finished
  unsigned long long *st_T;        // [R] the bound key T
  uint32_t *dcnt;                  // [R] completed tasks
  const int64_t *ftoff;            // [R + 1] fold-tile prefixes
  const unsigned long long *ctl;   // live (low word) and abort (high word), read together
  unsigned long long *head;        // next task index
  uint32_t *live;                  // unfinished requests
  uint32_t *abort_word;            // set on a timeout or an impossible state
  int R, Dv, max_rounds;
  int64_t Q;                       // tasks a round
  int64_t limit;                   // wall-clock ticks a wait may take
};
enum { kStT = 0, kStNp = 1, kStNb = 2, kStFin = 3 };

// ------------------------------------------------------------- LDS layouts
struct SmFold {
  uint4 ring[kFRing][kFStagePieces];
  int pick[kRP];
  double pnn[kRP], pinv[kRP];
};
struct SmCand {
  float part[kMaxChunks][1024];   // fp32 partial sums of each 128-column chunk
  int tok[2][32];
};
struct SmGreedy {
  alignas(16) float mat[kRB * kRB];
};
struct SmSelect {
  uint32_t v[kSelLds];            // key of each token: objective bits + 1, or 0
  uint32_t hist[kRWaves][257];    // per-wave digit counts (padded: waves on different banks)
  uint32_t tot[256];
};
union SmAll {
  SmFold f;
  SmCand c;
  SmGreedy g;
  SmSelect s;
};

// ----------------------------------------------------------- block helpers
__device__ unsigned long long block_max_u64(unsigned long long k, unsigned long long *sh) {
  k = wave_max_key((uint32_t)(k >> 32), (uint32_t)k);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = k;
  __syncthreads();
  unsigned long long m = sh[0];
#pragma unroll
  for (int w = 1; w < kRWaves; ++w) m = sh[w] > m ? sh[w] : m;
  __syncthreads();
  return uni64(m);
}
__device__ uint32_t block_max_u32(uint32_t v, unsigned long long *sh) {
  return (uint32_t)(block_max_u64((unsigned long long)v << 32, sh) >> 32);
}
__device__ uint32_t block_sum_u32(uint32_t v, unsigned long long *sh) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t s = 0;
#pragma unroll
  for (int w = 0; w < kRWaves; ++w) s += (uint32_t)sh[w];
  __syncthreads();
  return uniu(s);
}

// Tokens 0..N-1 in index order: thread t owns the contiguous run of E =
// ceil(N / kRThreads) <= 64 tokens from t E, tests them (loads issued eight at
// a time) into a bit mask, and one block-wide scan of the counts orders the
// runs. emit(rank, i) for the first `limit` tokens with test(load(i), i), on
// the thread that owns i. Returns how many were emitted.
template <typename Load, typename Test, typename Emit>
__device__ int ordered_scan(int N, int limit, Load load, Test test, Emit emit, int *sh) {
  const int E = (N + kRThreads - 1) / kRThreads;
  const int i0 = (int)threadIdx.x * E;
  // each thread starts its run at a different offset, so that the lanes of a
  // wave read different LDS banks
  const int rot = E > 1 ? (int)threadIdx.x % E : 0;
  unsigned long long flags = 0ull;
  for (int k0 = 0; k0 < E; k0 += 8) {
    uint32_t v[8];
    int e[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      e[u] = k0 + u + rot;
      e[u] -= e[u] >= E ? E : 0;
      const int i = i0 + e[u];
      v[u] = (k0 + u < E && i < N) ? load(i) : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + e[u];
      if (k0 + u < E && i < N && test(v[u], i)) flags |= 1ull << e[u];
    }
  }
  int total = 0;
  int rank = block_exclusive_scan(__popcll(flags), sh, &total);
  while (flags) {
    const int e = __ffsll((long long)flags) - 1;
    flags &= flags - 1ull;
    if (rank < limit) emit(rank, i0 + e);
    ++rank;
  }
  return min(uni(total), limit);
}
static_assert(kRoundMaxN <= 64 * kRThreads, "ordered_scan: one 64-bit mask a thread");

// ------------------------------------------------------------------- norms
// |x_i|^2 as the diagonal of a 32 x 32 MFMA Gram of 32 consecutive rows with
// themselves, in the Gram's 128-column chunks; 1 / |x_i| in fp64 (0 for a
// zero row). One wave per 32 rows; two chunks of loads in flight.
__global__ __launch_bounds__(256) void k_rnorm(const uint16_t *__restrict__ X, int64_t N_total, int Dv,
                                               double *__restrict__ nn, double *__restrict__ inv) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = ((int64_t)blockIdx.x * 4 + wave) * 32;
  if (row0 >= N_total) return;
  const int64_t row = min<int64_t>(row0 + (lane & 31), N_total - 1);
  const uint16_t *p = X + row * (int64_t)Dv + 8 * (lane >> 5);
  const int nc = Dv / 128;   // even
  // this lane's diagonal element, if any: column c = lane % 32 sits in half
  // (c % 8) / 4 at accumulator element 4 (c / 8) + c % 4
  const int c = lane & 31;
  const bool has = ((c & 7) >> 2) == (lane >> 5);
  const int vsel = 4 * (c >> 3) + (c & 3);
  double d = 0.0;
  uint4 f0[8], f1[8];
  auto load = [&](uint4 (&f)[8], int ch) {
#pragma unroll
    for (int s = 0; s < 8; ++s) f[s] = *reinterpret_cast<const uint4 *>(p + ch * 128 + 16 * s);
  };
  auto chunk = [&](const uint4 (&f)[8]) {
    f32x16 acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f[0]), as_bf16x8(f[0]), f32x16{}, 0, 0, 0);
#pragma unroll
    for (int s = 1; s < 8; ++s)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(f[s]), as_bf16x8(f[s]), acc, 0, 0, 0);
    float x = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) x = v == vsel ? acc[v] : x;
    d += (double)x;
  };
  load(f0, 0);
  for (int ch = 0; ch < nc; ch += 2) {
    load(f1, ch + 1);
    chunk(f0);
    if (ch + 2 < nc) load(f0, ch + 2);
    chunk(f1);
  }
  if (has && row0 + c < N_total) {
    nn[row0 + c] = d;
    inv[row0 + c] = d > 0.0 ? 1.0 / sqrt(d) : 0.0;
  }
}

// ------------------------------------------------------------------- prep
// Fold-tile prefixes (one F task per kFRows tokens of a request), the state,
// the counters. One block.
__global__ __launch_bounds__(1024) void k_rprep(const int32_t *__restrict__ cu_vis, int R, int64_t *__restrict__ ftoff,
                                                int32_t *__restrict__ st, uint32_t *__restrict__ dcnt,
                                                unsigned long long *__restrict__ head, uint32_t *__restrict__ live,
                                                uint32_t *__restrict__ abort_word) {
  __shared__ int64_t sh[16];
  __shared__ int64_t s_run;
  if (threadIdx.x == 0) {
    s_run = 0;
    *head = 0ull;
    *live = (uint32_t)R;
    *abort_word = 0u;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int base = 0; base < R; base += blockDim.x) {
    const int r = base + (int)threadIdx.x;
    int64_t c = 0;
    if (r < R) {
      const int N = cu_vis[r + 1] - cu_vis[r];
      c = (N + kFRows - 1) / kFRows;
      st[4 * r + kStT] = 0;
      st[4 * r + kStNp] = 0;
      st[4 * r + kStNb] = 0;
      st[4 * r + kStFin] = 0;
      dcnt[r] = 0u;
    }
    int64_t x = c;
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) sh[wave] = x;
    __syncthreads();
    int64_t before = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
      if (w < wave) before += sh[w];
      tot += sh[w];
    }
    if (r < R) ftoff[r] = s_run + before + x - c;
    __syncthreads();
    if (threadIdx.x == 0) s_run += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) ftoff[R] = s_run;
}

// ------------------------------------------------------------------ tasks
struct Req {
  int r;
  int64_t n0, k0;
  int N, K;
};

__device__ void finish_request(const RArgs &a, const Req &q, int *shi) {
  // kept = the tokens marked -inf, ascending (Eq. 12)
  const uint32_t *dl = reinterpret_cast<const uint32_t *>(a.dl + q.n0);
  ordered_scan(
      q.N, q.K, [&](int i) { return ld_u32(dl + i); },
      [&](uint32_t v, int) { return v == __float_as_uint(-INFINITY); },
      [&](int rank, int i) { a.kept[q.k0 + rank] = i; }, shi);
  if (threadIdx.x == 0) {
    st_i32(a.st + 4 * q.r + kStFin, 1);
    __hip_atomic_fetch_add(a.live, 0xFFFFFFFFu, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// S: the round's candidates, or the first pick, the degenerate end, the end.
__device__ void task_select(const RArgs &a, SmAll &sm, const Req &q, unsigned long long *shk, int *shi) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int t = uni(ld_i32(a.st + 4 * q.r + kStT));
  if (t == 0) {
    // delta starts at +inf; the first pick is the most relevant token (Eq. 9)
    unsigned long long best = 0ull;
    for (int i = tid; i < q.N; i += kRThreads) {
      st_f32(a.dl + q.n0 + i, INFINITY);
      const float w = clean_score(a.scores[q.n0 + i]);
      const unsigned long long k = ((unsigned long long)__float_as_uint(w) << 32) | (0xFFFFFFFFu - (unsigned)i);
      best = k > best ? k : best;
    }
    best = block_max_u64(best, shk);
    const int j = (int)(0xFFFFFFFFu - (uint32_t)best);
    vm_wait<0>();   // the +inf stores are complete before the pick's mark
    __syncthreads();
    if (tid == 0) {
      a.order[q.k0] = j;
      a.gains[q.k0] = __uint_as_float((uint32_t)(best >> 32));
      st_f32(a.dl + q.n0 + j, -INFINITY);
      st_i32(a.picks + (int64_t)q.r * kRP, j);
      st_i32(a.st + 4 * q.r + kStNp, 1);
      st_i32(a.st + 4 * q.r + kStNb, 0);
      st_i32(a.st + 4 * q.r + kStT, 1);
    }
    if (q.K == 1) {
      vm_wait<0>();
      __syncthreads();
      finish_request(a, q, shi);
    }
    return;
  }
  if (t >= q.K) {
    finish_request(a, q, shi);
    return;
  }

  // keys: v_i = objective bits + 1, or 0 when w_i delta_i is not a number
  // >= 0 (picked tokens: -inf or NaN)
  SmSelect &s = sm.s;
  uint32_t vmax = 0u, vmin = 0xFFFFFFFFu, nvalid = 0u;
  for (int base = 0; base < q.N; base += 8 * kRThreads) {
    float d[8], w[8];   // eight loads in flight a thread
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = base + u * kRThreads + tid;
      d[u] = i < q.N ? ld_f32(a.dl + q.n0 + i) : 0.f;
      w[u] = i < q.N ? a.scores[q.n0 + i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = base + u * kRThreads + tid;
      if (i >= q.N) continue;
      const float o = clean_score(w[u]) * d[u];
      const uint32_t v = o >= 0.f ? __float_as_uint(o) + 1u : 0u;
      s.v[i] = v;
      vmax = max(vmax, v);
      if (v != 0u) {
        vmin = min(vmin, v);
        ++nvalid;
      }
    }
  }
  vmax = block_max_u32(vmax, shk);
  vmin = ~block_max_u32(~vmin, shk);
  nvalid = block_sum_u32(nvalid, shk);

  if (vmax <= 1u) {
    // the best objective is 0 (or none is a number): from here on every step
    // takes the lowest-index token not yet picked
    const int t0 = t, need = q.K - t;
    const uint32_t *dl = reinterpret_cast<const uint32_t *>(a.dl + q.n0);
    ordered_scan(
        q.N, need, [&](int i) { return ld_u32(dl + i); },
        [&](uint32_t v, int) { return v != __float_as_uint(-INFINITY); },
        [&](int rank, int i) {
          a.order[q.k0 + t0 + rank] = i;
          a.gains[q.k0 + t0 + rank] = 0.f;
          st_f32(a.dl + q.n0 + i, -INFINITY);
        },
        shi);
    vm_wait<0>();
    __syncthreads();
    if (tid == 0) st_i32(a.st + 4 * q.r + kStT, q.K);
    finish_request(a, q, shi);
    return;
  }

  // Candidates: the tokens whose v exceeds a cut, at most kRB of them. The
  // cut is a boundary of 256 bins of width 2^shift over [lo, hi], refined
  // inside the bin that overflows kRB until at least kRB / 2 tokens lie above
  // it; if that bin has shrunk to a single value, its lowest-index tokens
  // fill the candidates up to kRB (at most four passes). T, the largest key
  // not taken, bounds every other token for the rest of the round.
  __shared__ uint32_t s_bin, s_acc;
  __shared__ int s_tie;
  uint32_t cut = 0u;   // candidates: v > cut, and (tie mode) v == cut at indices below tie
  int tie = 0;
  unsigned long long T = 0ull;
  if (nvalid > (uint32_t)kRB) {
    uint32_t lo = vmin, hi = vmax, above = 0u;   // `above`: valid tokens with v > hi
    bool tied = false;
    for (;;) {
      const uint32_t d = hi - lo;
      const int shift = d < 256u ? 0 : 24 - __clz(d);   // (hi - lo) >> shift < 256
      for (int x = tid; x < kRWaves * 257; x += kRThreads) (&s.hist[0][0])[x] = 0u;
      __syncthreads();
      const int wave = tid >> 6;
      for (int i = tid; i < q.N; i += kRThreads) {
        const uint32_t v = s.v[i];
        if (v >= lo && v <= hi && v != 0u) atomicAdd(&s.hist[wave][(v - lo) >> shift], 1u);
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t c = 0;
#pragma unroll
        for (int w = 0; w < kRWaves; ++w) c += s.hist[w][tid];
        s.tot[tid] = c;
      }
      __syncthreads();
      if (tid < 64) {
        // bins 4 lane .. 4 lane + 3; the one bin whose tokens push the count
        // (from the top) past kRB, and the count above it
        const uint32_t c0 = s.tot[4 * lane], c1 = s.tot[4 * lane + 1], c2 = s.tot[4 * lane + 2],
                       c3 = s.tot[4 * lane + 3];
        const uint32_t mine = c0 + c1 + c2 + c3;
        uint32_t incl = mine;   // suffix sum over lanes >= lane
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_down(incl, o);
          if (lane + o < 64) incl += y;
        }
        const uint32_t after = above + incl - mine;
        if (after <= (uint32_t)kRB && after + mine > (uint32_t)kRB) {
          uint32_t acc = after, b;
          if (acc + c3 > (uint32_t)kRB) {
            b = 4 * lane + 3;
          } else if ((acc += c3) + c2 > (uint32_t)kRB) {
            b = 4 * lane + 2;
          } else if ((acc += c2) + c1 > (uint32_t)kRB) {
            b = 4 * lane + 1;
          } else {
            acc += c1;
            b = 4 * lane;
          }
          s_bin = b;
          s_acc = acc;
        }
      }
      __syncthreads();
      const uint32_t b = uniu(s_bin), acc = uniu(s_acc);
      __syncthreads();
      const uint32_t blo = lo + (b << shift);
      const uint32_t bhi = (uint32_t)min<uint64_t>((uint64_t)hi, (uint64_t)blo + ((1ull << shift) - 1ull));
      if (acc >= (uint32_t)kRB / 2) {
        cut = bhi;
        break;
      }
      if (shift == 0) {   // one value: its lowest-index tokens fill the rest
        cut = blo;
        tied = true;
        above = acc;
        break;
      }
      lo = blo;
      hi = bhi;
      above = acc;
    }
    if (tied) {
      // the (kRB - above + 1)-th token (in index order) with v == cut bounds the rest
      const int want = kRB - (int)above + 1;
      if (tid == 0) s_tie = q.N;
      __syncthreads();
      const uint32_t c = cut;
      ordered_scan(
          q.N, want, [&](int i) { return s.v[i]; }, [&](uint32_t v, int) { return v == c; },
          [&](int rank, int i) {
            if (rank == want - 1) s_tie = i;
          },
          shi);
      tie = uni(s_tie);
      T = ((unsigned long long)(cut - 1u) << 32) | (0xFFFFFFFFu - (unsigned)tie);
    } else {
      // T: the largest key among the valid tokens at or below the cut
      unsigned long long best = 0ull;
      for (int i = tid; i < q.N; i += kRThreads) {
        const uint32_t v = s.v[i];
        const unsigned long long k =
            (v != 0u && v <= cut) ? ((unsigned long long)(v - 1u) << 32) | (0xFFFFFFFFu - (unsigned)i) : 0ull;
        best = k > best ? k : best;
      }
      T = block_max_u64(best, shk);
    }
  }
  const uint32_t vs = cut;
  const int ti = tie;
  const int nb = ordered_scan(
      q.N, kRB, [&](int i) { return s.v[i]; },
      [&](uint32_t v, int i) { return v > vs || (v == vs && v != 0u && i < ti); },
      [&](int rank, int i) { st_i32(a.cand + (int64_t)q.r * kRB + rank, i); }, shi);
  if (tid == 0) {
    st_i32(a.st + 4 * q.r + kStNb, nb);
    st_i32(a.st + 4 * q.r + kStNp, 0);
    st_u64(a.st_T + q.r, T);
  }
}

// C: candidate slots [32 sa, 32 sa + 32) against [32 sb, 32 sb + 32), both
// directions. The eight waves take the 128-column chunks in turn (chunk c on
// wave c % 8), keep each chunk's fp32 partial sums in LDS, and the chunks
// are then added in column order in fp64, as the Gram folds them. A wave's
// next chunk is loaded while the matrix cores work on the current one, and
// the norms the distances need are loaded before the chunks.
__device__ void task_cand(const RArgs &a, SmAll &sm, const Req &q, int pair) {
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  int sa = 0, rest = pair;
  while (rest >= kRSub - sa) {
    rest -= kRSub - sa;
    ++sa;
  }
  const int sb = sa + rest;
  const int nb = uni(ld_i32(a.st + 4 * q.r + kStNb));
  if (32 * sb >= nb) return;
  SmCand &c = sm.c;
  if (tid < 64) {
    const int side = tid >> 5, slot = (side ? sb : sa) * 32 + (tid & 31);
    c.tok[side][tid & 31] = ld_i32(a.cand + (int64_t)q.r * kRB + min(slot, nb - 1));
  }
  __syncthreads();
  // this thread's two outputs e = tid + 512 h: A row i, B column j of the
  // 32 x 32 accumulator layout, and the norms of their tokens
  constexpr int kOut = 1024 / kRThreads;
  int ti[kOut], tj[kOut];
  double nni[kOut], nnj[kOut], invi[kOut], invj[kOut];
#pragma unroll
  for (int h = 0; h < kOut; ++h) {
    const int e = tid + h * kRThreads, v = e >> 6, l = e & 63;
    ti[h] = c.tok[0][(l >> 5) * 4 + (v & 3) + 8 * (v >> 2)];
    tj[h] = c.tok[1][l & 31];
    nni[h] = a.nn[q.n0 + ti[h]];
    nnj[h] = a.nn[q.n0 + tj[h]];
    invi[h] = a.inv[q.n0 + ti[h]];
    invj[h] = a.inv[q.n0 + tj[h]];
  }
  const int nc = a.Dv / 128;
  const uint16_t *pa = a.X + (q.n0 + c.tok[0][lane & 31]) * (int64_t)a.Dv + 8 * (lane >> 5);
  const uint16_t *pb = a.X + (q.n0 + c.tok[1][lane & 31]) * (int64_t)a.Dv + 8 * (lane >> 5);
  auto load = [&](int ch, uint4 (&fa)[8], uint4 (&fb)[8]) {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      fa[s] = *reinterpret_cast<const uint4 *>(pa + ch * 128 + 16 * s);
      fb[s] = *reinterpret_cast<const uint4 *>(pb + ch * 128 + 16 * s);
    }
  };
  auto product = [&](int ch, const uint4 (&fa)[8], const uint4 (&fb)[8]) {
    f32x16 acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fa[0]), as_bf16x8(fb[0]), f32x16{}, 0, 0, 0);
#pragma unroll
    for (int s = 1; s < 8; ++s)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fa[s]), as_bf16x8(fb[s]), acc, 0, 0, 0);
#pragma unroll
    for (int v = 0; v < 16; ++v) c.part[ch][v * 64 + lane] = acc[v];
  };
  // chunks wave, wave + 8, ... in two register sets, one chunk ahead
  uint4 xa[8], xb[8], ya[8], yb[8];
  if (wave < nc) load(wave, xa, xb);
  for (int ch = wave; ch < nc; ch += 2 * kRWaves) {
    const int c1 = ch + kRWaves, c2 = ch + 2 * kRWaves;
    if (c1 < nc) load(c1, ya, yb);
    product(ch, xa, xb);
    if (c2 < nc) load(c2, xa, xb);
    if (c1 < nc) product(c1, ya, yb);
  }
  __syncthreads();
  float *M = a.cmat + (int64_t)q.r * kRB * kRB;
#pragma unroll
  for (int h = 0; h < kOut; ++h) {
    const int e = tid + h * kRThreads, v = e >> 6, l = e & 63;
    const int i = (l >> 5) * 4 + (v & 3) + 8 * (v >> 2), j = l & 31;   // A row, B column
    const int si = 32 * sa + i, sj = 32 * sb + j;
    if (si >= nb || sj >= nb) continue;
    double dot = 0.0;
    for (int ch = 0; ch < nc; ++ch) dot += (double)c.part[ch][e];
    st_f32(M + (int64_t)si * kRB + sj, coverage_dir(ti[h], tj[h], dot, nni[h], nnj[h], invi[h], invj[h]));
    if (sa != sb) st_f32(M + (int64_t)sj * kRB + si, coverage_dir(tj[h], ti[h], dot, nnj[h], nni[h], invj[h], invi[h]));
  }
}

// G: the greedy of Eq. 9-11 on the candidates while each pick is certified
// (its key above T), at most kRP picks. Wave 0 runs it; three slots a lane.
__device__ void task_greedy(const RArgs &a, SmAll &sm, const Req &q) {
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int nb = uni(ld_i32(a.st + 4 * q.r + kStNb));
  if (nb == 0) return;
  SmGreedy &g = sm.g;
  const float *M = a.cmat + (int64_t)q.r * kRB * kRB;
  // rows 0..nb-1 whole (columns past nb are never read), two floats a load,
  // eight loads in flight
  const int ne = nb * kRB / 2;
  const unsigned long long *M2 = reinterpret_cast<const unsigned long long *>(M);
  unsigned long long *mat2 = reinterpret_cast<unsigned long long *>(g.mat);
  for (int x0 = tid; x0 < ne; x0 += 8 * kRThreads) {
    unsigned long long v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = x0 + u * kRThreads < ne ? ld_u64(M2 + x0 + u * kRThreads) : 0ull;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (x0 + u * kRThreads < ne) mat2[x0 + u * kRThreads] = v[u];
  }
  __syncthreads();
  if (wave != 0) return;
  constexpr int E = kRB / 64;
  const unsigned long long T = uni64(ld_u64(a.st_T + q.r));
  int t = uni(ld_i32(a.st + 4 * q.r + kStT));
  int np = 0;
  int tok[E];
  float w[E], d[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int c = lane + 64 * e;
    const bool in = c < nb;
    tok[e] = in ? ld_i32(a.cand + (int64_t)q.r * kRB + c) : 0;
    w[e] = in ? clean_score(a.scores[q.n0 + tok[e]]) : 0.f;
    d[e] = in ? ld_f32(a.dl + q.n0 + tok[e]) : -INFINITY;
  }
  for (;;) {
    unsigned long long key[E], best = 0ull;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float o = w[e] * d[e];   // Eq. 11
      key[e] = o >= 0.f ? ((unsigned long long)__float_as_uint(o) << 32) | (0xFFFFFFFFu - (unsigned)tok[e]) : 0ull;
      best = key[e] > best ? key[e] : best;
    }
    const unsigned long long kb = wave_max_key((uint32_t)(best >> 32), (uint32_t)best);
    if ((kb >> 32) == 0ull || kb <= T) break;   // not certified (or the degenerate end)
    int slot = 0;
#pragma unroll
    for (int e = E - 1; e >= 0; --e) {
      const unsigned long long m = __ballot(key[e] == kb);
      if (m) slot = (int)__ffsll((long long)m) - 1 + 64 * e;
    }
    const int j = (int)(0xFFFFFFFFu - (uint32_t)kb);
    if (lane == 0) {
      a.order[q.k0 + t] = j;
      a.gains[q.k0 + t] = __uint_as_float((uint32_t)(kb >> 32));
      st_f32(a.dl + q.n0 + j, -INFINITY);
      st_i32(a.picks + (int64_t)q.r * kRP + np, j);
    }
    ++t;
    ++np;
    if (t >= q.K || np >= kRP) break;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int c = lane + 64 * e;
      if (c < nb) d[e] = fminf(d[e], g.mat[slot * kRB + c]);   // Eq. 10
    }
  }
  if (lane == 0) {
    st_i32(a.st + 4 * q.r + kStT, t);
    st_i32(a.st + 4 * q.r + kStNp, np);
  }
}

// F: fold the round's picks into delta of tokens [kFRows f, kFRows f + kFRows):
// a kFRows x kRP product (tokens x picks) on the matrix cores, both operands
// streamed through an LDS ring by LDS DMA, 64 columns a stage; each wave
// owns 32 tokens against one or two 32-pick tiles.
__device__ void task_fold(const RArgs &a, SmAll &sm, const Req &q, int f) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t = uni(ld_i32(a.st + 4 * q.r + kStT));
  if (t >= q.K) return;   // the last round's picks need no fold (they are marked)
  const int np = uni(ld_i32(a.st + 4 * q.r + kStNp));
  if (np <= 0) return;
  SmFold &F = sm.f;
  if (tid < kRP) {
    const int p = ld_i32(a.picks + (int64_t)q.r * kRP + min(tid, np - 1));
    F.pick[tid] = p;
    F.pnn[tid] = a.nn[q.n0 + p];
    F.pinv[tid] = a.inv[q.n0 + p];
  }
  __syncthreads();
  const int i0 = f * kFRows;
  const int nrows = min(kFRows, q.N - i0);
  const int Dv = a.Dv;
  const int ntn = np > 32 ? 2 : 1;

  // DMA: token instructions x < kFTokInstr cover slots (wave + 8 x) * 64 + lane
  // (rows 0..255); the pick instruction covers slots wave * 64 + lane of the
  // pick part (rows 0..63). Slot = row * 8 + (piece ^ ((row >> 1) & 7)).
  constexpr uint32_t kStageBytes = kFStagePieces * 16;
  uint32_t dst[kFPerWave], voff[kFPerWave];
#pragma unroll
  for (int x = 0; x < kFTokInstr; ++x) {
    const int slot = (wave + kRWaves * x) * 64 + lane, row = slot >> 3, piece = (slot & 7) ^ ((row >> 1) & 7);
    dst[x] = __builtin_amdgcn_readfirstlane(lds_u32(&F.ring[0][(wave + kRWaves * x) * 64]));
    voff[x] = (uint32_t)(((int64_t)min(row, nrows - 1) * Dv + piece * 8) * 2);
  }
  {
    const int slot = wave * 64 + lane, row = slot >> 3, piece = (slot & 7) ^ ((row >> 1) & 7);
    dst[kFTokInstr] = __builtin_amdgcn_readfirstlane(lds_u32(&F.ring[0][kFTokPieces + wave * 64]));
    voff[kFTokInstr] = (uint32_t)(((int64_t)F.pick[row] * Dv + piece * 8) * 2);
  }
  const char *tokbase = (const char *)uniform_ptr(a.X + (q.n0 + i0) * (int64_t)Dv);
  const char *pickbase = (const char *)uniform_ptr(a.X + q.n0 * (int64_t)Dv);
  const int nst = Dv / kFCols;   // even
  auto issue = [&](int st) {
    const uint32_t add = (uint32_t)(st % kFRing) * kStageBytes;
#pragma unroll
    for (int x = 0; x < kFTokInstr; ++x) dma16_nt(dst[x] + add, tokbase + (int64_t)st * kFCols * 2, voff[x]);
    dma16(dst[kFTokInstr] + add, pickbase + (int64_t)st * kFCols * 2, voff[kFTokInstr]);
  };

  int aslot[4], bslot[2][4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int piece = 2 * s + (lane >> 5);
    const int row = 32 * wave + (lane & 31);
    aslot[s] = row * 8 + (piece ^ ((row >> 1) & 7));
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
      const int prow = 32 * tn + (lane & 31);
      bslot[tn][s] = kFTokPieces + prow * 8 + (piece ^ ((prow >> 1) & 7));
    }
  }

  double acc64[2][16];
#pragma unroll
  for (int tn = 0; tn < 2; ++tn)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc64[tn][v] = 0.0;
  f32x16 acc[2] = {f32x16{}, f32x16{}};

  issue(0);
  if (nst > 1) issue(1);
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst)
      vm_wait<kFPerWave>();
    else
      vm_wait<0>();
    __syncthreads();
    if (st + 2 < nst) issue(st + 2);
    const uint4 *ring = F.ring[st % kFRing];
    const bool fresh = (st & 1) == 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bf16x8 fa = as_bf16x8(ring[aslot[s]]);
      const bf16x8 fb0 = as_bf16x8(ring[bslot[0][s]]);
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb0, (fresh && s == 0) ? f32x16{} : acc[0], 0, 0, 0);
      if (ntn > 1) {
        const bf16x8 fb1 = as_bf16x8(ring[bslot[1][s]]);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb1, (fresh && s == 0) ? f32x16{} : acc[1], 0, 0, 0);
      }
    }
    if (st & 1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) acc64[0][v] += (double)acc[0][v];
      if (ntn > 1)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc64[1][v] += (double)acc[1][v];
    }
  }

  // distances, their minimum over the picks (lanes of a half hold one pick
  // column each), and the fold into delta (Eq. 10)
  float m[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int il = 32 * wave + (lane >> 5) * 4 + (v & 3) + 8 * (v >> 2);
    const int i = i0 + il;
    const bool iok = il < nrows;
    const double nni = iok ? a.nn[q.n0 + i] : 1.0, invi = iok ? a.inv[q.n0 + i] : 1.0;
    float mv = INFINITY;
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
      const int k = 32 * tn + (lane & 31);
      if (tn < ntn && k < np && iok) {
        const int p = F.pick[k];
        mv = fminf(mv, coverage_dir(p, i, acc64[tn][v], F.pnn[k], nni, F.pinv[k], invi));
      }
    }
    m[v] = mv;
  }
#pragma unroll
  for (int o = 1; o < 32; o <<= 1)
#pragma unroll
    for (int v = 0; v < 16; ++v) m[v] = fminf(m[v], __shfl_xor(m[v], o));
  if ((lane & 31) < 16) {
    const int vs = lane & 15;
    float mv = m[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) mv = v == vs ? m[v] : mv;
    const int il = 32 * wave + (lane >> 5) * 4 + (vs & 3) + 8 * (vs >> 2);
    if (il < nrows) {
      float *p = a.dl + q.n0 + i0 + il;
      st_f32(p, fminf(ld_f32(p), mv));
    }
  }
}

// ------------------------------------------------------------- the rounds
// The task at position u of a macro-round. The requests form two halves,
// A = [0, RA) and B = [RA, R), half a round apart, so that one half's serial
// chain (select, candidate Gram, greedy) runs while the other half folds.
// Macro-round m lists, in this order:
//   S of A's round m; the first half of B's folds of round m - 1; C (kCT
//   each) of A's round m; G of A's round m; the rest of B's folds; S of B's
//   round m; the first half of A's folds of round m; C and G of B's round m;
//   the rest of A's folds.
// The folds listed between a select and its candidate tasks keep the blocks
// busy while the select runs. Each task depends only on tasks listed before
// it. Sets kind (0 S, 1 C, 2 G, 3 F), the request and the sub-index (C: the
// block pair; F: the fold tile within the request); returns -1 for B's folds
// (they belong to round m - 1), else 0. `ft(i)` is the first fold tile of
// request i (ft(R) the total). Every value is wave-uniform.
template <typename Ft>
__device__ __forceinline__ int64_t decode_task(int64_t u, int64_t R, Ft ft, int &kind, int &r, int &sub) {
  const int64_t RA = (R + 1) / 2, RB = R - RA;
  const int64_t FA = ft(RA), FB = ft(R) - FA, hA = FA / 2, hB = FB / 2;
  // fold tile g of the requests [r0, r0 + nr) (g counts from the first of them)
  auto fold = [&](int64_t r0, int64_t nr, int64_t g) {
    const int64_t f = ft(r0) + g;
    int64_t lo = r0, hi = r0 + nr - 1;   // the last request whose first tile is <= f
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (ft(mid) <= f)
        lo = mid;
      else
        hi = mid - 1;
    }
    kind = 3;
    r = (int)lo;
    sub = (int)(f - ft(lo));
  };
  int64_t x = u;
  if (x < RA) {
    kind = 0;
    r = (int)x;
    return 0;
  }
  x -= RA;
  if (x < hB) {
    fold(RA, RB, x);
    return -1;
  }
  x -= hB;
  if (x < RA * kCT) {
    kind = 1;
    r = (int)(x / kCT);
    sub = (int)(x % kCT);
    return 0;
  }
  x -= RA * kCT;
  if (x < RA) {
    kind = 2;
    r = (int)x;
    return 0;
  }
  x -= RA;
  if (x < FB - hB) {
    fold(RA, RB, hB + x);
    return -1;
  }
  x -= FB - hB;
  if (x < RB) {
    kind = 0;
    r = (int)(RA + x);
    return 0;
  }
  x -= RB;
  if (x < hA) {
    fold(0, RA, x);
    return 0;
  }
  x -= hA;
  if (x < RB * kCT) {
    kind = 1;
    r = (int)(RA + x / kCT);
    sub = (int)(x % kCT);
    return 0;
  }
  x -= RB * kCT;
  if (x < RB) {
    kind = 2;
    r = (int)(RA + x);
    return 0;
  }
  x -= RB;
  fold(0, RA, hA + x);
  return 0;
}

__global__ __launch_bounds__(kRThreads) void k_rounds(RArgs a) {
  __shared__ SmAll sm;
  __shared__ unsigned long long shk[kRWaves];
  __shared__ int shi[kRWaves];
  __shared__ int s_task[4];   // status (0 run, 1 skip, 2 exit, 3 no task), request, kind, sub-index
  __shared__ int s_ft[kFtLds];   // fold-tile prefixes of batches of fewer than kFtLds requests
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uni(tid >> 6);
  if (a.R < kFtLds)
    for (int x = tid; x <= a.R; x += kRThreads) s_ft[x] = (int)a.ftoff[x];
  __syncthreads();
  auto ft_at = [&](int64_t i) -> int64_t { return uni_i64(a.R < kFtLds ? (int64_t)s_ft[i] : a.ftoff[i]); };
  int prev = -1;   // the request of the task this block has just completed
  for (;;) {
    // Wave 0 publishes the completed task (every wave waited for its stores
    // before the last barrier) and takes the next one; all its lanes poll
    // the same words, so its branches stay uniform.
    if (wave == 0) {
      unsigned long long qi = 0ull;
      if (lane == 0) {
        if (prev >= 0) __hip_atomic_fetch_add(a.dcnt + prev, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        qi = __hip_atomic_fetch_add(a.head, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      qi = uni64(qi);
      int status = 0, r = 0, kind = 0, sub = 0;
      const unsigned long long ctl = uni64(ld_u64(a.ctl));   // live requests | abort word << 32
      if ((ctl >> 32) != 0ull || (uint32_t)ctl == 0u) {
        status = 2;
      } else {
        const int64_t m = (int64_t)(qi / (unsigned long long)a.Q);   // macro-round
        const int64_t u = (int64_t)qi - m * a.Q;
        if (m > a.max_rounds) {
          // every request ends by round K_r, and a block runs at most one
          // task ahead of the others: an index this far means a fault
          if (lane == 0) st_u32(a.abort_word, 1u);
          status = 2;
        } else {
          const int64_t tq = decode_task(u, a.R, ft_at, kind, r, sub);
          const int64_t n = m + tq;   // tq = -1: B's folds of the previous round
          const int64_t tiles = ft_at(r + 1) - ft_at(r);
          const int64_t c = 2 + kCT + tiles;
          const int64_t need = n * c + (kind == 0 ? 0 : kind == 1 ? 1 : kind == 2 ? 1 + kCT : 2 + kCT);
          if (n < 0) {
            status = 3;   // B's folds before its first round: no task (nothing to publish)
          } else if (uni(ld_i32(a.st + 4 * r + kStFin)) != 0) {
            status = 1;
          } else {
            const uint64_t t0 = wall_clock64();
            for (;;) {
              if ((int64_t)uniu(ld_u32(a.dcnt + r)) >= need) break;
              if (uni(ld_i32(a.st + 4 * r + kStFin)) != 0) {
                status = 1;
                break;
              }
              if (uniu(ld_u32(a.abort_word)) != 0u) {
                status = 2;
                break;
              }
              if ((int64_t)(wall_clock64() - t0) > a.limit) {
                if (lane == 0) st_u32(a.abort_word, 1u);
                status = 2;
                break;
              }
              __builtin_amdgcn_s_sleep(1);
            }
            if (status == 0 && uni(ld_i32(a.st + 4 * r + kStFin)) != 0) status = 1;
          }
        }
      }
      if (lane == 0) {
        s_task[0] = status;
        s_task[1] = r;
        s_task[2] = kind;
        s_task[3] = sub;
      }
    }
    __syncthreads();
    const int status = uni(s_task[0]);
    if (status == 2) break;
    const int r = uni(s_task[1]), kind = uni(s_task[2]), sub = uni(s_task[3]);
    __syncthreads();
    if (status == 0) {
      Req q;
      q.r = r;
      q.n0 = uni(a.cu_vis[r]);
      q.N = uni(a.cu_vis[r + 1]) - (int)q.n0;
      q.k0 = uni(a.cu_keep[r]);
      q.K = uni(a.cu_keep[r + 1]) - (int)q.k0;
      if (kind == 0)
        task_select(a, sm, q, shk, shi);
      else if (kind == 1)
        task_cand(a, sm, q, sub);
      else if (kind == 2)
        task_greedy(a, sm, q);
      else
        task_fold(a, sm, q, sub);
    }
    // this task's stores are complete before wave 0 publishes it
    vm_wait<0>();
    __syncthreads();
    prev = status == 3 ? -1 : r;
  }
}

// After a timeout: every request not finished gets kept = order = -1 and
// gains = NaN.
__global__ __launch_bounds__(256) void k_rfail(const uint32_t *__restrict__ abort_word, const int32_t *__restrict__ st,
                                               const int32_t *__restrict__ cu_keep, int R, int32_t *__restrict__ kept,
                                               int32_t *__restrict__ order, float *__restrict__ gains) {
  if (*abort_word == 0u) return;
  for (int r = blockIdx.x; r < R; r += gridDim.x) {
    if (st[4 * r + kStFin] != 0) continue;
    for (int k = cu_keep[r] + (int)threadIdx.x; k < cu_keep[r + 1]; k += blockDim.x) {
      kept[k] = -1;
      order[k] = -1;
      gains[k] = __builtin_nanf("");
    }
  }
}

}  // namespace

// ------------------------------------------------------------------- host
bool rounds_supported(int32_t N_max, int32_t Dv, last_dtype fdtype) {
  return fdtype == LAST_BF16 && Dv % 256 == 0 && Dv <= kRoundMaxDv && N_max <= kRoundMaxN &&
         (int64_t)N_max * Dv * 2 < ((int64_t)1 << 32);
}

hipError_t launch_round_norms(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats,
                              hipStream_t s) {
  if (p.N_total == 0) return hipSuccess;
  launch_begin("norms", s);
  hipLaunchKernelGGL(k_rnorm, dim3((unsigned)((p.N_total + 127) / 128)), dim3(256), 0, s,
                     static_cast<const uint16_t *>(feats), p.N_total, Dv, w.nn, w.inv);
  return launch_end(s);
}

hipError_t launch_round_pick(int32_t R, int32_t Dv, const SelectPlan &p, const SelectWs &w, const float *scores,
                             const void *feats, const int32_t *cu_vis, const int32_t *cu_keep, int32_t *kept,
                             int32_t *order, float *gains, hipStream_t s) {
  const int64_t Q = p.round_Q;
  int64_t wait_us = 10000000;
  if (const char *env = getenv("LAST_MC_WAIT_US")) wait_us = std::max<int64_t>(0, atoll(env));
  RArgs a{};
  a.scores = scores;
  a.X = static_cast<const uint16_t *>(feats);
  a.nn = w.nn;
  a.inv = w.inv;
  a.cu_vis = cu_vis;
  a.cu_keep = cu_keep;
  a.kept = kept;
  a.order = order;
  a.gains = gains;
  a.dl = w.r_dl;
  a.cand = w.r_cand;
  a.picks = w.r_picks;
  a.cmat = w.r_cmat;
  a.st = w.r_st;
  a.st_T = w.r_T;
  a.dcnt = w.r_dcnt;
  a.ftoff = w.r_qoff;
  a.head = w.r_ctl;
  a.live = reinterpret_cast<uint32_t *>(w.r_ctl + 1);
  a.abort_word = reinterpret_cast<uint32_t *>(w.r_ctl + 1) + 1;
  a.ctl = w.r_ctl + 1;
  a.R = R;
  a.Dv = Dv;
  const int grid = std::max(1, device_cus());
  // macro-rounds: at most K_max + 1 rounds per request, one more for the
  // second half's last folds, plus those the blocks can be ahead of the last
  // one (each holds one task)
  a.max_rounds = (int)std::min<int64_t>(INT_MAX / 2, p.K_max + 4 + (grid + Q - 1) / Q);
  a.Q = Q;
  a.limit = device_wall_khz() * wait_us / 1000;
  launch_begin("rounds", s);
  hipLaunchKernelGGL(k_rprep, dim3(1), dim3(1024), 0, s, cu_vis, R, w.r_qoff, w.r_st, w.r_dcnt, a.head, a.live,
                     a.abort_word);
  hipLaunchKernelGGL(k_rounds, dim3((unsigned)grid), dim3(kRThreads), 0, s, a);
  hipLaunchKernelGGL(k_rfail, dim3((unsigned)std::min(R, 1024)), dim3(256), 0, s, a.abort_word, w.r_st, cu_keep, R,
                     kept, order, gains);
  return launch_end(s);
}

}  // namespace last
