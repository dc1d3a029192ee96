// Selection of LAST (arXiv 2607.27952, Sec. 3.4, Eq. 9-12; Sec. 4.3 Table 5)
// for gfx950, on the coverage distances of gram.hip.
//
//   k_greedy        one block per request; w and delta live in registers.
//                   Step t loads row j_{t-1} of the distance block, folds it
//                   into delta with min, and takes the block-wide argmax of
//                   w * delta (ties -> lowest index, via a 64-bit key of
//                   (value bits, ~index)); picked tokens drop out through the
//                   -inf diagonal. The kept set is compacted in ascending
//                   order at the end (Eq. 12).
//
// Top-k mode (Table 5): k_topk, one block per request, radix-selects the K
// largest scores on their fp32 bit patterns (non-negative floats order like
// their bits), breaks ties at the threshold towards the lowest index, and
// ranks the kept tokens for the pick order.
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <atomic>
#include <math.h>

#include "last_internal.h"

using namespace last_dev;

namespace {

using last::cov_blocks;
using last::cov_elems;
using last::kCovTileElems;

constexpr int kTile = last::kGramTile;   // 128

// ------------------------------------------------------------ greedy
__device__ __forceinline__ unsigned long long obj_key(float o, int i) {
  // o >= 0 here; its bit pattern orders like its value. Ties -> lowest index.
  return ((unsigned long long)__float_as_uint(o) << 32) | (unsigned long long)(0xFFFFFFFFu - (unsigned)i);
}

__device__ __forceinline__ float clean_score(float w) { return w > 0.f ? w : 0.f; }  // NaN -> 0

// Ascending compaction of flagged elements (element e of thread t is index
// value0 + t + e * blockDim). Writes dst[rank] = index.
template <int EPT, typename Flag>
__device__ void compact_ascending(Flag flag, int32_t *dst, int *sh, int32_t value0 = 0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int base = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const bool f = flag(e);
    const unsigned long long m = __ballot(f);
    const int before_lane = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) sh[wave] = __popcll(m);
    __syncthreads();
    int before_wave = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
      if (w < wave) before_wave += sh[w];
      tot += sh[w];
    }
    if (f) dst[base + before_wave + before_lane] = value0 + (int32_t)(threadIdx.x + e * blockDim.x);
    base += tot;
    __syncthreads();
  }
}

// Eq. 9-11 for one request per block of NTH threads (64, 256, 512 or 1024);
// thread t holds tokens t + e * NTH. w is the relevance (NaN for tokens past N_r), dl
// the running minimum coverage distance to the picks so far. A pick j's row of
// the coverage matrix carries -inf at j, so after it is folded in, the pick's
// objective w * dl is -inf or NaN and never wins again. Each thread keeps the
// best (objective, lowest index) of its tokens with a strict compare in
// ascending index order; the block then takes the maximum 64-bit key
// (objective bits, ~index), which orders by objective and breaks ties towards
// the lowest index (objectives are >= 0 here, so their bits order like them).
// req_order (nullable): block b takes the request of rank rank0 + b.
template <int EPT, int NTH>
__global__ __launch_bounds__(NTH) void k_greedy(const float *__restrict__ scores,
                                                const float *__restrict__ dmat,
                                                const int64_t *__restrict__ d_off,
                                                const int32_t *__restrict__ cu_vis,
                                                const int32_t *__restrict__ cu_keep,
                                                const int32_t *__restrict__ req_order, int rank0,
                                                int32_t *__restrict__ kept,
                                                int32_t *__restrict__ order,
                                                float *__restrict__ gains) {
  constexpr int kNW = NTH / 64;
  __shared__ unsigned long long s_key[2][kNW];
  __shared__ int s_cnt[16];
  const int r = req_order ? req_order[rank0 + (int)blockIdx.x] : (int)blockIdx.x;
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const float *D = dmat + d_off[r];
  const int64_t nbr = cov_blocks(N);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // offset of this thread's element e within a row of the tile-major
  // coverage matrix (index clamped into the request, so the tail re-reads
  // element N - 1; those lanes carry NaN relevance and never win). With 1024
  // threads a wave has 128 registers, too few to hold the offsets: there
  // they are rebuilt every step as base + e * 8 tiles (1024 tokens span
  // exactly eight 128-token tile columns), clamped at element N - 1's offset
  // (offsets grow with the index, so the clamp maps exactly the tail).
  constexpr bool kHoldOff = NTH < 1024;
  static_assert(kHoldOff || NTH % kTile == 0, "rebuilt offsets need whole tile columns per e");
  auto cov_off = [&](int e) -> int32_t {
    const int i = min(tid + e * NTH, N - 1);
    return (int32_t)((i / kTile) * kCovTileElems + i % kTile);
  };
  int32_t coff[kHoldOff ? EPT : 1];
  if constexpr (kHoldOff) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) coff[e] = cov_off(e);
  }
  const int32_t off0 = (int32_t)((tid / kTile) * kCovTileElems + tid % kTile);
  const int32_t off_last = (int32_t)(((N - 1) / kTile) * kCovTileElems + (N - 1) % kTile);

  float w[EPT], dl[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) w[e] = scores[n0 + min(tid + e * NTH, N - 1)];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    // tokens past N_r get NaN: every product with NaN is NaN and loses every
    // comparison (-inf could meet the -inf self-mark that a clamped load
    // returns and give +inf, i.e. pick an index past the request)
    w[e] = tid + e * NTH < N ? clean_score(w[e]) : __builtin_nanf("");
    dl[e] = INFINITY;
  }
  // block-wide maximum of a 64-bit key (wave-uniform result)
  auto block_max = [&](unsigned long long k, int t) {
    unsigned long long key = wave_max_key((uint32_t)(k >> 32), (uint32_t)k);
    if (kNW == 1) return key;
    if (lane == 0) s_key[t & 1][wave] = key;
    __syncthreads();
    key = s_key[t & 1][0];
#pragma unroll
    for (int wv = 1; wv < kNW; ++wv) {
      const unsigned long long other = s_key[t & 1][wv];
      key = other > key ? other : key;
    }
    return key;
  };
  auto key_of = [](float bo, int bi) -> unsigned long long {
    return bo >= 0.f ? ((unsigned long long)__float_as_uint(bo) << 32) | (0xFFFFFFFFu - (unsigned)bi) : 0ull;
  };

  // The best (value, lowest index) of this thread's values v[e], in two
  // independent chains (even and odd e, ascending) merged at the end, so that
  // a single wave is not held up by one long chain of dependent compares.
  auto thread_best = [&](const float (&v)[EPT], float &bo, int &bi) {
    float b0 = -1.f, b1 = -1.f;
    int i0 = 0, i1 = 0;
#pragma unroll
    for (int e = 0; e < EPT; e += 2) {
      if (v[e] > b0) {
        b0 = v[e];
        i0 = tid + e * NTH;
      }
      if (e + 1 < EPT && v[e + 1] > b1) {
        b1 = v[e + 1];
        i1 = tid + (e + 1) * NTH;
      }
    }
    const bool take1 = b1 > b0 || (b1 == b0 && i1 < i0);
    bo = take1 ? b1 : b0;
    bi = take1 ? i1 : i0;
  };

  // t = 0: j_1 = argmax w (Eq. 9)
  float bo;
  int bi;
  thread_best(w, bo, bi);
  unsigned long long best = block_max(key_of(bo, bi), 0);
  int j = (int)(0xFFFFFFFFu - (unsigned)(best & 0xFFFFFFFFull));
  if (tid == 0) {
    order[k0] = j;
    gains[k0] = __uint_as_float((unsigned)(best >> 32));
  }
  int taken = 1;
  for (int t = 1; t < K; ++t) {
    // fold the last pick's coverage row into the running minimum (Eq. 10);
    // every load is issued before any is used
    const float *row = D + ((int64_t)(j / kTile) * nbr) * kCovTileElems + (j % kTile) * kTile;
    float o[EPT];   // the row, then the objective in place
    if constexpr (kHoldOff) {
#pragma unroll
      for (int e = 0; e < EPT; ++e) o[e] = row[coff[e]];
    } else {
      int32_t lim = off_last;
      asm volatile("" : "+v"(lim));   // opaque per step: the offsets are not hoisted into registers
#pragma unroll
      for (int e = 0; e < EPT; ++e) o[e] = row[min(off0 + e * (int32_t)((NTH / kTile) * kCovTileElems), lim)];
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      dl[e] = fminf(dl[e], o[e]);
      o[e] = w[e] * dl[e];   // Eq. 11 objective; -inf or NaN once picked, NaN past N_r
    }
    thread_best(o, bo, bi);
    best = block_max(key_of(bo, bi), t);
    if ((best >> 32) == 0ull) {
      // The best objective is 0, or every unpicked token's objective is NaN
      // (+inf relevance at coverage distance 0). Both count as 0, so the pick
      // is the lowest-index token not yet picked (block-uniform branch; never
      // taken while some objective is positive).
      int lo = 0x7FFFFFFF;
#pragma unroll
      for (int e = EPT - 1; e >= 0; --e)
        if (tid + e * NTH < N && dl[e] != -INFINITY) lo = tid + e * NTH;
      // every wave has read this step's exchange slots before they are reused
      if (kNW > 1) __syncthreads();
      best = block_max(lo < N ? (0xFFFFFFFFull - (unsigned)lo) : 0ull, t);
      if (best == 0ull) break;   // every token already picked (cannot happen for K <= N)
    }
    j = (int)(0xFFFFFFFFu - (unsigned)(best & 0xFFFFFFFFull));
    if (tid == 0) {
      order[k0 + t] = j;
      gains[k0 + t] = __uint_as_float((unsigned)(best >> 32));
    }
    ++taken;
  }
  // selected = marked by their own row, plus the last pick (never folded in)
  bool sel[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = tid + e * NTH;
    sel[e] = i < N && (dl[e] == -INFINITY || i == j);
  }
  (void)taken;
  __syncthreads();
  compact_ascending<EPT>([&](int e) { return sel[e]; }, kept + k0, s_cnt);
}
// The greedy of Eq. 9-11 over several compute units, for requests longer than
// one block's registers hold. Request rb of the launch runs on S blocks of
// kMcThreads; block s holds tokens [s SL, (s + 1) SL), SL = kMcThreads * EPT,
// EPT a thread in registers. Every step each block folds its slice of the
// newest pick's coverage row into delta, takes its slice's best (objective,
// lowest index) and publishes it as a tagged 64-bit key in its slot of the
// step's parity; wave 0 then polls the request's S slots until all carry this
// step's tag and takes their maximum, the next pick, which every block of the
// request so computes alike. Key: tag (bits 63-62) | objective bits (61-30) |
// 2^30 - 1 - index (29-0); objectives are >= 0, so the maximum orders by
// objective and breaks ties towards the lowest index, and a slice with nothing
// left publishes the tag alone. The tag, step % 3 + 1, is never 0 (the slots
// start zeroed) and tells a step from the one two steps earlier, the only
// other content a slot of that parity can hold: a block cannot publish step
// t + 2 before every block has published step t + 1, which each does only
// after reading step t. An objective that is NaN (+inf relevance at distance
// 0) counts as 0, as does relevance that is not > 0, as in the one-block
// greedy. At the end the blocks exchange their pick counts the same way and
// write their picks into `kept` at their offsets, in ascending order.
//
// The S blocks of a request must run at the same time: the host launches at
// most a quarter of the blocks the device holds at once, so each request's
// blocks are all resident as soon as other work leaves room. Every wait is
// bounded by `limit` ticks of the constant-rate wall clock (the slots of the
// launch's ranks are zeroed before it); a block that times out sets the
// request's abort word, and every block that sees it, or times out itself,
// fills the request's kept and order with -1 and its gains with NaN.
constexpr int kMcThreads = 256;
constexpr int kMcMaxS = 64;                // slices a request (one per lane of the polling wave)
constexpr int kMcSlotWords = last::kMcSlotWords;  // per request: two step parities, the counts, the abort word
static_assert(kMcSlotWords == 4 * kMcMaxS, "exchange words: two step parities, the counts, the abort word");

__device__ __forceinline__ unsigned long long mc_key(unsigned tag, unsigned obits, int i) {
  return ((unsigned long long)tag << 62) | ((unsigned long long)obits << 30) |
         (unsigned long long)((1u << 30) - 1u - (unsigned)i);
}

__global__ __launch_bounds__(256) void k_zero_u64(unsigned long long *__restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = 0ull;
}

template <int EPT>
__global__ __launch_bounds__(kMcThreads) void k_greedy_mc(const float *__restrict__ scores,
                                                          const float *__restrict__ dmat,
                                                          const int64_t *__restrict__ d_off,
                                                          const int32_t *__restrict__ cu_vis,
                                                          const int32_t *__restrict__ cu_keep,
                                                          const int32_t *__restrict__ req_order, int rank0, int nreq,
                                                          int S, int spread,
                                                          unsigned long long *__restrict__ slots, int64_t limit,
                                                          int32_t *__restrict__ kept, int32_t *__restrict__ order,
                                                          float *__restrict__ gains) {
  constexpr int NTH = kMcThreads, kNW = NTH / 64, SL = NTH * EPT;
  __shared__ unsigned long long s_key[2][kNW];
  __shared__ unsigned long long s_pick, s_next;
  __shared__ float s_pre[2][SL];   // this slice of two prefetched coverage rows
  __shared__ int s_cnt[16];
  __shared__ int s_abort;
  // Workgroup b runs on XCD b % 8. Alone on the device, the S blocks of a
  // request share an XCD (request rb of the launch on XCD rb % 8), whose
  // exchange is about a fifth faster than one spread over XCDs; beside the
  // Gram (`spread`), whose persistent grid leaves a few compute units free on
  // every XCD, consecutive blocks form a request and so spread over the XCDs.
  // Blocks past the last request exit.
  const int xcd = (int)blockIdx.x % 8, kx = (int)blockIdx.x / 8;
  const int rb = spread ? (int)blockIdx.x / S : (kx / S) * 8 + xcd;
  const int sl = spread ? (int)blockIdx.x % S : kx % S;
  if (rb >= nreq) return;
  const int r = req_order ? req_order[rank0 + rb] : rank0 + rb;
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const float *D = dmat + d_off[r];
  const int64_t nbr = cov_blocks(N);
  unsigned long long *slot = slots + (int64_t)(rank0 + rb) * kMcSlotWords;
  unsigned long long *abort_word = slot + 3 * kMcMaxS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int base = sl * SL;
  if (tid == 0) s_abort = 0;

  // tokens past N_r count as picked (delta -inf) and read element N_r - 1
  int32_t coff[EPT];
  float w[EPT], dl[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = min(base + tid + e * NTH, N - 1);
    coff[e] = (int32_t)((i / kTile) * kCovTileElems + i % kTile);
    const bool in = base + tid + e * NTH < N;
    w[e] = in ? clean_score(scores[n0 + i]) : 0.f;
    dl[e] = in ? INFINITY : -INFINITY;
  }
  auto block_max = [&](unsigned long long k, int t) {
    unsigned long long key = wave_max_key((uint32_t)(k >> 32), (uint32_t)k);
    if (lane == 0) s_key[t & 1][wave] = key;
    __syncthreads();
    key = s_key[t & 1][0];
#pragma unroll
    for (int wv = 1; wv < kNW; ++wv) {
      const unsigned long long other = s_key[t & 1][wv];
      key = other > key ? other : key;
    }
    return key;
  };
  // Wave 0: publish `mine` in slot `at + sl`, then wait until every slot
  // at .. at + S - 1 carries `tag` in bits 63-62, or the abort word is set, or
  // `limit` ticks pass (then set the abort word). Returns the slots' maximum
  // (lanes >= S read as the tag alone) and the per-lane values in `v`.
  auto publish_wait = [&](unsigned long long *at, unsigned long long mine, unsigned tag,
                          unsigned long long &v) -> unsigned long long {
    if (lane == 0) __hip_atomic_store(at + sl, mine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long none = (unsigned long long)tag << 62;
    const uint64_t t0 = wall_clock64();
    for (;;) {
      v = lane < S ? __hip_atomic_load(at + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : none;
      if (__all((unsigned)(v >> 62) == tag)) break;
      const unsigned long long ab = __hip_atomic_load(abort_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (ab != 0ull) {
        if (lane == 0) s_abort = 1;
        break;
      }
      if ((int64_t)(wall_clock64() - t0) > limit) {
        if (lane == 0) {
          __hip_atomic_store(abort_word, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          s_abort = 1;
        }
        break;
      }
    }
    return wave_max_key((uint32_t)(v >> 32), (uint32_t)v);
  };
  // the slice's best as a request-wide pick (block-uniform, after a barrier)
  auto exchange = [&](const float (&o)[EPT], int t) -> unsigned long long {
    float b0 = -1.f, b1 = -1.f;
    int i0 = 0, i1 = 0;
#pragma unroll
    for (int e = 0; e < EPT; e += 2) {   // two chains, ascending index in each
      if (o[e] > b0) {
        b0 = o[e];
        i0 = base + tid + e * NTH;
      }
      if (o[e + 1] > b1) {
        b1 = o[e + 1];
        i1 = base + tid + (e + 1) * NTH;
      }
    }
    const bool take1 = b1 > b0 || (b1 == b0 && i1 < i0);
    const float bo = take1 ? b1 : b0;
    const int bi = take1 ? i1 : i0;
    const unsigned long long lk =
        block_max(bo >= 0.f ? ((unsigned long long)__float_as_uint(bo) << 32) | (0xFFFFFFFFu - (unsigned)bi) : 0ull, t);
    if (wave == 0) {
      const unsigned tag = (unsigned)(t % 3) + 1u;
      const unsigned long long mine =
          lk ? mc_key(tag, (unsigned)(lk >> 32), (int)(0xFFFFFFFFu - (unsigned)lk)) : (unsigned long long)tag << 62;
      unsigned long long v;
      const unsigned long long best = publish_wait(slot + (t & 1) * kMcMaxS, mine, tag, v);
      // the runner-up: the best of the other slices' candidates
      const unsigned long long v2 = v == best ? (unsigned long long)tag << 62 : v;
      const unsigned long long next = wave_max_key((uint32_t)(v2 >> 32), (uint32_t)v2);
      if (lane == 0) {
        s_pick = best;
        s_next = next;
      }
    }
    __syncthreads();
    return s_pick;
  };
  auto pick_of = [](unsigned long long k) { return (int)((1u << 30) - 1u - (unsigned)(k & ((1ull << 30) - 1ull))); };
  auto gain_of = [](unsigned long long k) { return __uint_as_float((unsigned)(k >> 30)); };

  // The runner-up of a step's exchange is usually the next step's pick. Its
  // row (this slice of it) is copied into LDS straight away, into s_pre[t & 1]
  // at step t, with one LDS-DMA load per token a thread, each wave filling the
  // part its own threads read; if it is the pick, step t + 2 folds it from LDS
  // instead of waiting on memory. pre[b]: the row in s_pre[b] (block-uniform),
  // or -1; dma_t: the step whose exchange issued the newest copy.
  int pre[2] = {-1, -1};
  int dma_t = -2;
  // this slice of row u into s_pre[b], each wave the tokens of its own threads
  auto copy_row = [&](int u, int b) {
    const float *urow = D + ((int64_t)(u / kTile) * nbr) * kCovTileElems + (u % kTile) * kTile;
    const void *ub = uniform_ptr(urow);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      dma4(__builtin_amdgcn_readfirstlane(lds_u32(&s_pre[b][e * NTH + wave * 64])), ub, (uint32_t)coff[e] * 4u);
  };
  auto prefetch = [&](int t) {
    const unsigned long long nk = s_next;
    const int u = (nk & ((1ull << 62) - 1ull)) != 0ull ? pick_of(nk) : -1;
    pre[t & 1] = u;
    if (u < 0) return;
    dma_t = t;
    copy_row(u, t & 1);
  };

  // t = 0: j_1 = argmax w (Eq. 9)
  float o[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) o[e] = dl[e] == -INFINITY ? -1.f : w[e];
  unsigned long long pk = exchange(o, 0);
  int j = pick_of(pk);
  if (sl == 0 && tid == 0 && !s_abort) {
    order[k0] = j;
    gains[k0] = gain_of(pk);
  }
  if (!s_abort) prefetch(0);
  for (int t = 1; t < K && !s_abort; ++t) {
    // fold the last pick's coverage row into the running minimum (Eq. 10).
    // The row always arrives through s_pre[t & 1]: copied at step t - 2 if the
    // pick was that step's runner-up, else now. (Loading it into registers
    // instead would leave the compiler, which does not see the copies, waiting
    // for every load in flight on either path.)
    if (pre[t & 1] != j) {
      copy_row(j, t & 1);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    } else if (dma_t == t - 1) {
      // the copy issued at step t - 1 (EPT loads a wave, the newest) may
      // still be in flight; the older one has landed once at most EPT remain
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(EPT) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) o[e] = s_pre[t & 1][e * NTH + tid];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      dl[e] = fminf(dl[e], o[e]);
      const float p = w[e] * dl[e];
      o[e] = dl[e] == -INFINITY ? -1.f : (p == p ? p : 0.f);   // Eq. 11
    }
    pk = exchange(o, t);
    // no slice had a candidate left (cannot happen for K_r <= N_r: coverage
    // distances off the diagonal are never -inf); every block of the request
    // sees the same key and stops
    if ((pk & ((1ull << 62) - 1ull)) == 0ull) break;
    j = pick_of(pk);
    if (sl == 0 && tid == 0 && !s_abort) {
      order[k0 + t] = j;
      gains[k0 + t] = gain_of(pk);
    }
    if (!s_abort && t + 1 < K) prefetch(t);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no LDS copy outlives the loop
  // this slice's picks: marked by their own rows, and the last pick
  bool sel[EPT];
  int cnt = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int i = base + tid + e * NTH;
    sel[e] = i < N && (dl[e] == -INFINITY || i == j);
    cnt += sel[e] ? 1 : 0;
  }
  for (int x = 1; x < 64; x <<= 1) cnt += __shfl_xor(cnt, x);
  if (lane == 0) s_cnt[wave] = cnt;
  __syncthreads();
  if (wave == 0 && !s_abort) {
    int tot = 0;
    for (int wv = 0; wv < kNW; ++wv) tot += s_cnt[wv];
    unsigned long long v;
    publish_wait(slot + 2 * kMcMaxS, (1ull << 62) | (unsigned)tot, 1u, v);
    int before = lane < sl ? (int)(v & 0xFFFFFFFFull) : 0;
    for (int x = 1; x < 64; x <<= 1) before += __shfl_xor(before, x);
    if (lane == 0) {
      s_cnt[8] = before;
      // a block of the request that timed out after publishing its count
      if (__hip_atomic_load(abort_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0ull) s_abort = 1;
    }
  }
  __syncthreads();
  if (s_abort) {
    for (int x = tid; x < K; x += NTH) {
      kept[k0 + x] = -1;
      order[k0 + x] = -1;
      gains[k0 + x] = __builtin_nanf("");
    }
    return;
  }
  const int before = s_cnt[8];
  __syncthreads();
  compact_ascending<EPT>([&](int e) { return sel[e]; }, kept + k0 + before, s_cnt, base);
}

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

  // validity and the take flags are recomputed or kept as bits: with 1024
  // threads and 32 keys a thread, a wave has no registers to spare
  unsigned key[EPT];
  auto valid = [&](int e) { return tid + e * nth < N; };
#pragma unroll
  for (int e = 0; e < EPT; ++e) key[e] = valid(e) ? __float_as_uint(clean_score(scores[n0 + tid + e * nth])) : 0u;
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
      if (valid(e) && (key[e] & mask) == prefix) atomicAdd(&hist[(key[e] >> shift) & 255u], 1);
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
  static_assert(EPT <= 32, "take flags are one 32-bit mask");
  uint32_t take = 0u;
  // rank the threshold-equal keys by index
  {
    const int lane = tid & 63, wave = tid >> 6, nw = nth >> 6;
    int base = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool eq = valid(e) && key[e] == thr;
      const unsigned long long m = __ballot(eq);
      if (lane == 0) s_cnt[wave] = __popcll(m);
      __syncthreads();
      int bw = 0, tot = 0;
      for (int w = 0; w < nw; ++w) {
        if (w < wave) bw += s_cnt[w];
        tot += s_cnt[w];
      }
      const int rank = base + bw + __popcll(m & ((1ull << lane) - 1ull));
      take |= (valid(e) && (key[e] > thr || (eq && rank < need)) ? 1u : 0u) << e;
      base += tot;
      __syncthreads();
    }
  }
  compact_ascending<EPT>([&](int e) { return ((take >> e) & 1u) != 0u; }, kept + k0, s_cnt);
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
      if (!((take >> e) & 1u)) continue;
      const unsigned long long mine = obj_key(__uint_as_float(key[e]), tid + e * nth);
      int c = 0;
      for (int x = 0; x < ns; ++x) c += s_keys[x] > mine ? 1 : 0;
      rank[e] += c;
    }
    __syncthreads();
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    if (!((take >> e) & 1u)) continue;
    if (order) order[k0 + rank[e]] = tid + e * nth;
    if (gains) gains[k0 + rank[e]] = __uint_as_float(key[e]);
  }
}


// Top-k (Table 5) for requests longer than one block's registers hold: one
// block per request radix-selects the K largest scores as k_topk does, reading
// the keys from memory on each of the four passes, then writes the kept tokens
// in ascending order in rounds of one token a thread (threshold ties ranked by
// index). The pick order is k_topk_rank's.
__global__ __launch_bounds__(1024) void k_topk_large(const float *__restrict__ scores,
                                                     const int32_t *__restrict__ cu_vis,
                                                     const int32_t *__restrict__ cu_keep,
                                                     int32_t *__restrict__ kept) {
  __shared__ int hist[256];
  __shared__ int s_cnt[2][16];
  __shared__ unsigned s_prefix;
  __shared__ int s_remaining;
  const int r = blockIdx.x;
  const int64_t n0 = cu_vis[r];
  const int N = cu_vis[r + 1] - (int)n0;
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const int tid = threadIdx.x, nth = blockDim.x, lane = tid & 63, wave = tid >> 6, nw = nth >> 6;
  auto key_at = [&](int i) { return __float_as_uint(clean_score(scores[n0 + i])); };
  if (tid == 0) {
    s_prefix = 0u;
    s_remaining = K;
  }
  unsigned mask = 0u;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += nth) hist[b] = 0;
    __syncthreads();
    const unsigned prefix = s_prefix;
    for (int i = tid; i < N; i += nth) {
      const unsigned k = key_at(i);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
    }
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
  const int need = s_remaining;   // threshold-equal keys to take, lowest index first
  // the rank of a flag among the round's earlier threads, and the round's total
  auto count = [&](bool f, int buf, int &before, int &total) {
    const unsigned long long m = __ballot(f);
    if (lane == 0) s_cnt[buf][wave] = __popcll(m);
    __syncthreads();
    before = __popcll(m & ((1ull << lane) - 1ull));
    total = 0;
    for (int w = 0; w < nw; ++w) {
      if (w < wave) before += s_cnt[buf][w];
      total += s_cnt[buf][w];
    }
  };
  int eq_seen = 0, out = 0;
  for (int c = 0; c < N; c += nth) {
    const int i = c + tid;
    const unsigned k = i < N ? key_at(i) : 0u;
    const bool eq = i < N && k == thr;
    int eb, et, tb, tt;
    count(eq, 0, eb, et);
    const bool take = i < N && (k > thr || (eq && eq_seen + eb < need));
    count(take, 1, tb, tt);
    if (take) kept[k0 + out + tb] = i;
    eq_seen += et;
    out += tt;
    __syncthreads();   // the counts are read before the next round rewrites them
  }
}

// The pick order of Top-k: kept token i of request blockIdx.y goes to position
// (number of kept tokens with a larger score, or an equal score and a lower
// index), i.e. decreasing score, ties by index. Block x ranks kept slots
// [1024 x, 1024 x + 1024) against all K_r, staged through LDS.
__global__ __launch_bounds__(1024) void k_topk_rank(const float *__restrict__ scores,
                                                    const int32_t *__restrict__ cu_vis,
                                                    const int32_t *__restrict__ cu_keep,
                                                    const int32_t *__restrict__ kept,
                                                    int32_t *__restrict__ order, float *__restrict__ gains) {
  constexpr int kStage = 4096;
  __shared__ unsigned long long s_keys[kStage];
  const int r = blockIdx.y;
  const int64_t n0 = cu_vis[r];
  const int64_t k0 = cu_keep[r];
  const int K = cu_keep[r + 1] - (int)k0;
  const int slot = (int)blockIdx.x * (int)blockDim.x + (int)threadIdx.x;
  if ((int)blockIdx.x * (int)blockDim.x >= K) return;   // block-uniform
  const int i = slot < K ? kept[k0 + slot] : 0;
  const float sc = clean_score(scores[n0 + i]);
  const unsigned long long mine = obj_key(sc, i);
  int rank = 0;
  for (int s0 = 0; s0 < K; s0 += kStage) {
    const int ns = min(kStage, K - s0);
    for (int x = threadIdx.x; x < ns; x += blockDim.x) {
      const int ix = kept[k0 + s0 + x];
      s_keys[x] = obj_key(clean_score(scores[n0 + ix]), ix);
    }
    __syncthreads();
    for (int x = 0; x < ns; ++x) rank += s_keys[x] > mine ? 1 : 0;
    __syncthreads();
  }
  if (slot < K) {
    order[k0 + rank] = i;
    gains[k0 + rank] = sc;
  }
}

}  // namespace

namespace last {

// Greedy block shape for `nreq` requests of up to n tokens each. Past
// kGreedyMaxN tokens, and past kMcMinN tokens when the requests' blocks fit in
// `budget` compute units, S <= 16 blocks of kMcThreads a request (slices of
// 2048 tokens, 4096 past 32768, 8192 past 65536) that exchange their
// candidates every step; else one block a request: one wave up to 1024 tokens
// (no block barrier per step), else 256, 512 or 1024 threads with up to 32
// tokens each.
constexpr int kMcMinN = 8192;
constexpr double kMcStepUs = 1.9;   // a step of the multi-block greedy (measured, 16k-32k tokens)
static void greedy_shape(int32_t n, int32_t nreq, int32_t budget, int32_t *threads, int32_t *ept,
                         int32_t *slices) {
  *slices = 0;
  if (n > kMcMinN) {
    const int e = n <= 32768 ? 8 : n <= 65536 ? 16 : 32;
    const int S = (n + kMcThreads * e - 1) / (kMcThreads * e);
    if (n > kGreedyMaxN || (int64_t)nreq * S <= budget) {
      *threads = kMcThreads;
      *ept = e;
      *slices = S;
      return;
    }
  }
  if (n <= 1024) {
    *threads = 64;
    const int e = (n + 63) / 64;
    *ept = e <= 2 ? 2 : e <= 4 ? 4 : e <= 6 ? 6 : e <= 8 ? 8 : e <= 10 ? e : e <= 12 ? 12 : e <= 14 ? 14 : 16;
  } else if (n <= 8192) {
    *threads = 256;
    const int e = (n + 255) / 256;
    *ept = e <= 8 ? 8 : e <= 16 ? 16 : 32;
  } else if (n <= 16384) {
    *threads = 512;   // 32 tokens a thread
    *ept = 32;
  } else {
    *threads = 1024;  // up to kGreedyMaxN tokens, 32 a thread
    *ept = 32;
  }
}

// The k-center's form: the matrix (gram.hip + the greedy here) or the rounds
// (rounds.hip). LAST_KCENTER_FORM=gram or =rounds, read at every call, forces
// one (rounds only where rounds_supported); by default the rounds take
// batches whose every request has kRoundAutoN tokens or more.
static bool want_rounds(int32_t N_min, int32_t N_max, int32_t Dv, last_dtype fdtype) {
  if (!rounds_supported(N_max, Dv, fdtype)) return false;
  if (const char *env = getenv("LAST_KCENTER_FORM")) {
    if (strcmp(env, "gram") == 0) return false;
    if (strcmp(env, "rounds") == 0) return true;
  }
  return N_min >= kRoundAutoN;
}

SelectPlan make_select_plan(int32_t R, const int32_t *cu_vis_h, const int32_t *cu_keep_h,
                            last_sel_mode mode, int32_t Dv, last_dtype fdtype, bool allow_groups,
                            bool allow_rounds) {
  SelectPlan p{};
  p.N_total = cu_vis_h[R];
  p.K_total = cu_keep_h[R];
  for (int r = 0; r < R; ++r) {
    const int64_t N = cu_vis_h[r + 1] - cu_vis_h[r];
    const int64_t K = cu_keep_h[r + 1] - cu_keep_h[r];
    p.N_max = std::max<int32_t>(p.N_max, (int32_t)N);
    p.K_max = std::max<int32_t>(p.K_max, (int32_t)K);
    const int64_t tb = (N + kTile - 1) / kTile;
    p.tiles_diag += tb;
    p.tiles_off += tb * (tb - 1) / 2;
    p.d_elems += cov_elems(N);
  }
  p.threads = p.N_max > 1024 ? 1024 : std::max(64, (p.N_max + 63) / 64 * 64);
  const int ept = (p.N_max + p.threads - 1) / p.threads;
  p.ept = ept <= 1 ? 1 : ept <= 2 ? 2 : ept <= 4 ? 4 : ept <= 8 ? 8 : ept <= 16 ? 16 : 32;
  greedy_shape(p.N_max, R, device_cus(), &p.g_threads, &p.g_ept, &p.g_slices);
  p.groups = 1;
  p.group_tile0[0] = 0;
  p.group_tile0[1] = p.tiles_off;
  p.group_rank0[0] = 0;
  p.group_rank0[1] = R;
  p.group_threads[0] = p.g_threads;
  p.group_ept[0] = p.g_ept;
  p.group_slices[0] = p.g_slices;
  int32_t N_min = p.N_max;
  for (int r = 0; r < R; ++r) N_min = std::min<int32_t>(N_min, cu_vis_h[r + 1] - cu_vis_h[r]);
  if (allow_rounds && mode == LAST_SEL_KCENTER && want_rounds(N_min, p.N_max, Dv, fdtype)) {
    p.rounds = true;
    for (int r = 0; r < R; ++r)
      p.round_Q += kRoundCandTasks + 2 + (cu_vis_h[r + 1] - cu_vis_h[r] + kRoundFoldRows - 1) / kRoundFoldRows;
    return p;
  }
  if (!allow_groups || mode != LAST_SEL_KCENTER || R < 2 || R > kRankMaxR) return p;

  // Ragged batches. A greedy takes about K_r (0.6 + 1.1e-4 N_r) microseconds
  // on one compute unit (one dependent step per pick, each a coverage row of
  // N_r floats), or K_r kMcStepUs on S of them (the multi-block greedy), about
  // 1.6 times that while the Gram loads the memory system (measured), and an off-diagonal Gram tile about 0.8 us per 64 columns of Dv
  // plus 3 us on one compute unit. When the longest greedy is several times the
  // median one, the requests are ordered by decreasing size and the
  // off-diagonal Gram runs in groups; each group's greedies start, on side
  // streams and on compute units the Gram leaves free, as soon as that group's
  // Gram is done. The grouping (2 to kMaxGroups groups, with geometric or even
  // tile shares) and the number of free compute units are chosen by simulating
  // that schedule with these costs.
  auto n_of = [&](int r) { return cu_vis_h[r + 1] - cu_vis_h[r]; };
  auto k_of = [&](int r) { return cu_keep_h[r + 1] - cu_keep_h[r]; };
  auto greedy_us = [&](int r) { return k_of(r) * (0.6 + 1.1e-4 * n_of(r)); };
  std::vector<int32_t> ord(R);
  std::vector<double> cost(R);
  for (int r = 0; r < R; ++r) {
    ord[r] = r;
    cost[r] = greedy_us(r);
  }
  std::vector<double> sorted_cost(cost);
  std::nth_element(sorted_cost.begin(), sorted_cost.begin() + R / 2, sorted_cost.end());
  const double median = sorted_cost[R / 2];
  const double longest = *std::max_element(cost.begin(), cost.end());
  if (!(longest >= 4.0 * median && longest >= 500.0) || p.tiles_off < 16 * 256) return p;
  // the same order as k_select_plan: decreasing size, ties by index
  std::sort(ord.begin(), ord.end(), [&](int a, int b) { return n_of(a) != n_of(b) ? n_of(a) > n_of(b) : a < b; });
  std::vector<int64_t> cum(R + 1, 0);   // off-diagonal tiles of the first k ranks
  for (int k = 0; k < R; ++k) {
    const int64_t nb = (n_of(ord[k]) + kTile - 1) / kTile;
    cum[k + 1] = cum[k] + nb * (nb - 1) / 2;
  }
  const int cus = device_cus();
  const double tile_us = 0.8 * (Dv > 0 ? Dv : 1024) / 64.0 + 3.0;
  struct Cand {
    int G;
    int32_t rank0[kMaxGroups + 1];
    int reserve;
    double span;
  };
  // group boundaries (ranks) for tile shares `frac` (cumulative, last 1)
  auto split = [&](const double *frac, int G, Cand &c) {
    c.G = 0;
    c.rank0[0] = 0;
    int k = 0;
    for (int g = 0; g < G - 1; ++g) {
      while (k < R - 1 && (double)cum[k + 1] < frac[g] * (double)cum[R]) ++k;
      const int b = std::max(k + 1, c.rank0[c.G] + 1);
      if (b >= R) break;
      c.rank0[++c.G] = b;
      k = b;
    }
    c.rank0[++c.G] = R;
  };
  // the schedule's length, and the free compute units its greedies need at once
  auto simulate = [&](Cand &c) {
    double best = 1e300;
    for (int reserve : {8, 16, 24, 32, 48, 64}) {
      const double rate = (cus - reserve) / tile_us;   // tiles per microsecond
      double t = 0, span = 0;
      std::vector<std::pair<double, double>> busy;      // greedy intervals
      std::vector<int> width;                           // compute units of each greedy
      double free_at[kSideStreams] = {};                // when each side stream's last greedies end
      for (int g = 0; g < c.G; ++g) {
        // the group's Gram, plus about one tile time for its launch's tail
        t += (double)(cum[c.rank0[g + 1]] - cum[c.rank0[g]]) / rate + tile_us;
        // a group whose blocks fit the reserve runs the multi-block greedy;
        // a group's greedies start after the previous ones on its stream
        int32_t th, ep, S;
        greedy_shape(n_of(ord[c.rank0[g]]), c.rank0[g + 1] - c.rank0[g], reserve, &th, &ep, &S);
        const double start = std::max(t, free_at[g % kSideStreams]);
        double end = start;
        for (int k = c.rank0[g]; k < c.rank0[g + 1]; ++k) {
          busy.push_back({start, start + 1.6 * (S > 0 ? k_of(ord[k]) * kMcStepUs : cost[ord[k]])});
          width.push_back(S > 0 ? S : 1);
          end = std::max(end, busy.back().second);
        }
        free_at[g % kSideStreams] = end;
      }
      const double gram_end = t;
      // concurrency before the Gram ends must fit the reserve; after it, every
      // unit is free (a sweep over the interval ends)
      std::vector<std::pair<double, int>> ev;
      ev.reserve(2 * busy.size());
      for (size_t i = 0; i < busy.size(); ++i) {
        ev.push_back({busy[i].first, +width[i]});
        ev.push_back({busy[i].second, -width[i]});
      }
      std::sort(ev.begin(), ev.end(), [](const std::pair<double, int> &a, const std::pair<double, int> &b) {
        return a.first != b.first ? a.first < b.first : a.second < b.second;   // ends before starts
      });
      int peak = 0, now = 0;
      for (auto &e : ev) {
        if (e.first >= gram_end) break;
        now += e.second;
        peak = std::max(peak, now);
      }
      for (auto &x : busy) span = std::max(span, x.second);
      span = std::max(span, gram_end);
      if (peak > reserve) span += (double)(peak - reserve) / reserve * longest;   // queued greedies
      if (span < best) {
        best = span;
        c.reserve = reserve;
      }
    }
    c.span = best;
  };
  Cand best{};
  best.span = 1e300;
  for (int G = 2; G <= std::min<int>(kMaxGroups, R); ++G) {
    for (int shape = 0; shape < 2; ++shape) {
      double frac[kMaxGroups];
      double tot = 0, x = 1;
      for (int g = 0; g < G; ++g) {
        tot += shape ? x : 1.0;
        frac[g] = tot;
        x *= 2;
      }
      for (int g = 0; g < G; ++g) frac[g] /= tot;
      Cand c{};
      split(frac, G, c);
      if (c.G < 2) continue;
      simulate(c);
      if (c.span < best.span) best = c;
    }
  }
  // the m longest requests alone first (their greedies, the longest, start
  // earliest), then the rest in groups of even tile shares
  for (int m : {1, 2, 4}) {
    if (m >= R) break;
    for (int G = 2; G <= std::min<int>(kMaxGroups, R - m + 1); ++G) {
      Cand c{};
      c.G = 1;
      c.rank0[0] = 0;
      c.rank0[1] = m;
      int k = m;
      for (int g = 1; g < G - 1; ++g) {   // group g ends at share g / (G - 1) of the rest
        while (k < R - 1 && (double)(cum[k + 1] - cum[m]) * (G - 1) < (double)g * (cum[R] - cum[m])) ++k;
        const int b = std::max(k, c.rank0[c.G] + 1);
        if (b >= R) break;
        c.rank0[++c.G] = b;
        k = b;
      }
      c.rank0[++c.G] = R;
      if (c.G < 2) continue;
      simulate(c);
      if (c.span < best.span) best = c;
    }
  }
  if (best.span >= 1e299) return p;
  p.groups = best.G;
  for (int g = 0; g <= p.groups; ++g) {
    p.group_rank0[g] = best.rank0[g];
    p.group_tile0[g] = cum[best.rank0[g]];
  }
  p.ranked = true;
  p.reserve = best.reserve;
  // a group's greedies run beside the later groups' Gram, on the compute units
  // it leaves free
  for (int x = 0; x < p.groups; ++x)
    greedy_shape(n_of(ord[p.group_rank0[x]]), p.group_rank0[x + 1] - p.group_rank0[x], p.reserve,
                 &p.group_threads[x], &p.group_ept[x], &p.group_slices[x]);
  return p;
}

SelectWs carve_select_ws(void *ws, int32_t R, const SelectPlan &p, last_sel_mode mode,
                         size_t *bytes) {
  Carver cv(ws);
  SelectWs w{};
  if (mode == LAST_SEL_KCENTER && p.rounds) {
    w.nn = cv.take<double>(p.N_total + kTile);
    w.inv = cv.take<double>(p.N_total + kTile);
    w.r_dl = cv.take<float>(p.N_total);
    w.r_cand = cv.take<int32_t>((int64_t)R * kRoundCands);
    w.r_picks = cv.take<int32_t>((int64_t)R * kRoundPicks);
    w.r_cmat = cv.take<float>((int64_t)R * kRoundCands * kRoundCands);
    w.r_st = cv.take<int32_t>((int64_t)R * 4);
    w.r_T = cv.take<unsigned long long>(R);
    w.r_dcnt = cv.take<uint32_t>(R);
    w.r_qoff = cv.take<int64_t>(R + 1);
    w.r_ctl = cv.take<unsigned long long>(2);
  } else if (mode == LAST_SEL_KCENTER) {
    w.dtile_off = cv.take<int32_t>(R + 1);
    w.otile_off = cv.take<int32_t>(R + 1);
    w.dtile = cv.take<TileMeta>(p.tiles_diag);
    w.otile = cv.take<TileMeta>(p.tiles_off);
    w.d_off = cv.take<int64_t>(R + 1);
    w.nn = cv.take<double>(p.N_total + kTile);
    w.inv = cv.take<double>(p.N_total + kTile);
    w.dmat = cv.take<float>(p.d_elems);
    w.req_order = cv.take<int32_t>(R);
    w.mc_slots = cv.take<unsigned long long>((int64_t)R * kMcSlotWords);
  }
  *bytes = cv.size();
  return w;
}

// beside_gram: a launch on a side stream, overlapping the Gram (timed as
// "greedy_side"; a multi-block greedy then spreads its blocks over the XCDs).
static hipError_t launch_greedy(int32_t threads, int32_t ept, int32_t slices, int32_t blocks,
                                const int32_t *req_order, int32_t rank0, const SelectWs &w, const float *scores,
                                const int32_t *cu_vis, const int32_t *cu_keep, int32_t *kept, int32_t *order,
                                float *gains, hipStream_t s, bool beside_gram = false);
static hipError_t launch_pipelined(int32_t R, int32_t Dv, const SelectPlan &p, const SelectWs &w,
                                   const float *scores, const void *feats, const int32_t *cu_vis,
                                   const int32_t *cu_keep, int32_t *kept, int32_t *order, float *gains,
                                   hipStream_t s);

hipError_t launch_select(int32_t R, int32_t Dv, last_dtype fdtype, last_sel_mode mode,
                         const SelectPlan &p, const SelectWs &w, const float *scores,
                         const void *feats, const int32_t *cu_vis, const int32_t *cu_keep,
                         int32_t *kept, int32_t *order, float *gains, hipStream_t s) {
  if (mode == LAST_SEL_KCENTER && p.rounds) {
    const hipError_t e = launch_round_norms(Dv, p, w, feats, s);
    if (e != hipSuccess) return e;
    return launch_round_pick(R, Dv, p, w, scores, feats, cu_vis, cu_keep, kept, order, gains, s);
  }
  if (mode == LAST_SEL_KCENTER && p.groups > 1 && gram_streamed(fdtype, Dv))
    return launch_pipelined(R, Dv, p, w, scores, feats, cu_vis, cu_keep, kept, order, gains, s);
  if (mode == LAST_SEL_KCENTER) {
    const hipError_t e = launch_similarity(R, Dv, fdtype, p, w, feats, cu_vis, s);
    if (e != hipSuccess) return e;
  }
  return launch_pick(R, mode, p, w, scores, cu_vis, cu_keep, kept, order, gains, s);
}

hipError_t launch_pick(int32_t R, last_sel_mode mode, const SelectPlan &p, const SelectWs &w,
                       const float *scores, const int32_t *cu_vis, const int32_t *cu_keep,
                       int32_t *kept, int32_t *order, float *gains, hipStream_t s) {
  if (mode == LAST_SEL_TOPK && p.N_max > kGreedyMaxN) {
    launch_begin("topk", s);
    hipLaunchKernelGGL(k_topk_large, dim3(R), dim3(1024), 0, s, scores, cu_vis, cu_keep, kept);
    hipLaunchKernelGGL(k_topk_rank, dim3((p.K_max + 1023) / 1024, R), dim3(1024), 0, s, scores, cu_vis, cu_keep, kept,
                       order, gains);
    return launch_end(s);
  }
  if (mode == LAST_SEL_TOPK) {
    launch_begin("topk", s);
#define LAST_TOPK(E) \
  hipLaunchKernelGGL(k_topk<E>, dim3(R), dim3(p.threads), 0, s, scores, cu_vis, cu_keep, kept, order, gains)
    switch (p.ept) {
      case 1: LAST_TOPK(1); break;
      case 2: LAST_TOPK(2); break;
      case 4: LAST_TOPK(4); break;
      case 8: LAST_TOPK(8); break;
      case 16: LAST_TOPK(16); break;
      default: LAST_TOPK(32); break;
    }
#undef LAST_TOPK
    return launch_end(s);
  }

  return launch_greedy(p.g_threads, p.g_ept, p.g_slices, R, nullptr, 0, w, scores, cu_vis, cu_keep, kept, order,
                       gains, s);
}

// The blocks of k_greedy_mc<EPT> the current device holds at once.
template <int EPT>
static int mc_capacity() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_greedy_mc<EPT>, kMcThreads, 0) != hipSuccess ||
      per_cu <= 0)
    return 0;
  v = per_cu * device_cus();
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// The multi-block greedy over `nreq` requests (ranks rank0 .. rank0 + nreq - 1),
// in launches of at most as many blocks as the device holds at once, each after
// zeroing its ranks' exchange words (a kernel, not a memset, so that a caller
// may capture the sequence in a graph). A wait may last 10 s.
template <int EPT>
static hipError_t launch_mc(int32_t slices, int32_t nreq, const int32_t *req_order, int32_t rank0,
                            const SelectWs &w, const float *scores, const int32_t *cu_vis, const int32_t *cu_keep,
                            int32_t *kept, int32_t *order, float *gains, bool spread, hipStream_t s) {
  // A launch takes at most a quarter of what the device holds, so that as many
  // such launches as the device has hardware queues (4) fit beside each other:
  // a request's blocks never wait on blocks of another launch that in turn
  // wait for room.
  const int cap = mc_capacity<EPT>() / 4;
  if (cap < slices) return hipErrorInvalidConfiguration;
  const int per_launch = cap / slices;
  // 10 s in wall-clock ticks; LAST_MC_WAIT_US overrides it (tests force the
  // timeout path with a tiny value)
  int64_t wait_us = 10000000;
  if (const char *env = getenv("LAST_MC_WAIT_US")) wait_us = std::max<int64_t>(0, atoll(env));
  const int64_t limit = device_wall_khz() * wait_us / 1000;
  for (int32_t c = 0; c < nreq; c += per_launch) {
    const int32_t n = std::min<int32_t>(per_launch, nreq - c);
    unsigned long long *slots = w.mc_slots + (int64_t)(rank0 + c) * kMcSlotWords;
    const int64_t words = (int64_t)n * kMcSlotWords;
    hipLaunchKernelGGL(k_zero_u64, dim3((unsigned)std::min<int64_t>((words + 255) / 256, 1024)), dim3(256), 0, s,
                       slots, words);
    const unsigned grid = spread ? (unsigned)(n * slices) : (unsigned)(8 * slices * ((n + 7) / 8));
    hipLaunchKernelGGL(k_greedy_mc<EPT>, dim3(grid), dim3(kMcThreads), 0, s, scores, w.dmat, w.d_off, cu_vis,
                       cu_keep, req_order, rank0 + c, n, slices, spread ? 1 : 0, w.mc_slots, limit, kept, order,
                       gains);
  }
  return hipGetLastError();
}

// One greedy launch: `blocks` requests (ranks rank0 .. rank0 + blocks - 1 of
// req_order, or requests rank0 .. rank0 + blocks - 1 when req_order is null;
// the one-block greedy takes rank0 = 0 there).
static hipError_t launch_greedy(int32_t threads, int32_t ept, int32_t slices, int32_t blocks,
                                const int32_t *req_order, int32_t rank0, const SelectWs &w, const float *scores,
                                const int32_t *cu_vis, const int32_t *cu_keep, int32_t *kept, int32_t *order,
                                float *gains, hipStream_t s, bool beside_gram) {
  const char *what = beside_gram ? "greedy_side" : "greedy";
  launch_begin(what, s);
  if (slices > 0) {
    // beside the Gram (the side launches) a request's blocks spread over the XCDs
    const bool spread = beside_gram;
    const hipError_t e =
        ept == 8    ? launch_mc<8>(slices, blocks, req_order, rank0, w, scores, cu_vis, cu_keep, kept, order, gains,
                                   spread, s)
        : ept == 16 ? launch_mc<16>(slices, blocks, req_order, rank0, w, scores, cu_vis, cu_keep, kept, order, gains,
                                    spread, s)
                    : launch_mc<32>(slices, blocks, req_order, rank0, w, scores, cu_vis, cu_keep, kept, order, gains,
                                    spread, s);
    const hipError_t e2 = launch_end(s);
    return e != hipSuccess ? e : e2;
  }
#define LAST_GREEDY(E, T)                                                                          \
  hipLaunchKernelGGL((k_greedy<E, T>), dim3(blocks), dim3(T), 0, s, scores, w.dmat, w.d_off, cu_vis, cu_keep, \
                     req_order, rank0, kept, order, gains)
  if (threads == 64) {
    switch (ept) {
      case 2: LAST_GREEDY(2, 64); break;
      case 4: LAST_GREEDY(4, 64); break;
      case 6: LAST_GREEDY(6, 64); break;
      case 8: LAST_GREEDY(8, 64); break;
      case 9: LAST_GREEDY(9, 64); break;
      case 10: LAST_GREEDY(10, 64); break;
      case 12: LAST_GREEDY(12, 64); break;
      case 14: LAST_GREEDY(14, 64); break;
      default: LAST_GREEDY(16, 64); break;
    }
  } else if (threads == 256) {
    switch (ept) {
      case 8: LAST_GREEDY(8, 256); break;
      case 16: LAST_GREEDY(16, 256); break;
      default: LAST_GREEDY(32, 256); break;
    }
  } else if (threads == 512) {
    LAST_GREEDY(32, 512);
  } else {
    LAST_GREEDY(32, 1024);
  }
#undef LAST_GREEDY
  return launch_end(s);
}

// Library-owned streams per host thread and device, one per group, for the
// greedies that run beside the Gram of a ragged batch, with their events
// (reused call after call: a wait takes the event's latest record at the time
// it is enqueued). Created on first use, default priority, kept until the
// process ends.
namespace {
struct SideStream {
  hipStream_t s[kSideStreams] = {};      // group g's greedies run on s[g % kSideStreams]
  hipEvent_t gram[kSideStreams] = {};    // a group's Gram done (recorded on the caller's stream)
  hipEvent_t done[kSideStreams] = {};    // the stream's greedies done
  bool ok = false;
};
constexpr int kSideDevices = 64;
thread_local SideStream t_side[kSideDevices];

SideStream *side_stream() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kSideDevices) return nullptr;
  SideStream &x = t_side[dev];
  if (!x.ok) {
    for (int g = 0; g < kSideStreams; ++g) {
      if (!x.s[g] && hipStreamCreateWithFlags(&x.s[g], hipStreamNonBlocking) != hipSuccess) return nullptr;
      if (!x.gram[g] && hipEventCreateWithFlags(&x.gram[g], hipEventDisableTiming) != hipSuccess) return nullptr;
      if (!x.done[g] && hipEventCreateWithFlags(&x.done[g], hipEventDisableTiming) != hipSuccess) return nullptr;
    }
    x.ok = true;
  }
  return &x;
}
}  // namespace

// Ragged k-center: the plan (off-diagonal tiles in rank order) and every
// diagonal tile, then the off-diagonal Gram group by group on `s`, each group's
// greedies on its own side stream once that group's Gram is done, beside the
// next groups' Gram. The Gram's persistent grid leaves p.reserve compute units
// free for them. `s` waits for every side stream at the end.
static hipError_t launch_pipelined(int32_t R, int32_t Dv, const SelectPlan &p, const SelectWs &w,
                                   const float *scores, const void *feats, const int32_t *cu_vis,
                                   const int32_t *cu_keep, int32_t *kept, int32_t *order, float *gains,
                                   hipStream_t s) {
  SideStream *side = side_stream();
  if (!side) {   // no side stream: the whole Gram, then every greedy, on `s`
    SelectPlan q = p;
    q.groups = 1;
    hipError_t e = launch_similarity(R, Dv, LAST_BF16, q, w, feats, cu_vis, s);
    if (e != hipSuccess) return e;
    return launch_greedy(p.g_threads, p.g_ept, p.g_slices, R, p.ranked ? w.req_order : nullptr, 0, w, scores,
                         cu_vis, cu_keep,
                         kept, order, gains, s);
  }
  hipError_t e;
  if ((e = launch_gram_plan(R, p, w, cu_vis, s)) != hipSuccess) return e;
  const int cus = device_cus();
  if ((e = launch_gram_diag(Dv, p, w, feats, cus, s)) != hipSuccess) return e;
  const int gram_cus = std::max(8, cus - p.reserve);
  for (int g = 0; g < p.groups; ++g) {
    const int64_t t0 = p.group_tile0[g], nt = p.group_tile0[g + 1] - t0;
    const int q = g % kSideStreams;
    if ((e = launch_gram_off(Dv, p, w, feats, t0, nt, gram_cus, s)) != hipSuccess) return e;
    // (each wait is enqueued right after its record, so one event per side
    // stream serves every group)
    if ((e = hipEventRecord(side->gram[q], s)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(side->s[q], side->gram[q], 0)) != hipSuccess) return e;
    const int32_t r0 = p.group_rank0[g], nr = p.group_rank0[g + 1] - r0;
    e = launch_greedy(p.group_threads[g], p.group_ept[g], p.group_slices[g], nr, w.req_order, r0, w, scores,
                      cu_vis, cu_keep, kept, order, gains, side->s[q], true);
    if (e != hipSuccess) return e;
  }
  for (int q = 0; q < std::min(p.groups, kSideStreams); ++q) {
    if ((e = hipEventRecord(side->done[q], side->s[q])) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(s, side->done[q], 0)) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace last
