// Internal declarations of liblast: device helpers, launch bookkeeping and
// the kernel launchers each source file provides to the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "last.h"

namespace last {

// ----------------------------------------------------------------- host side

// Every launch goes through launch_begin / launch_end so that optional
// per-kernel event timing can bracket it; launch_end also checks the launch.
void launch_begin(const char *name, hipStream_t s);
hipError_t launch_end(hipStream_t s);

// Remember the last HIP error text for last_status_string (thread-local).
void note_hip_error(hipError_t e);

// Compute units of the current device (cached per device).
int device_cus();
// Ticks per millisecond of the current device's wall_clock64 (cached per device).
int64_t device_wall_khz();

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace carving: consecutive 256-byte aligned segments.
struct Carver {
  char *base;
  size_t off = 0;
  explicit Carver(void *b) : base(static_cast<char *>(b)) {}
  template <typename T>
  T *take(size_t count) {
    off = align_up(off, 256);
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t size() const { return align_up(off, 256); }
};

// ------------------------------------------------------------ score pass
struct ScorePlan {
  bool stream;            // contiguous all-heads kernel (Hkv divides 32, Hq/Hkv <= 8)
  int32_t chunk_tokens;   // tokens per work chunk
  int32_t head_groups;    // query-head groups per KV head (g split in <= 8)
  int32_t g_max;          // heads per group template: 1, 2, 4 or 8
  int64_t C_total;        // chunks over all requests
  int64_t S_total;        // finalize slices over all requests
  int32_t slice_tokens;   // visual tokens per finalize block
  int64_t T_total, N_total;
};

struct ScoreWs {
  int32_t *chunk_off, *slice_off;  // [R + 1] count prefixes (written only for large batches)
  float4 *stats;  // [G][Hq][C_total] (chunk max, sum exp, visual sum exp, 0)
  float *vlog;    // [G][N_total][Hq] scaled logits of visual columns, layer-major
  float2 *rowstat;  // [R][G * Hq] merged (max, 1 / sum exp) of every row
  float *rowmass;   // [R][G * Hq] each row's visual mass V / Z (S sums them)
};

// row_pos (nullable, one entry per request): score the causal row at that
// position instead of the last token's; the row sees keys 0 .. row_pos[r].
ScorePlan make_score_plan(const last_batch *b, const int32_t *row_pos_h = nullptr);
ScoreWs carve_score_ws(void *ws, const last_batch *b, const ScorePlan &p, size_t *bytes);
hipError_t launch_scores(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                         const void *q, const void *k, const int32_t *row_pos, float *scores,
                         float *attn_rows, float scale, hipStream_t s);
// The count prefixes (run only for batches too large for the blocks' own scan,
// or when `always`), and merge + finalize alone (for scores whose chunk
// statistics and visual logits another kernel wrote).
hipError_t launch_score_plan(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                             const int32_t *row_pos, hipStream_t s, bool always = false);
hipError_t launch_score_tail(const last_batch *b, const ScorePlan &p, const ScoreWs &w,
                             const int32_t *row_pos, float *scores, hipStream_t s);

// ------------------------------------------------ prefill attention
// Query blocks of 128 positions over all requests.
int64_t prefill_query_blocks(const last_batch *b);
// Causal attention of every position (bf16), and the last row's score-pass
// statistics as one chunk per request (stats[(l * Hq + h) * R + r], vlog).
hipError_t launch_prefill(const last_batch *b, int64_t QB_total, int32_t *qb_off, int32_t *qb_req,
                          const void *q, const void *k, const void *v, void *out, float *vlog,
                          float4 *stats, float scale, hipStream_t s);

// ------------------------------------------------ several rows per request
// Query rows are taken 32 at a time (one matrix-core tile). A block of
// kRowWaves waves takes RT such row tiles (a row group) and splits each stage
// of keys among the kRowWaves / RT waves that share a row tile; RT is 4, 2 or
// 1, from the largest request's tile count. Keys go in chunks of kRowChunk.
constexpr int kRowWaves = 4;
constexpr int kRowChunk = 1024;

struct RowsPlan {
  int64_t M_total, N_total, T_total;
  int64_t items1, items2;   // (request, row group, key chunk) and (.., visual chunk) work items
  int64_t SC_total;         // per layer: sum_r Hq * M_r * key chunks_r row statistics
  int32_t RG_max;           // most row groups of any request
  int32_t RT;               // row tiles per block
  int32_t MB;               // merge blocks per request (256 rows each, for the largest request)
};

struct RowsWs {
  int32_t *off1, *off2;     // [R+1] item prefixes per request
  int64_t *sc_off;          // [R+1] statistics prefixes per request
  int4 *rinfo;              // [R] (key chunks, visual chunks, row groups, last row position)
  int4 *items1, *items2;    // (request, row group, chunk, 0)
  float4 *stats;            // [G][SC_total] (max, sum exp, visual sum exp, 0) per row and chunk
  float2 *rowstat;          // [G][Hq][M_total] (max, 1 / sum exp) per row
  float *mass;              // [R] sum over rows of visual mass V / Z
  float *mass_part;         // [R][MB] the merge blocks' shares of it
  float *part;              // [G][Hkv][RG_max][N_total] visual probability sums per row group
};

RowsPlan make_rows_plan(const last_batch *b, const int32_t *cu_rows_h, const int32_t *row_pos_h);
RowsWs carve_rows_ws(void *ws, const last_batch *b, const RowsPlan &p, size_t *bytes);
hipError_t launch_rows(const last_batch *b, const RowsPlan &p, const RowsWs &w,
                       const int32_t *cu_rows, const int32_t *row_pos, const void *q,
                       const void *k, float *scores, float scale, hipStream_t s);

// ------------------------------------------------------------ selection
constexpr int kGramTile = 128;       // Gram tile edge (rows of X per side)
constexpr int kSelMaxN = 131072;     // largest request diverse_select takes
constexpr int kGreedyMaxN = 32768;   // largest request one block's registers hold (k_greedy, k_topk)
constexpr int kMcSlotWords = 256;    // exchange words per request of the multi-block greedy

// The k-center in rounds (rounds.hip), without the N x N matrix: candidates
// a round, picks a round, tokens a fold task, and the largest Dv and N_r it
// takes (its candidate-Gram chunks and select keys live in LDS).
constexpr int kRoundCands = 192;
constexpr int kRoundPicks = 64;
constexpr int kRoundPairs = (kRoundCands / 32) * (kRoundCands / 32 + 1) / 2;   // 32 x 32 block pairs of the candidate Gram
constexpr int kRoundCandTasks = kRoundPairs;                                      // one block pair a task
constexpr int kRoundFoldRows = 256;
constexpr int kRoundMaxDv = 4096;
constexpr int kRoundMaxN = 32768;
// diverse_select takes the rounds by default when every request has at least
// this many tokens (measured: the matrix form is faster on batches with
// shorter requests)
constexpr int kRoundAutoN = 8192;

// A request's coverage matrix is stored as nb x nb tiles of 128 x 128 floats
// (nb = ceil(N_r / 128)), tile (I, J) at element (I * nb + J) * 128 * 128 and
// row-major inside. A Gram tile then writes two contiguous 64 KB blocks (its
// own and the mirror), and the greedy reads row j as nb pieces of 512 bytes.
// Entries past N_r in the last row or column block are padding, never read.
constexpr int64_t kCovTileElems = (int64_t)kGramTile * kGramTile;
__host__ __device__ inline int64_t cov_blocks(int64_t n) { return (n + kGramTile - 1) / kGramTile; }
__host__ __device__ inline int64_t cov_elems(int64_t n) { return cov_blocks(n) * cov_blocks(n) * kCovTileElems; }
// element (i, j) of a matrix with nb row blocks
__host__ __device__ inline int64_t cov_index(int64_t i, int64_t j, int64_t nb) {
  return ((i / kGramTile) * nb + j / kGramTile) * kCovTileElems + (i % kGramTile) * kGramTile + j % kGramTile;
}

// One Gram tile: the request's first feature row, N_r, the row blocks
// I << 16 | J, the request, and the element offset of its coverage matrix.
struct alignas(16) TileMeta {
  int32_t n0, n, ij, r;
  int64_t doff, pad;
};
static_assert(sizeof(TileMeta) == 32, "two 16-byte pieces");

// Ragged batches: the requests in decreasing size (their ranks) are split into
// at most kMaxGroups groups. The off-diagonal Gram runs group by group, and a
// group's greedy runs on a side stream beside the Gram of the later groups,
// group g on side stream g mod kSideStreams. Three side streams: with the
// caller's stream they use four hardware queues, the default number per
// process; more streams would share queues and serialise.
constexpr int kMaxGroups = 3;
constexpr int kSideStreams = 3;
constexpr int kRankMaxR = 1024;   // larger batches keep the natural order, one group
struct SelectPlan {
  int64_t N_total, K_total;
  int32_t N_max, K_max;
  int64_t tiles_diag;      // diagonal Gram tiles over all requests
  int64_t tiles_off;       // Gram tiles strictly above the diagonal
  int64_t d_elems;         // sum of cov_elems(N_r) (coverage matrices)
  int32_t threads, ept;    // top-k block shape
  int32_t g_threads, g_ept;  // greedy block shape
  int32_t g_slices;        // > 0: blocks per request of the multi-block greedy (then g_ept is its EPT)
  int32_t groups;          // 1: the whole Gram, then every greedy
  bool ranked;             // off-diagonal tiles listed in rank order (groups > 1)
  int32_t reserve;         // compute units the Gram leaves to concurrent greedies
  int64_t group_tile0[kMaxGroups + 1];  // off-diagonal tile range of each group
  int32_t group_rank0[kMaxGroups + 1];  // rank range of each group
  int32_t group_threads[kMaxGroups], group_ept[kMaxGroups];  // greedy shape per group
  int32_t group_slices[kMaxGroups];
  bool rounds;             // the k-center in rounds (rounds.hip) instead of the matrix
  int64_t round_Q;         // tasks a round of the rounds kernel
};

struct SelectWs {
  int32_t *dtile_off, *otile_off;  // [R+1] diagonal / off-diagonal tile prefixes per request
  TileMeta *dtile, *otile;         // every diagonal / off-diagonal tile
  int64_t *d_off;                  // [R+1] element offsets of each request's coverage matrix
  double *nn, *inv;                // [N_total + 128] squared feature norms and 1 / norm
                                   // (the tail lets a tile read 128 entries from any row)
  float *dmat;                     // coverage distances, tile-major per request (cov_index)
  int32_t *req_order;              // [R] the request of each rank (ranked plans)
  unsigned long long *mc_slots;    // [R][kMcSlotWords] exchange words of the multi-block greedy, by rank
  // the rounds form (nn and inv as above; nothing else of the matrix form)
  float *r_dl;                     // [N_total] running minimum coverage distance
  int32_t *r_cand, *r_picks;       // [R][kRoundCands], [R][kRoundPicks]
  float *r_cmat;                   // [R][kRoundCands][kRoundCands] candidate distances
  int32_t *r_st;                   // [R][4] request state
  unsigned long long *r_T;         // [R] bound keys
  uint32_t *r_dcnt;                // [R] completed tasks
  int64_t *r_qoff;                 // [R + 1] fold-tile prefixes
  unsigned long long *r_ctl;       // [2] next task, live requests and the abort word
};

// allow_groups: a single diverse_select call may pipeline a ragged batch (the
// two-call form keeps one group, so both of its calls see the same plan); Dv
// enters that schedule's cost model. allow_rounds: the k-center may run in
// rounds (single calls only: the pick call of the two-call form has no
// features); whether it does depends on the shapes and LAST_KCENTER_FORM.
SelectPlan make_select_plan(int32_t R, const int32_t *cu_vis_h, const int32_t *cu_keep_h,
                            last_sel_mode mode, int32_t Dv, last_dtype fdtype, bool allow_groups,
                            bool allow_rounds);
// The rounds form: the shapes it takes, the norms (the first half, features
// only), and the rounds themselves.
bool rounds_supported(int32_t N_max, int32_t Dv, last_dtype fdtype);
hipError_t launch_round_norms(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats,
                              hipStream_t s);
hipError_t launch_round_pick(int32_t R, int32_t Dv, const SelectPlan &p, const SelectWs &w, const float *scores,
                             const void *feats, const int32_t *cu_vis, const int32_t *cu_keep, int32_t *kept,
                             int32_t *order, float *gains, hipStream_t s);
SelectWs carve_select_ws(void *ws, int32_t R, const SelectPlan &p, last_sel_mode mode,
                         size_t *bytes);
hipError_t launch_select(int32_t R, int32_t Dv, last_dtype fdtype, last_sel_mode mode,
                         const SelectPlan &p, const SelectWs &w, const float *scores,
                         const void *feats, const int32_t *cu_vis, const int32_t *cu_keep,
                         int32_t *kept, int32_t *order, float *gains, hipStream_t s);
// The two halves of launch_select for k-center: the plan and the coverage
// matrices (features only), then the greedy (or Top-k, which needs no first
// half) on what the first half left in the workspace.
hipError_t launch_similarity(int32_t R, int32_t Dv, last_dtype fdtype, const SelectPlan &p,
                             const SelectWs &w, const void *feats, const int32_t *cu_vis,
                             hipStream_t s);
// The pieces of launch_similarity for the bf16 matrix-core path (gram.hip):
// the plan, every diagonal tile (with the norms), and off-diagonal tiles
// [t0, t0 + nt) of the list on a persistent grid for `cus` compute units.
bool gram_streamed(last_dtype fdtype, int32_t Dv);
hipError_t launch_gram_plan(int32_t R, const SelectPlan &p, const SelectWs &w, const int32_t *cu_vis,
                            hipStream_t s);
hipError_t launch_gram_diag(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats, int cus,
                            hipStream_t s);
hipError_t launch_gram_off(int32_t Dv, const SelectPlan &p, const SelectWs &w, const void *feats, int64_t t0,
                           int64_t nt, int cus, hipStream_t s);
hipError_t launch_pick(int32_t R, last_sel_mode mode, const SelectPlan &p, const SelectWs &w,
                       const float *scores, const int32_t *cu_vis, const int32_t *cu_keep,
                       int32_t *kept, int32_t *order, float *gains, hipStream_t s);

// ------------------------------------------------------------ gather
hipError_t launch_gather(int32_t R, int64_t row_bytes, int64_t K_total, int64_t N_total,
                         const void *feats, const int32_t *cu_vis, const int32_t *kept,
                         const int32_t *cu_keep, void *out, hipStream_t s);

// ------------------------------------------------------------ connector
// Dims the connector kernels take: Dv, Dh multiples of the 64-column stage,
// Do of the 4-feature store, and a product grid that fits one launch.
bool connector_shape_ok(int64_t K, int32_t Dv, int32_t Dh, int32_t Do);
hipError_t launch_connector(int64_t K, int32_t Dv, int32_t Dh, int32_t Do, float eps, const void *x,
                            const float *gamma, const float *beta, const void *w1, const float *b1,
                            const void *w2, const float *b2, void *out, void *xn, void *hid,
                            hipStream_t s);

}  // namespace last

// ----------------------------------------------------------------- device side
namespace last_dev {

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// DPP lane permutations within rows of 16 lanes.
__device__ __forceinline__ float dpp_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_half_mirror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
}
// Sum over each aligned group of 8 lanes; every lane of the group gets the total.
__device__ __forceinline__ float sum8(float v) {
  v += dpp_xor1(v);
  v += dpp_xor2(v);
  v += dpp_half_mirror(v);
  return v;
}

// Wave-wide max / sum, returned wave-uniform: DPP inside each row of 16
// lanes, then the four row results in a fixed order (deterministic). Every
// lane of the wave must be active.
__device__ __forceinline__ float dpp_mirror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
}
__device__ __forceinline__ float row_lane15(float v, int row) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16 * row + 15));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_xor1(v));
  v = fmaxf(v, dpp_xor2(v));
  v = fmaxf(v, dpp_half_mirror(v));
  v = fmaxf(v, dpp_mirror(v));
  return fmaxf(fmaxf(row_lane15(v, 0), row_lane15(v, 1)), fmaxf(row_lane15(v, 2), row_lane15(v, 3)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_xor1(v);
  v += dpp_xor2(v);
  v += dpp_half_mirror(v);
  v += dpp_mirror(v);
  return (row_lane15(v, 0) + row_lane15(v, 1)) + (row_lane15(v, 2) + row_lane15(v, 3));
}
// Wave-wide maximum of the 64-bit key (hi << 32) | lo, returned
// wave-uniform, in two 32-bit passes: the maximum hi by DPP exchanges inside
// each row of 16 lanes (xor 1, xor 2, half-mirror, mirror) and a readlane of
// the four rows; then the lo of the lanes holding that hi. A single such lane
// (the usual case) gives its lo directly; ties take a second pass over lo.
// Every lane of the wave must be active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp_u32<0xB1>(v));
  v = max(v, dpp_u32<0x4E>(v));
  v = max(v, dpp_u32<0x141>(v));
  v = max(v, dpp_u32<0x140>(v));
  const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane(v, 15), (uint32_t)__builtin_amdgcn_readlane(v, 31));
  const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane(v, 47), (uint32_t)__builtin_amdgcn_readlane(v, 63));
  return max(a, b);
}
__device__ __forceinline__ unsigned long long wave_max_key(uint32_t hi, uint32_t lo) {
  const uint32_t mh = wave_max_u32(hi);
  const unsigned long long tied = __ballot(hi == mh);
  uint32_t ml;
  if (__popcll(tied) == 1)
    ml = (uint32_t)__builtin_amdgcn_readlane(lo, (int)__ffsll((long long)tied) - 1);
  else
    ml = wave_max_u32(hi == mh ? lo : 0u);
  return ((unsigned long long)mh << 32) | ml;
}

// LDS byte address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_u32(const void *p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) void *)p);
}

// global_load_lds_dwordx4: lane i's 16 bytes at base + voff land in LDS at
// lds + 16 i. lds: wave-uniform LDS byte address (goes to M0); base:
// wave-uniform global address; voff: this lane's byte offset from base. The
// load is issued from inline assembly so that the compiler does not order LDS
// reads behind it; the caller waits for it (vm_wait) before publishing the
// LDS it wrote.
__device__ __forceinline__ void dma16(uint32_t lds, const void *base, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(base) : "memory");
}
// global_load_lds_dword: lane i's 4 bytes at base + voff land in LDS at
// lds + 4 i (same conventions as dma16).
__device__ __forceinline__ void dma4(uint32_t lds, const void *base, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(voff), "s"(base) : "memory");
}
// The same with the non-temporal hint: for data read exactly once, which
// then streams past the caches instead of displacing lines others reuse.
__device__ __forceinline__ void dma16_nt(uint32_t lds, const void *base, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(lds), "v"(voff), "s"(base) : "memory");
}
__device__ __forceinline__ const void *uniform_ptr(const void *p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void *)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ int64_t uniform_i64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
// Blocks are dealt to the 8 XCDs in turn (block b to XCD b % 8). This maps
// block b to a logical index so that each XCD runs one contiguous range of
// the grid (the last gridDim % 8 blocks keep their own index): neighbouring
// logical blocks, which read the same data, then share that XCD's L2.
__device__ __forceinline__ int64_t xcd_contiguous(int64_t b, int64_t nblocks) {
  const int64_t per = nblocks / 8;
  return b < per * 8 ? (b % 8) * per + b / 8 : b;
}

// Wait until at most N vector memory loads of this wave are outstanding.
template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Exclusive scan of one int per thread over the block; returns the prefix and
// writes the block total. `sh` needs blockDim/64 ints.
__device__ inline int block_exclusive_scan(int v, int *sh, int *total) {
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

}  // namespace last_dev
