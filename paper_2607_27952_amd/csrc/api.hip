// C ABI of liblast: argument validation on the host, workspace sizing, and the
// launch sequences of the three calls declared in include/last.h. Also the
// status strings and the optional per-kernel event timing.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "last_internal.h"

namespace last {

int score_max_pairs();

// ------------------------------------------------------------ diagnostics
static thread_local char g_err[256] = "";

void note_hip_error(hipError_t e) {
  snprintf(g_err, sizeof g_err, "%s (%d)", hipGetErrorString(e), (int)e);
}

namespace {
struct Pending {
  int kernel;
  hipEvent_t start, stop;
};
struct Totals {
  const char *name;  // a string literal of the launch site
  int64_t launches = 0;
  double ms = 0.0;
};
// Per-kernel event timing. The switch is an atomic read on every launch; the
// pools and totals are touched only while timing is on, under one lock. The
// launch being bracketed is per calling thread, so concurrent calls from
// different host threads never see each other's half-open pair.
struct Profiler {
  std::atomic<bool> on{false};
  std::mutex mu;
  std::vector<hipEvent_t> free_events;
  std::vector<Pending> pending;
  std::vector<Totals> totals;
  int created = 0;
};
Profiler &prof() {
  static Profiler p;
  return p;
}
thread_local Pending t_open{-1, nullptr, nullptr};
constexpr int kMaxEventPairs = 8192;

hipEvent_t take_event(Profiler &p) {  // p.mu held
  if (!p.free_events.empty()) {
    hipEvent_t e = p.free_events.back();
    p.free_events.pop_back();
    return e;
  }
  if (p.created >= 2 * kMaxEventPairs) return nullptr;
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  ++p.created;
  return e;
}

int kernel_id(Profiler &p, const char *name) {  // p.mu held
  for (size_t i = 0; i < p.totals.size(); ++i)
    if (strcmp(p.totals[i].name, name) == 0) return (int)i;
  p.totals.push_back(Totals{name, 0, 0.0});
  return (int)p.totals.size() - 1;
}
}  // namespace

void launch_begin(const char *name, hipStream_t s) {
  t_open = Pending{-1, nullptr, nullptr};
  Profiler &p = prof();
  if (!p.on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lock(p.mu);
  hipEvent_t a = take_event(p), b = take_event(p);
  if (!a || !b) {
    if (a) p.free_events.push_back(a);
    if (b) p.free_events.push_back(b);
    return;
  }
  if (hipEventRecord(a, s) != hipSuccess) {
    p.free_events.push_back(a);
    p.free_events.push_back(b);
    return;
  }
  t_open = Pending{kernel_id(p, name), a, b};
}

hipError_t launch_end(hipStream_t s) {
  hipError_t e = hipGetLastError();
  if (t_open.kernel >= 0) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> lock(p.mu);
    if (hipEventRecord(t_open.stop, s) == hipSuccess) {
      p.pending.push_back(t_open);
    } else {
      p.free_events.push_back(t_open.start);
      p.free_events.push_back(t_open.stop);
    }
    t_open = Pending{-1, nullptr, nullptr};
  }
  if (e != hipSuccess) note_hip_error(e);
  return e;
}

// Compute units of the current device, queried once per device.
int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// Ticks per millisecond of the device's constant-rate wall clock (wall_clock64),
// queried once per device.
int64_t device_wall_khz() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 100000;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeWallClockRate, dev) != hipSuccess || v <= 0) v = 100000;
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// ------------------------------------------------------------ validation
static bool csr_ok(const int32_t *cu, int32_t R, int32_t min_len) {
  if (!cu || cu[0] != 0) return false;
  for (int32_t r = 0; r < R; ++r)
    if ((int64_t)cu[r + 1] - cu[r] < min_len) return false;
  return true;
}

static last_status check_batch(const last_batch *b) {
  if (!b) return LAST_ERR_INVALID;
  if (b->R < 1 || b->G < 1 || b->Hq < 1 || b->Hkv < 1 || b->Dh < 1) return LAST_ERR_INVALID;
  if (b->Hq % b->Hkv != 0) return LAST_ERR_INVALID;
  if (b->qk_dtype != LAST_F32 && b->qk_dtype != LAST_BF16) return LAST_ERR_INVALID;
  if (!isfinite(b->softmax_scale)) return LAST_ERR_INVALID;
  if (!b->cu_seqlens || !b->vis_start || !b->cu_vis) return LAST_ERR_INVALID;
  if (!csr_ok(b->cu_seqlens_h, b->R, 2) || !csr_ok(b->cu_vis_h, b->R, 1) || !b->vis_start_h)
    return LAST_ERR_INVALID;
  for (int32_t r = 0; r < b->R; ++r) {
    const int64_t P = (int64_t)b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r];
    const int64_t N = (int64_t)b->cu_vis_h[r + 1] - b->cu_vis_h[r];
    const int64_t v = b->vis_start_h[r];
    if (v < 0 || v + N > P - 1) return LAST_ERR_INVALID;
  }
  if (b->Dh != 64 && b->Dh != 128) return LAST_ERR_UNSUPPORTED;
  if ((int64_t)b->G * b->Hq > score_max_pairs()) return LAST_ERR_UNSUPPORTED;
  return LAST_OK;
}

static last_status check_select(int32_t R, const int32_t *cu_vis_h, int32_t Dv, last_dtype fdtype,
                                last_sel_mode mode, const int32_t *cu_keep_h) {
  if (R < 1 || Dv < 1 || Dv > 65536) return LAST_ERR_INVALID;
  if (fdtype != LAST_F32 && fdtype != LAST_BF16) return LAST_ERR_INVALID;
  if (mode != LAST_SEL_KCENTER && mode != LAST_SEL_TOPK) return LAST_ERR_INVALID;
  if (!csr_ok(cu_vis_h, R, 1)) return LAST_ERR_INVALID;
  if (cu_keep_h) {
    if (!csr_ok(cu_keep_h, R, 1)) return LAST_ERR_INVALID;
    for (int32_t r = 0; r < R; ++r)
      if (cu_keep_h[r + 1] - cu_keep_h[r] > cu_vis_h[r + 1] - cu_vis_h[r]) return LAST_ERR_INVALID;
  }
  for (int32_t r = 0; r < R; ++r)
    if (cu_vis_h[r + 1] - cu_vis_h[r] > kSelMaxN) return LAST_ERR_UNSUPPORTED;
  if (mode == LAST_SEL_KCENTER && Dv % (fdtype == LAST_BF16 ? 8 : 4) != 0) return LAST_ERR_UNSUPPORTED;
  return LAST_OK;
}

static bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Query rows of last_rows_scores: at least one per request, each between the
// start of its request's visual span and the last token.
static last_status check_rows(const last_batch *b, const int32_t *cu_rows_h, const int32_t *row_pos_h) {
  if (!csr_ok(cu_rows_h, b->R, 1) || !row_pos_h) return LAST_ERR_INVALID;
  for (int32_t r = 0; r < b->R; ++r) {
    const int64_t P = (int64_t)b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r];
    for (int32_t m = cu_rows_h[r]; m < cu_rows_h[r + 1]; ++m)
      if (row_pos_h[m] < b->vis_start_h[r] || row_pos_h[m] >= P) return LAST_ERR_INVALID;
  }
  return LAST_OK;
}

static bool one_row_each(const last_batch *b, const int32_t *cu_rows_h) {
  for (int32_t r = 0; r < b->R; ++r)
    if (cu_rows_h[r + 1] - cu_rows_h[r] != 1) return false;
  return true;
}

}  // namespace last

using namespace last;

extern "C" {

size_t last_token_scores_workspace(const last_batch *b) {
  if (check_batch(b) != LAST_OK) return 0;
  const ScorePlan p = make_score_plan(b);
  size_t bytes = 0;
  carve_score_ws(nullptr, b, p, &bytes);
  return bytes;
}

last_status last_token_scores(const last_batch *b, const void *q, const void *k, float *scores,
                              float *attn_rows, void *ws, size_t ws_bytes, void *stream) {
  last_status st = check_batch(b);
  if (st != LAST_OK) return st;
  if (!q || !k || !scores) return LAST_ERR_INVALID;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(scores, 4) || (attn_rows && !aligned(attn_rows, 4)))
    return LAST_ERR_INVALID;
  const ScorePlan p = make_score_plan(b);
  size_t need = 0;
  carve_score_ws(nullptr, b, p, &need);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  const ScoreWs w = carve_score_ws(ws, b, p, &need);
  const float scale = b->softmax_scale > 0.f ? b->softmax_scale : 1.0f / sqrtf((float)b->Dh);
  const hipError_t e = launch_scores(b, p, w, q, k, nullptr, scores, attn_rows, scale, (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

}  // extern "C"

// ------------------------------------------------------------ static scratch
// The scratch of last_token_scores_static: one copy on every device that loads
// the library, kept until the process ends. Host code never passes this name to
// a kernel (on the host it is only a stand-in for the symbol); it uses the
// device address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[LAST_STATIC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};
}  // namespace

// The current device's address of `scratch`, looked up on the device's first call.
static last_status static_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    note_hip_error(e);
    return LAST_ERR_DEVICE;
  }
  if (dev < 0 || dev >= kMaxDevices) return LAST_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      note_hip_error(e);
      return LAST_ERR_DEVICE;
    }
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return LAST_OK;
}

extern "C" {

last_status last_token_scores_static(const last_batch *b, const void *q, const void *k, float *scores,
                                     float *attn_rows, void *stream) {
  last_status st = check_batch(b);
  if (st != LAST_OK) return st;
  if (!q || !k || !scores) return LAST_ERR_INVALID;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(scores, 4) || (attn_rows && !aligned(attn_rows, 4)))
    return LAST_ERR_INVALID;
  const ScorePlan p = make_score_plan(b);
  size_t need = 0;
  carve_score_ws(nullptr, b, p, &need);
  if (need > LAST_STATIC_SCRATCH_BYTES) return LAST_ERR_WORKSPACE;
  void *ws = nullptr;
  st = static_scratch(&ws);
  if (st != LAST_OK) return st;
  const ScoreWs w = carve_score_ws(ws, b, p, &need);
  const float scale = b->softmax_scale > 0.f ? b->softmax_scale : 1.0f / sqrtf((float)b->Dh);
  const hipError_t e = launch_scores(b, p, w, q, k, nullptr, scores, attn_rows, scale, (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

int32_t last_source_rows(last_source src, int32_t q_begin, int32_t q_end, int32_t *pos_h) {
  if (q_begin < 0 || q_end <= q_begin || !pos_h) return -1;
  const int32_t M = q_end - q_begin;
  switch (src) {
    case LAST_SRC_LAST: pos_h[0] = q_end - 1; return 1;
    case LAST_SRC_FIRST: pos_h[0] = q_begin; return 1;
    case LAST_SRC_MIDDLE: pos_h[0] = q_begin + (M - 1) / 2; return 1;   // q_ceil(M/2), 1-based
    case LAST_SRC_ALL_MEAN:
      for (int32_t m = 0; m < M; ++m) pos_h[m] = q_begin + m;
      return M;
  }
  return -1;
}

size_t last_rows_scores_workspace(const last_batch *b, const int32_t *cu_rows_h, const int32_t *row_pos_h) {
  if (check_batch(b) != LAST_OK || check_rows(b, cu_rows_h, row_pos_h) != LAST_OK) return 0;
  size_t bytes = 0;
  if (one_row_each(b, cu_rows_h)) {
    const ScorePlan p = make_score_plan(b, row_pos_h);
    carve_score_ws(nullptr, b, p, &bytes);
  } else {
    const RowsPlan p = make_rows_plan(b, cu_rows_h, row_pos_h);
    carve_rows_ws(nullptr, b, p, &bytes);
  }
  return bytes;
}

last_status last_rows_scores(const last_batch *b, const int32_t *cu_rows, const int32_t *cu_rows_h,
                             const int32_t *row_pos, const int32_t *row_pos_h, const void *q,
                             const void *k, float *scores, void *ws, size_t ws_bytes, void *stream) {
  last_status st = check_batch(b);
  if (st != LAST_OK) return st;
  st = check_rows(b, cu_rows_h, row_pos_h);
  if (st != LAST_OK) return st;
  if (!cu_rows || !row_pos || !q || !k || !scores) return LAST_ERR_INVALID;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(scores, 4)) return LAST_ERR_INVALID;
  const size_t need = last_rows_scores_workspace(b, cu_rows_h, row_pos_h);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  const float scale = b->softmax_scale > 0.f ? b->softmax_scale : 1.0f / sqrtf((float)b->Dh);
  hipError_t e;
  size_t used = 0;
  if (one_row_each(b, cu_rows_h)) {
    // one row per request: q is [G][R][Hq][Dh], the streamed single-row kernels
    const ScorePlan p = make_score_plan(b, row_pos_h);
    const ScoreWs w = carve_score_ws(ws, b, p, &used);
    e = launch_scores(b, p, w, q, k, row_pos, scores, nullptr, scale, (hipStream_t)stream);
  } else {
    const RowsPlan p = make_rows_plan(b, cu_rows_h, row_pos_h);
    const RowsWs w = carve_rows_ws(ws, b, p, &used);
    e = launch_rows(b, p, w, cu_rows, row_pos, q, k, scores, scale, (hipStream_t)stream);
  }
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

// The prefill's score-pass plan: one chunk per request (the prefill kernel
// writes each request's last-row statistics as a single chunk).
static ScorePlan prefill_score_plan(const last_batch *b) {
  ScorePlan p = make_score_plan(b);
  int32_t pmax = 1;
  for (int32_t r = 0; r < b->R; ++r) pmax = std::max(pmax, b->cu_seqlens_h[r + 1] - b->cu_seqlens_h[r]);
  p.chunk_tokens = pmax;
  p.C_total = b->R;
  return p;
}

static size_t prefill_ws(const last_batch *b, void *ws, ScoreWs *sw, int32_t **qb_off, int32_t **qb_req) {
  const ScorePlan p = prefill_score_plan(b);
  size_t used = 0;
  const ScoreWs w = carve_score_ws(ws, b, p, &used);
  if (sw) *sw = w;
  Carver cv(ws ? static_cast<char *>(ws) + used : nullptr);
  int32_t *a = cv.take<int32_t>(b->R + 1);
  int32_t *c = cv.take<int32_t>(prefill_query_blocks(b));
  if (qb_off) *qb_off = a;
  if (qb_req) *qb_req = c;
  return used + cv.size();
}

size_t last_prefill_attention_workspace(const last_batch *b) {
  if (check_batch(b) != LAST_OK || b->qk_dtype != LAST_BF16) return 0;
  return prefill_ws(b, nullptr, nullptr, nullptr, nullptr);
}

last_status last_prefill_attention(const last_batch *b, const void *q, const void *k, const void *v,
                                   void *out, float *scores, void *ws, size_t ws_bytes, void *stream) {
  last_status st = check_batch(b);
  if (st != LAST_OK) return st;
  if (!q || !k || !v || !out || !scores) return LAST_ERR_INVALID;
  if (b->qk_dtype != LAST_BF16) return LAST_ERR_UNSUPPORTED;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) || !aligned(scores, 4))
    return LAST_ERR_INVALID;
  const size_t need = prefill_ws(b, nullptr, nullptr, nullptr, nullptr);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  ScoreWs w;
  int32_t *qb_off = nullptr, *qb_req = nullptr;
  prefill_ws(b, ws, &w, &qb_off, &qb_req);
  const ScorePlan p = prefill_score_plan(b);
  const float scale = b->softmax_scale > 0.f ? b->softmax_scale : 1.0f / sqrtf((float)b->Dh);
  const hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_score_plan(b, p, w, nullptr, s);
  if (e == hipSuccess)
    e = launch_prefill(b, prefill_query_blocks(b), qb_off, qb_req, q, k, v, out, w.vlog, w.stats, scale, s);
  if (e == hipSuccess) e = launch_score_tail(b, p, w, nullptr, scores, s);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

// Workspace of a selection plan: its carve, then scratch for the pick order
// and gains when the caller does not want them.
static size_t select_ws_bytes(int32_t R, const SelectPlan &p, last_sel_mode mode) {
  size_t bytes = 0;
  carve_select_ws(nullptr, R, p, mode, &bytes);
  bytes += align_up((size_t)p.N_total * sizeof(int32_t), 256) + align_up((size_t)p.N_total * sizeof(float), 256);
  return bytes;
}

size_t diverse_select_workspace(int32_t R, const int32_t *cu_vis_h, int32_t Dv, last_dtype fdtype,
                                last_sel_mode mode) {
  if (check_select(R, cu_vis_h, Dv, fdtype, mode, nullptr) != LAST_OK) return 0;
  // The budgets change neither the form nor the workspace; plan with K_r = N_r.
  const SelectPlan p = make_select_plan(R, cu_vis_h, cu_vis_h, mode, Dv, fdtype, false, true);
  return select_ws_bytes(R, p, mode);
}

size_t diverse_select_similarity_workspace(int32_t R, const int32_t *cu_vis_h, int32_t Dv, last_dtype fdtype) {
  if (check_select(R, cu_vis_h, Dv, fdtype, LAST_SEL_KCENTER, nullptr) != LAST_OK) return 0;
  const SelectPlan p = make_select_plan(R, cu_vis_h, cu_vis_h, LAST_SEL_KCENTER, Dv, fdtype, false, false);
  return select_ws_bytes(R, p, LAST_SEL_KCENTER);
}

last_status diverse_select(int32_t R, int32_t Dv, last_dtype fdtype, last_sel_mode mode,
                           const float *scores, const void *feats, const int32_t *cu_vis,
                           const int32_t *cu_vis_h, const int32_t *cu_keep, const int32_t *cu_keep_h,
                           int32_t *kept, int32_t *order, float *gains, void *ws, size_t ws_bytes,
                           void *stream) {
  if (!cu_keep_h) return LAST_ERR_INVALID;
  last_status st = check_select(R, cu_vis_h, Dv, fdtype, mode, cu_keep_h);
  if (st != LAST_OK) return st;
  if (!scores || !feats || !cu_vis || !cu_keep || !kept) return LAST_ERR_INVALID;
  if (!aligned(feats, 16)) return LAST_ERR_INVALID;
  const SelectPlan p = make_select_plan(R, cu_vis_h, cu_keep_h, mode, Dv, fdtype, true, true);
  const size_t need = select_ws_bytes(R, p, mode);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  size_t used = 0;
  const SelectWs w = carve_select_ws(ws, R, p, mode, &used);
  char *tail = static_cast<char *>(ws) + used;
  int32_t *order_ws = reinterpret_cast<int32_t *>(tail);
  float *gains_ws = reinterpret_cast<float *>(tail + align_up((size_t)p.N_total * sizeof(int32_t), 256));
  const hipError_t e = launch_select(R, Dv, fdtype, mode, p, w, scores, feats, cu_vis, cu_keep, kept,
                                     order ? order : order_ws, gains ? gains : gains_ws,
                                     (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

// Workspace check and carve shared by the two k-center phases: the same
// (R, cu_vis_h, Dv, fdtype) give the same layout in both calls.
static last_status kcenter_ws(int32_t R, const int32_t *cu_vis_h, int32_t Dv, last_dtype fdtype,
                              void *ws, size_t ws_bytes, SelectPlan *p, SelectWs *w) {
  *p = make_select_plan(R, cu_vis_h, cu_vis_h, LAST_SEL_KCENTER, Dv, fdtype, false, false);
  const size_t need = select_ws_bytes(R, *p, LAST_SEL_KCENTER);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  size_t used = 0;
  *w = carve_select_ws(ws, R, *p, LAST_SEL_KCENTER, &used);
  return LAST_OK;
}

last_status diverse_select_similarity(int32_t R, int32_t Dv, last_dtype fdtype, const void *feats,
                                      const int32_t *cu_vis, const int32_t *cu_vis_h, void *ws,
                                      size_t ws_bytes, void *stream) {
  last_status st = check_select(R, cu_vis_h, Dv, fdtype, LAST_SEL_KCENTER, nullptr);
  if (st != LAST_OK) return st;
  if (!feats || !cu_vis) return LAST_ERR_INVALID;
  if (!aligned(feats, 16)) return LAST_ERR_INVALID;
  SelectPlan p;
  SelectWs w;
  if ((st = kcenter_ws(R, cu_vis_h, Dv, fdtype, ws, ws_bytes, &p, &w)) != LAST_OK) return st;
  const hipError_t e = launch_similarity(R, Dv, fdtype, p, w, feats, cu_vis, (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

last_status diverse_select_pick(int32_t R, int32_t Dv, last_dtype fdtype, const float *scores,
                                const int32_t *cu_vis, const int32_t *cu_vis_h, const int32_t *cu_keep,
                                const int32_t *cu_keep_h, int32_t *kept, int32_t *order, float *gains,
                                void *ws, size_t ws_bytes, void *stream) {
  if (!cu_keep_h) return LAST_ERR_INVALID;
  last_status st = check_select(R, cu_vis_h, Dv, fdtype, LAST_SEL_KCENTER, cu_keep_h);
  if (st != LAST_OK) return st;
  if (!scores || !cu_vis || !cu_keep || !kept) return LAST_ERR_INVALID;
  SelectPlan p;
  SelectWs w;
  if ((st = kcenter_ws(R, cu_vis_h, Dv, fdtype, ws, ws_bytes, &p, &w)) != LAST_OK) return st;
  size_t used = 0;
  carve_select_ws(nullptr, R, p, LAST_SEL_KCENTER, &used);
  char *tail = static_cast<char *>(ws) + used;
  int32_t *order_ws = reinterpret_cast<int32_t *>(tail);
  float *gains_ws = reinterpret_cast<float *>(tail + align_up((size_t)p.N_total * sizeof(int32_t), 256));
  const hipError_t e = launch_pick(R, LAST_SEL_KCENTER, p, w, scores, cu_vis, cu_keep, kept,
                                   order ? order : order_ws, gains ? gains : gains_ws, (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

last_status gather_kept(int32_t R, int32_t Dv, size_t elem_bytes, const void *feats,
                        const int32_t *cu_vis, const int32_t *cu_vis_h, const int32_t *kept,
                        const int32_t *cu_keep, const int32_t *cu_keep_h, void *out, void *stream) {
  if (R < 1 || Dv < 1 || Dv > 65536) return LAST_ERR_INVALID;
  if (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4 && elem_bytes != 8) return LAST_ERR_INVALID;
  if (!csr_ok(cu_vis_h, R, 0) || !csr_ok(cu_keep_h, R, 0)) return LAST_ERR_INVALID;
  if (!cu_vis || !cu_keep) return LAST_ERR_INVALID;
  const int64_t K_total = cu_keep_h[R];
  if (K_total > 0 && (!feats || !kept || !out)) return LAST_ERR_INVALID;
  const hipError_t e = launch_gather(R, (int64_t)Dv * (int64_t)elem_bytes, K_total, cu_vis_h[R],
                                     feats, cu_vis, kept, cu_keep, out, (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

static bool connector_dims_ok(int64_t K, int32_t Dv, int32_t Dh) {
  return K >= 0 && K < ((int64_t)1 << 31) && Dv >= 1 && Dh >= 1 && Dv <= 65536 && Dh <= 65536;
}

static size_t connector_ws(int64_t K, int32_t Dv, int32_t Dh) {
  Carver c(nullptr);
  c.take<uint16_t>((size_t)K * Dv);
  c.take<uint16_t>((size_t)K * Dh);
  return c.size();
}

size_t last_connector_workspace(int64_t K, int32_t Dv, int32_t Dh) {
  if (!connector_dims_ok(K, Dv, Dh)) return 0;
  return connector_ws(K, Dv, Dh);
}

last_status last_connector(last_dtype dtype, int64_t K, int32_t Dv, int32_t Dh, int32_t Do, float eps,
                           const void *x, const float *gamma, const float *beta, const void *w1,
                           const float *b1, const void *w2, const float *b2, void *out, void *ws,
                           size_t ws_bytes, void *stream) {
  if (!connector_dims_ok(K, Dv, Dh) || Do < 1 || Do > 65536) return LAST_ERR_INVALID;
  if (!(eps > 0.0f) || !std::isfinite(eps)) return LAST_ERR_INVALID;
  if (dtype != LAST_BF16 && dtype != LAST_F32) return LAST_ERR_INVALID;
  if (dtype != LAST_BF16 || Dv < 64 || Dh < 64 || Do < 64 || !connector_shape_ok(K, Dv, Dh, Do))
    return LAST_ERR_UNSUPPORTED;
  if (K == 0) return LAST_OK;
  if (!x || !gamma || !beta || !w1 || !b1 || !w2 || !b2 || !out) return LAST_ERR_INVALID;
  if (!aligned(x, 16) || !aligned(w1, 16) || !aligned(w2, 16) || !aligned(b1, 16) || !aligned(b2, 16) ||
      !aligned(out, 16) || !aligned(gamma, 16) || !aligned(beta, 16))
    return LAST_ERR_INVALID;
  const size_t need = connector_ws(K, Dv, Dh);
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return LAST_ERR_WORKSPACE;
  Carver c(ws);
  void *xn = c.take<uint16_t>((size_t)K * Dv);
  void *hid = c.take<uint16_t>((size_t)K * Dh);
  const hipError_t e = launch_connector(K, Dv, Dh, Do, eps, x, gamma, beta, w1, b1, w2, b2, out, xn, hid,
                                        (hipStream_t)stream);
  return e == hipSuccess ? LAST_OK : LAST_ERR_DEVICE;
}

int32_t last_budget(int32_t N, int32_t rho_num, int32_t rho_den) {
  if (N < 1 || rho_num < 1 || rho_den < 1 || rho_num > rho_den) return -1;
  int64_t k = ((int64_t)N * rho_num + rho_den - 1) / rho_den;
  if (k < 1) k = 1;
  if (k > N) k = N;
  return (int32_t)k;
}

const char *last_status_string(last_status s) {
  static thread_local char buf[320];
  switch (s) {
    case LAST_OK: return "ok";
    case LAST_ERR_INVALID: return "invalid argument";
    case LAST_ERR_UNSUPPORTED: return "unsupported configuration";
    case LAST_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case LAST_ERR_DEVICE:
      snprintf(buf, sizeof buf, "device error: %s", g_err[0] ? g_err : "unknown");
      return buf;
  }
  return "unknown status";
}

int32_t last_version(void) { return 100; }

last_status last_profile_enable(int32_t on) {
  prof().on.store(on != 0, std::memory_order_relaxed);
  return LAST_OK;
}

last_status last_profile_collect(void) {
  Profiler &p = prof();
  std::lock_guard<std::mutex> lock(p.mu);
  std::vector<Pending> keep;
  for (const Pending &x : p.pending) {
    float ms = 0.f;
    const hipError_t e = hipEventElapsedTime(&ms, x.start, x.stop);
    if (e == hipErrorNotReady) {
      keep.push_back(x);
      continue;
    }
    if (e == hipSuccess) {
      p.totals[x.kernel].launches += 1;
      p.totals[x.kernel].ms += ms;
    }
    p.free_events.push_back(x.start);
    p.free_events.push_back(x.stop);
  }
  p.pending.swap(keep);
  return p.pending.empty() ? LAST_OK : LAST_ERR_DEVICE;
}

void last_profile_reset(void) {
  Profiler &p = prof();
  std::lock_guard<std::mutex> lock(p.mu);
  for (Totals &t : p.totals) {
    t.launches = 0;
    t.ms = 0.0;
  }
}

int32_t last_profile_count(void) {
  Profiler &p = prof();
  std::lock_guard<std::mutex> lock(p.mu);
  return (int32_t)p.totals.size();
}

int32_t last_profile_kernel(int32_t i, const char **name, int64_t *launches, double *total_ms) {
  Profiler &p = prof();
  std::lock_guard<std::mutex> lock(p.mu);
  if (i < 0 || i >= (int32_t)p.totals.size()) return 0;
  if (name) *name = p.totals[i].name;
  if (launches) *launches = p.totals[i].launches;
  if (total_ms) *total_ms = p.totals[i].ms;
  return 1;
}

}  // extern "C"
