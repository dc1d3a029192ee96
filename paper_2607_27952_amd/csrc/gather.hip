// Payload build of LAST (arXiv 2607.27952, Sec. 3.4, Eq. 12): the kept rows
// of X, in the ascending order of the kept indices, copied byte for byte.
//
// One wave per output row. The row's request is found with a 64-ary search
// over cu_keep (one probe per lane per level), then the row is copied with
// 16-byte vector loads/stores when the row size and both base pointers allow
// it, else byte by byte. An out-of-range kept index yields a zero row.
#include "last_internal.h"

namespace {

__global__ __launch_bounds__(256) void k_gather(const uint8_t *__restrict__ feats,
                                                const int32_t *__restrict__ cu_vis,
                                                const int32_t *__restrict__ kept,
                                                const int32_t *__restrict__ cu_keep, int R,
                                                int64_t row_bytes, int64_t K_total,
                                                int64_t N_total, int vec16,
                                                uint8_t *__restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < K_total; t += stride) {
    // largest r with cu_keep[r] <= t
    int lo = 0, hi = R;
    while (hi - lo > 1) {
      const int step = (hi - lo + 63) / 64;
      const int idx = lo + lane * step;
      const bool ok = idx < hi && cu_keep[idx] <= t;
      const unsigned long long m = __ballot(ok);
      const int last = 63 - __clzll(m);
      lo = lo + last * step;
      hi = min(hi, lo + step);
    }
    const int r = lo;
    const int64_t k = kept[t];
    const int64_t n_r = cu_vis[r + 1] - cu_vis[r];
    const int64_t src_row = cu_vis[r] + k;
    const bool valid = k >= 0 && k < n_r && src_row < N_total;
    uint8_t *dst = out + t * row_bytes;
    if (vec16) {
      uint4 *d4 = reinterpret_cast<uint4 *>(dst);
      const uint4 *s4 = reinterpret_cast<const uint4 *>(feats + (valid ? src_row : 0) * row_bytes);
      const int64_t n4 = row_bytes >> 4;
      for (int64_t x = lane; x < n4; x += 64) d4[x] = valid ? s4[x] : make_uint4(0, 0, 0, 0);
    } else {
      const uint8_t *s1 = feats + (valid ? src_row : 0) * row_bytes;
      for (int64_t x = lane; x < row_bytes; x += 64) dst[x] = valid ? s1[x] : (uint8_t)0;
    }
  }
}

}  // namespace

namespace last {

hipError_t launch_gather(int32_t R, int64_t row_bytes, int64_t K_total, int64_t N_total,
                         const void *feats, const int32_t *cu_vis, const int32_t *kept,
                         const int32_t *cu_keep, void *out, hipStream_t s) {
  if (K_total == 0) return hipSuccess;
  const int vec16 = (row_bytes % 16 == 0) && ((uintptr_t)feats % 16 == 0) && ((uintptr_t)out % 16 == 0);
  int64_t blocks = (K_total + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  launch_begin("gather", s);
  hipLaunchKernelGGL(k_gather, dim3((unsigned)blocks), dim3(256), 0, s, (const uint8_t *)feats,
                     cu_vis, kept, cu_keep, R, row_bytes, K_total, N_total,
                     vec16, (uint8_t *)out);
  return launch_end(s);
}

}  // namespace last
