/*
 * last.h -- C ABI of the MI355X (gfx950) LAST token-selection library.
 *
 * LAST (arXiv 2607.27952) prunes visual tokens before edge-to-cloud
 * transmission. This library implements the data-parallel hot path:
 *
 *   last_token_scores  Sec. 3.3, Eq. 6-8: the attention row of the last query
 *                      token against every key of the guidance model's prefill
 *                      (softmax over the whole visual + text context), its
 *                      visual columns summed over guidance layers and heads,
 *                      normalised over the visual tokens.
 *   last_rows_scores   Sec. 4.3, Table 4: the same scores from other causal
 *                      query rows (first, middle or every query token).
 *   last_prefill_attention  Sec. 3.3: the guidance model's causal prefill
 *                      attention, with the same scores read from its last row.
 *   diverse_select     Sec. 3.4, Eq. 9-12: importance-weighted greedy k-center
 *                      over unit-normalised encoder features under a budget
 *                      K = ceil(rho N) (Eq. 2); or the Top-k ablation of
 *                      Sec. 4.3, Table 5. Kept indices come out ascending.
 *   diverse_select_similarity, diverse_select_pick  the k-center of
 *                      diverse_select in two calls (distances, then greedy),
 *                      so the distances can overlap the score pass.
 *   gather_kept        Sec. 3.4, Eq. 12: the kept rows X_S, in original order,
 *                      copied byte for byte for transmission.
 *
 * Conventions shared by every call
 *   - Pointers without a suffix are device pointers; pointers suffixed _h are
 *     host copies of the same small arrays, used for validation and launch
 *     planning. Each _h array must hold exactly what its device twin holds.
 *   - The caller owns every buffer, including the workspace (size it with the
 *     matching *_workspace query). The library never allocates device memory,
 *     never synchronises, and only enqueues work on `stream` (a hipStream_t;
 *     NULL is the default stream).
 *   - Every argument is validated on the host, from the _h copies, before any
 *     HIP call. On error nothing is enqueued, outputs are left untouched, and
 *     a non-zero last_status is returned. A failed kernel launch returns
 *     LAST_ERR_DEVICE (possibly after earlier kernels of the same call have
 *     been enqueued).
 *   - Ragged batches of R requests are packed with CSR offsets (int32, length
 *     R+1, starting at 0, non-decreasing). Indices into a request's visual
 *     tokens are request-local int32 in [0, N_r).
 *   - Results are deterministic: the same inputs give bitwise-identical
 *     outputs on every run (fixed reduction orders, ties to the lowest index).
 *   - Calls on different streams are independent if their workspaces and
 *     outputs do not overlap.
 */
#ifndef LAST_H
#define LAST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LAST_OK = 0,
  LAST_ERR_INVALID = 1,     /* malformed arguments (shapes, CSR, budgets, NULLs) */
  LAST_ERR_UNSUPPORTED = 2, /* valid but outside what the kernels implement */
  LAST_ERR_WORKSPACE = 3,   /* workspace pointer NULL or smaller than required */
  LAST_ERR_DEVICE = 4       /* a HIP call failed; see last_status_string */
} last_status;

typedef enum { LAST_F32 = 0, LAST_BF16 = 1 } last_dtype;

typedef enum {
  LAST_SEL_KCENTER = 0, /* Eq. 9-11: greedy argmax of w_i * delta_i */
  LAST_SEL_TOPK = 1     /* Table 5 "LAST (Top-k)": the K largest w_i */
} last_sel_mode;

/*
 * Batch description for last_token_scores.
 *   R          number of requests (>= 1)
 *   G          guidance layers whose rows are summed (Eq. 7 sums over layers;
 *              any subset of a model's layers can be passed, G >= 1)
 *   Hq, Hkv    query and key heads; Hq % Hkv == 0. Query head h reads KV head
 *              h / (Hq / Hkv) (grouped-query attention). Eq. 7 sums over all
 *              Hq query heads.
 *   Dh         head dimension, 64 or 128 (others: LAST_ERR_UNSUPPORTED)
 *   qk_dtype   storage type of q and k (LAST_F32 or LAST_BF16)
 *   softmax_scale  sigma in softmax(sigma q.k); <= 0 selects 1/sqrt(Dh)
 *   cu_seqlens [R+1] token offsets into k; P_r = cu_seqlens[r+1]-cu_seqlens[r]
 *              is the prefill length of request r (>= 2). Its last token,
 *              position P_r - 1, is the query token whose row is scored.
 *   vis_start  [R] start of request r's visual span within its sequence
 *   cu_vis     [R+1] offsets into scores (and into the features given to
 *              diverse_select); N_r = cu_vis[r+1]-cu_vis[r] >= 1 visual tokens
 *              occupy positions [vis_start[r], vis_start[r] + N_r), which must
 *              end before the last token: vis_start[r] + N_r <= P_r - 1.
 */
typedef struct last_batch {
  int32_t R, G, Hq, Hkv, Dh;
  last_dtype qk_dtype;
  float softmax_scale;
  const int32_t *cu_seqlens, *cu_seqlens_h;
  const int32_t *vis_start, *vis_start_h;
  const int32_t *cu_vis, *cu_vis_h;
} last_batch;

/* Workspace bytes last_token_scores needs for this batch (0 if invalid). */
size_t last_token_scores_workspace(const last_batch *b);

/*
 * Sec. 3.3, Eq. 6-8.
 *   q          [G][R][Hq][Dh] the last query token of each request, per layer
 *              (after rotary embedding, as the attention sees it)
 *   k          [G][T_total][Hkv][Dh] keys of every prefill token (after rotary
 *              embedding), T_total = cu_seqlens[R]
 *   scores     [N_total] out: w~ per visual token; each request's entries are
 *              >= 0 and sum to 1 (Eq. 8)
 *   attn_rows  optional [G][Hq][T_total] out (NULL to skip): the full softmax
 *              rows A^(l,h)[p*, :] of every request, for inspection
 *   ws         device workspace of at least last_token_scores_workspace(b)
 *              bytes, 256-byte aligned
 */
last_status last_token_scores(const last_batch *b, const void *q, const void *k,
                              float *scores, float *attn_rows, void *ws,
                              size_t ws_bytes, void *stream);

/*
 * last_token_scores without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Same arguments, kernels and results as
 * last_token_scores; its scratch is a static device array of
 * LAST_STATIC_SCRATCH_BYTES that every device running the library holds until
 * the process ends. The call itself allocates nothing: the array's address is
 * looked up once per device, on that device's first call.
 *   - A batch whose workspace (last_token_scores_workspace) exceeds
 *     LAST_STATIC_SCRATCH_BYTES is rejected with LAST_ERR_WORKSPACE before any
 *     HIP call.
 *   - The current device must be the one `stream` belongs to.
 *   - All calls on one device share its array: calls that overlap in time on
 *     one device (different streams, or different host threads) race and give
 *     undefined results. Nothing in the array needs to start at zero; each call
 *     writes every part it reads.
 */
#define LAST_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
last_status last_token_scores_static(const last_batch *b, const void *q,
                                     const void *k, float *scores,
                                     float *attn_rows, void *stream);

/*
 * Sec. 4.3, Table 4 (attention-source ablation): the sources compared there,
 * for a text query of M tokens q_1 .. q_M at positions q_begin .. q_end - 1
 * of a request (M = q_end - q_begin; q_M is the last query token p*).
 *   LAST_SRC_LAST      q_M            (the method's choice, Eq. 7)
 *   LAST_SRC_FIRST     q_1
 *   LAST_SRC_MIDDLE    q_ceil(M/2)    (indices count query tokens)
 *   LAST_SRC_ALL_MEAN  q_1 .. q_M     (rows averaged; the average and the sum
 *                                      give the same scores after Eq. 8)
 */
typedef enum {
  LAST_SRC_LAST = 0,
  LAST_SRC_FIRST = 1,
  LAST_SRC_MIDDLE = 2,
  LAST_SRC_ALL_MEAN = 3
} last_source;

/* Host helper: writes the request-local positions of source `src`'s rows to
 * pos_h (room for q_end - q_begin entries) in increasing order and returns
 * how many; -1 for q_begin < 0, q_end <= q_begin or an unknown source. */
int32_t last_source_rows(last_source src, int32_t q_begin, int32_t q_end, int32_t *pos_h);

/* Workspace bytes last_rows_scores needs (0 if the arguments are invalid). */
size_t last_rows_scores_workspace(const last_batch *b, const int32_t *cu_rows_h,
                                  const int32_t *row_pos_h);

/*
 * Sec. 4.3, Table 4, generalising Eq. 6-8 from the last query token's row to
 * any set of query rows per request:
 *   s_i = sum_l sum_h sum_{m in rows(r)} A^(l,h)[p_m, v_r + i],  w~ = s / sum s
 * Under the causal mask the row at position p attends to keys 0 .. p only:
 * its softmax runs over those p + 1 keys and visual tokens after p get
 * nothing from it.
 *   b          as for last_token_scores
 *   cu_rows    [R+1] CSR offsets of each request's rows; M_r >= 1
 *   row_pos    [M_total] request-local position of each row, with
 *              vis_start[r] <= p < P_r (every row sees a visual token)
 *   q          [G][M_total][Hq][Dh] the queries of those rows (after rotary
 *              embedding), same dtype as k
 *   k, scores, ws, stream   as for last_token_scores
 * One row per request (Last, First, Middle) runs the streamed single-row
 * kernels; several rows (All Mean) run two matrix-core passes over the keys:
 * row statistics, then the visual probabilities summed over rows and heads.
 * The result with one row per request at P_r - 1 equals last_token_scores.
 */
last_status last_rows_scores(const last_batch *b, const int32_t *cu_rows,
                             const int32_t *cu_rows_h, const int32_t *row_pos,
                             const int32_t *row_pos_h, const void *q, const void *k,
                             float *scores, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes last_prefill_attention needs (0 if invalid). */
size_t last_prefill_attention_workspace(const last_batch *b);

/*
 * Sec. 3.3: the guidance model's causal prefill attention, whose attention
 * tensors LAST reads, with the relevance of Eq. 6-8 taken from the same pass
 * (no second pass over the keys):
 *   out_p = sum_{j <= p} softmax_j(sigma q_p . k_j) v_j   for every position p
 *   scores = w~ from the rows of the last position of each request, exactly
 *            as last_token_scores computes them.
 *   b          as for last_token_scores; qk_dtype must be LAST_BF16 (others:
 *              LAST_ERR_UNSUPPORTED)
 *   q          [G][T_total][Hq][Dh] queries of every prefill position (after
 *              rotary embedding); each request's last position is its last
 *              query token
 *   k, v       [G][T_total][Hkv][Dh] keys and values
 *   out        [G][T_total][Hq][Dh] out, bf16 (rounded to nearest even)
 *   scores     [N_total] out, as for last_token_scores
 * The products use bf16 inputs with fp32 accumulation; the probabilities
 * enter the value product rounded to bf16 (relative error <= 2^-8 each).
 */
last_status last_prefill_attention(const last_batch *b, const void *q, const void *k,
                                   const void *v, void *out, float *scores, void *ws,
                                   size_t ws_bytes, void *stream);

/* Workspace bytes diverse_select needs (0 if the arguments are invalid):
 * for the k-center, those of the form it will take (see diverse_select),
 * which LAST_KCENTER_FORM, read at every call, can change. */
size_t diverse_select_workspace(int32_t R, const int32_t *cu_vis_h, int32_t Dv,
                                last_dtype fdtype, last_sel_mode mode);

/*
 * Sec. 3.4, Eq. 9-12 (mode LAST_SEL_KCENTER) or Sec. 4.3, Table 5
 * (mode LAST_SEL_TOPK).
 *   scores     [N_total] non-negative, finite fp32 relevance per visual token
 *              (normally the output of last_token_scores; any source works;
 *              negative or NaN entries are treated as 0)
 *   feats      [N_total][Dv] encoder features X of the visual tokens,
 *              row-major, fdtype (LAST_F32 or LAST_BF16); 1 <= Dv <= 65536
 *   cu_vis     [R+1] as in last_batch; N_r <= 131072 per request. The
 *              k-center takes one of two forms with the same results, bit
 *              for bit:
 *              - the matrix: all coverage distances of each request at once
 *                (4 ceil(N_r/128)^2 128^2 bytes of workspace per request:
 *                17 GB at 65536 tokens, 69 GB at 131072), then the greedy;
 *              - the rounds (bf16 features, Dv a multiple of 256 up to 4096,
 *                N_r <= 32768): only the distances to the tokens picked (the
 *                paper's O(K N d_v) form, about 1 KB of workspace per token
 *                and 148 KB per request), computed for up to 64 picks at a
 *                time; the picks of a round are certified exact against every
 *                token outside its 192 candidates.
 *              By default the rounds take batches whose every request has
 *              8192 tokens or more and the shapes above; the environment
 *              variable LAST_KCENTER_FORM=gram or =rounds forces one (rounds
 *              only where those shapes allow). The rounds run as a queue of
 *              tasks on one block per compute unit in which no block waits
 *              for one that has not started; a wait longer than 10 s (the
 *              device kept busy by other work) fills every unfinished
 *              request's kept and order with -1 and its gains with NaN.
 *              In the matrix form, requests longer than 32768 tokens (and longer than
 *              8192 when the batch is small) run the greedy on several
 *              compute units that exchange their candidates every step; if
 *              they cannot all run at once for 10 s (the device kept full
 *              by other work), the request's kept and order are filled
 *              with -1 and its gains with NaN (blocks that time out at the
 *              very end may leave some of the request's valid indices
 *              beside the -1 entries; either way the request is invalid).
 *              The environment variable LAST_MC_WAIT_US, read at every
 *              call, replaces the 10 s of either form (in microseconds)
 *   cu_keep    [R+1] budgets: K_r = cu_keep[r+1]-cu_keep[r], 1 <= K_r <= N_r
 *              (use last_budget for K = ceil(rho N), Eq. 2)
 *   kept       [K_total] out: the selected request-local indices, ascending
 *              within each request (Eq. 12)
 *   order      optional [K_total] out: the pick sequence j_1..j_K (k-center),
 *              or the kept indices by decreasing score (Top-k)
 *   gains      optional [K_total] out: w_j1 at t = 1 and w_jt * delta_jt at
 *              t >= 2 (k-center), or the scores in pick order (Top-k)
 * Ties in every argmax go to the lowest index. The coverage distance of
 * Eq. 10 is 1 - cos clamped at 0; a zero-norm feature has cosine 0 with
 * every token; bitwise-identical features are at distance exactly 0.
 */
last_status diverse_select(int32_t R, int32_t Dv, last_dtype fdtype,
                           last_sel_mode mode, const float *scores,
                           const void *feats, const int32_t *cu_vis,
                           const int32_t *cu_vis_h, const int32_t *cu_keep,
                           const int32_t *cu_keep_h, int32_t *kept,
                           int32_t *order, float *gains, void *ws,
                           size_t ws_bytes, void *stream);

/*
 * diverse_select in mode LAST_SEL_KCENTER, as two calls (Sec. 3.4): the
 * pairwise coverage distances of Eq. 10 depend only on the features, the
 * greedy of Eq. 9-11 also on the relevance scores. Splitting them lets a
 * caller compute the distances on a second stream while the scores of the
 * same batch are still being computed (Eq. 6-8), and join the streams before
 * the pick call. Together the two calls enqueue the same kernels as one
 * diverse_select call and give bit-identical kept, order and gains.
 *   ws         the diverse_select_similarity_workspace(R, cu_vis_h, Dv,
 *              fdtype) bytes, 256-byte aligned. The two calls always take the
 *              matrix form (the pick call has no features to fold rounds
 *              with). The similarity
 *              call writes the distances there; the pick call reads them, so
 *              both calls take the same workspace and the same R, Dv, fdtype
 *              and cu_vis (checked only for shape; distances of other
 *              features give a selection over those features).
 *   ordering   the pick call must run after the similarity call has
 *              finished (same stream, or an event the pick stream waits on),
 *              and no other call may reuse the workspace in between.
 * Arguments, errors and outputs are otherwise those of diverse_select; the
 * similarity call does not need the scores, the pick call not the features.
 */
size_t diverse_select_similarity_workspace(int32_t R, const int32_t *cu_vis_h,
                                           int32_t Dv, last_dtype fdtype);
last_status diverse_select_similarity(int32_t R, int32_t Dv, last_dtype fdtype,
                                      const void *feats, const int32_t *cu_vis,
                                      const int32_t *cu_vis_h, void *ws,
                                      size_t ws_bytes, void *stream);
last_status diverse_select_pick(int32_t R, int32_t Dv, last_dtype fdtype,
                                const float *scores, const int32_t *cu_vis,
                                const int32_t *cu_vis_h, const int32_t *cu_keep,
                                const int32_t *cu_keep_h, int32_t *kept,
                                int32_t *order, float *gains, void *ws,
                                size_t ws_bytes, void *stream);

/*
 * Sec. 3.4, Eq. 12: out[t] = feats[cu_vis[r] + kept[t]] for every kept slot
 * t of request r, copied byte for byte (row_bytes = Dv * elem_bytes).
 *   kept       [K_total] request-local indices (e.g. from diverse_select);
 *              an index outside [0, N_r) yields a zero-filled row
 *   out        [K_total][Dv] out, same element type as feats
 */
last_status gather_kept(int32_t R, int32_t Dv, size_t elem_bytes,
                        const void *feats, const int32_t *cu_vis,
                        const int32_t *cu_vis_h, const int32_t *kept,
                        const int32_t *cu_keep, const int32_t *cu_keep_h,
                        void *out, void *stream);

/* Workspace bytes last_connector needs for K rows: the normalised rows and
 * the hidden activations, bf16 (0 if the arguments are invalid). */
size_t last_connector_workspace(int64_t K, int32_t Dv, int32_t Dh);

/*
 * Sec. 3.4 after Eq. 12 (H_S = phi_c(X_S)) and Sec. 3.2: the cloud connector
 * applied token by token to the K rows the edge transmitted. The paper names
 * phi_c without a formula; this is the token-wise connector of the model
 * family it builds on:
 *   xhat = (x - mean(x)) / sqrt(var(x) + eps) * gamma + beta   (biased var)
 *   h    = GELU(W1 xhat + b1),  GELU(u) = u (1 + erf(u / sqrt 2)) / 2
 *   y    = W2 h + b2
 *   dtype      LAST_BF16 (others: LAST_ERR_UNSUPPORTED)
 *   K          rows, 0 <= K < 2^31 (0: nothing to do)
 *   x          [K][Dv] transmitted rows X_S (normally gather_kept's out)
 *   gamma,beta [Dv] fp32 LayerNorm scale and shift
 *   w1, b1     [Dh][Dv] (one hidden feature per row, dtype) and [Dh] fp32
 *   w2, b2     [Do][Dh] (one output feature per row, dtype) and [Do] fp32
 *   out        [K][Do] out, dtype (rounded to nearest even)
 *   eps        > 0 and finite (LAST_ERR_INVALID otherwise)
 * Dv and Dh must be multiples of 64 and Do of 4, each in [64, 65536], and
 * ceil(K / 256) ceil(max(Dh, Do) / 256) below 2^31 (LAST_ERR_UNSUPPORTED
 * otherwise). Every pointer must be 16-byte aligned (LAST_ERR_INVALID).
 * xhat and h are rounded to bf16 before the products, which accumulate in
 * fp32; GELU's erf is evaluated to within 1e-6 (1 + |u|). The workspace (256-byte aligned,
 * last_connector_workspace bytes) holds xhat and h; the caller owns every
 * buffer.
 */
last_status last_connector(last_dtype dtype, int64_t K, int32_t Dv, int32_t Dh, int32_t Do,
                           float eps, const void *x, const float *gamma, const float *beta,
                           const void *w1, const float *b1, const void *w2, const float *b2,
                           void *out, void *ws, size_t ws_bytes, void *stream);

/* Sec. 3.2, Eq. 2: K = ceil(N * rho_num / rho_den), integer-exact, clamped
 * to [1, N]; returns -1 for N < 1 or a ratio outside (0, 1]. */
int32_t last_budget(int32_t N, int32_t rho_num, int32_t rho_den);

/* Human-readable text for a status (static storage). For LAST_ERR_DEVICE it
 * includes the most recent HIP error message seen by this thread. */
const char *last_status_string(last_status s);

/* Library version, as major * 10000 + minor * 100 + patch. */
int32_t last_version(void);

/*
 * Optional per-kernel timing, for benchmarking. While enabled, every kernel
 * the library launches is bracketed by a pair of HIP events on its stream
 * (event creation happens on first use; no device memory is allocated).
 * After the caller has synchronised the streams, last_profile_collect()
 * folds the finished pairs into per-kernel totals, which
 * last_profile_kernel() reports. The totals are process-wide and guarded by a
 * lock; with timing off (the default) a launch only reads an atomic flag, so
 * the compute calls stay free of shared mutable state. Event pairs beyond the
 * internal pool of 8192 are not recorded. A name returned by
 * last_profile_kernel() stays valid until the process ends.
 */
last_status last_profile_enable(int32_t on);
last_status last_profile_collect(void);
void last_profile_reset(void);
int32_t last_profile_count(void);
/* i-th kernel's name, launch count and total milliseconds; returns 0 if
 * there is no such entry. */
int32_t last_profile_kernel(int32_t i, const char **name, int64_t *launches,
                            double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* LAST_H */
