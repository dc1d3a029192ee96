/*
 * CPU oracle for the LAST token-selection path -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the slow, plain, obviously-correct reference that the HIP
 * library is checked against. Only the test-suite, the smoke check and the
 * benchmark's cpu_baseline leg may load it; the product path never does.
 * It shares no source, header, table or helper with the HIP library.
 *
 * Everything is computed in fp64. Inputs arrive in their storage formats
 * (IEEE fp32, or bf16 as raw 16-bit patterns) and are widened exactly:
 * bf16 -> fp64 is a 16-bit left shift into an fp32 pattern, then a
 * conversion, both exact.
 *
 * Paper passages followed (arXiv 2607.27952, Section 3 "Method"):
 *   - Sec. 3.3, Eq. 6: causal softmax attention A^(l,h) over the P-token
 *     prefill sequence; only the row of the last query position p* is needed,
 *     and that row sees every key of the prefix (causal masking removes
 *     nothing from the last row).
 *   - Sec. 3.3, Eq. 7: s_i = sum over layers and heads of A^(l,h)[p*, p_i].
 *   - Sec. 3.3, Eq. 8: w_i = s_i / sum_j s_j.
 *   - Sec. 3.4, features normalised to unit L2 norm; Eq. 9 j_1 = argmax w;
 *     Eq. 10 coverage distance delta_i = min over selected j of
 *     (1 - xbar_i . xbar_j); Eq. 11 j_t = argmax over unselected of
 *     w_i * delta_i; incremental delta updates, no N x N matrix.
 *   - Sec. 3.4, Eq. 12: kept indices restored to ascending order, rows of X
 *     gathered in that order.
 *   - Sec. 4.3, Table 5: the "Top-k" ablation keeps the K largest w.
 *   - Sec. 3.2, Eq. 2: K = ceil(rho * N).
 *   - Sec. 4.3, Table 4: other attention sources (first, middle or every
 *     query token instead of the last), each row causal.
 *   - Sec. 3.4 (after Eq. 12) and Sec. 3.2: the cloud's token-wise connector on the kept rows
 *     (a LayerNorm and a two-layer GELU MLP; a reading of the model family).
 *   - Sec. 3.3: the causal prefill attention of the guidance model itself
 *     (every query row, softmax-weighted sum of the values), whose last row
 *     is the one Eq. 7 reads.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - softmax scale sigma is an explicit argument (1/sqrt(Dh) when <= 0);
 *   - query head h reads KV head h / (Hq/Hkv) (grouped-query attention);
 *   - no per-head renormalisation over the visual span before Eq. 7;
 *   - every argmax breaks ties towards the lowest index;
 *   - each coverage term is clamped at 0 (1 - cos can round below 0);
 *   - a zero-norm feature normalises to the zero vector;
 *   - the cosine is evaluated as x_i.x_j / sqrt(|x_i|^2 |x_j|^2), so that
 *     bitwise-identical features are at coverage distance exactly 0;
 *   - the selection consumes the fp32 relevance scores it is given; one that
 *     is not > 0 (negative, NaN) counts as 0, and a NaN objective (+inf
 *     relevance times a coverage distance of 0) counts as 0. Eq. 8's scores
 *     are probabilities, so neither rule touches the paper's inputs.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_F32 0
#define ORC_BF16 1

static double orc_widen(const void *base, int64_t idx, int dtype) {
  if (dtype == ORC_BF16) {
    uint32_t bits = ((uint32_t)((const uint16_t *)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return (double)((const float *)base)[idx];
}

static void orc_set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Eq. 2: K = ceil(N * num / den), integer-exact. */
int64_t oracle_budget(int64_t n, int64_t num, int64_t den) {
  return (n * num + den - 1) / den;
}

/*
 * Eq. 6-8. For request r: P_r = cu_seqlens[r+1]-cu_seqlens[r] tokens, the
 * visual span is [vis_start[r], vis_start[r] + N_r) with
 * N_r = cu_vis[r+1]-cu_vis[r], and the last query token is position P_r-1.
 * q: [G][R][Hq][Dh] (last query token), k: [G][T_total][Hkv][Dh].
 * w_out: [N_total] normalised scores. rows_out (nullable): [G][Hq][T_total],
 * the full last-token attention rows.
 */
int oracle_scores(int R, int G, int Hq, int Hkv, int Dh, int qk_dtype,
                  double scale, const int32_t *cu_seqlens,
                  const int32_t *vis_start, const int32_t *cu_vis,
                  const void *q, const void *k, double *w_out,
                  double *rows_out, int nthreads) {
  if (R < 0 || G < 1 || Hq < 1 || Hkv < 1 || Dh < 1 || Hq % Hkv != 0)
    return 1;
  const int g = Hq / Hkv;
  const int64_t T_total = cu_seqlens[R];
  if (scale <= 0.0) scale = 1.0 / sqrt((double)Dh);
  orc_set_threads(nthreads);
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int r = 0; r < R; ++r) {
    const int64_t tok0 = cu_seqlens[r];
    const int64_t P = (int64_t)cu_seqlens[r + 1] - tok0;
    const int64_t v0 = vis_start[r];
    const int64_t N = (int64_t)cu_vis[r + 1] - cu_vis[r];
    double *logit = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    double *s = (double *)calloc((size_t)(N > 0 ? N : 1), sizeof(double));
    if (!logit || !s) {
      bad = 1;
      free(logit);
      free(s);
      continue;
    }
    for (int l = 0; l < G; ++l) {
      for (int h = 0; h < Hq; ++h) {
        const int kv = h / g;
        const int64_t qoff = (((int64_t)l * R + r) * Hq + h) * Dh;
        /* logits of the last query row against every key of the prefix */
        for (int64_t j = 0; j < P; ++j) {
          const int64_t koff = (((int64_t)l * T_total + tok0 + j) * Hkv + kv) * Dh;
          double acc = 0.0;
          for (int d = 0; d < Dh; ++d)
            acc += orc_widen(q, qoff + d, qk_dtype) * orc_widen(k, koff + d, qk_dtype);
          logit[j] = scale * acc;
        }
        /* softmax over the whole row (Eq. 6) */
        double m = -INFINITY;
        for (int64_t j = 0; j < P; ++j)
          if (logit[j] > m) m = logit[j];
        double Z = 0.0;
        for (int64_t j = 0; j < P; ++j) Z += exp(logit[j] - m);
        if (rows_out) {
          double *row = rows_out + ((int64_t)l * Hq + h) * T_total + tok0;
          for (int64_t j = 0; j < P; ++j) row[j] = exp(logit[j] - m) / Z;
        }
        /* visual columns summed over layers and heads (Eq. 7) */
        for (int64_t i = 0; i < N; ++i) s[i] += exp(logit[v0 + i] - m) / Z;
      }
    }
    /* normalisation over the visual tokens (Eq. 8) */
    double tot = 0.0;
    for (int64_t i = 0; i < N; ++i) tot += s[i];
    for (int64_t i = 0; i < N; ++i) w_out[cu_vis[r] + i] = s[i] / tot;
    free(logit);
    free(s);
  }
  return bad ? 2 : 0;
}

/*
 * Sec. 4.3, Table 4 (which attention rows supply the relevance). Eq. 7 with
 * its single row p* replaced by a set of query rows per request: request r
 * uses the rows at positions row_pos[cu_rows[r] .. cu_rows[r+1]), and their
 * attention over the visual tokens is summed over rows, layers and heads
 * ("All Mean" averages the rows; a common factor cancels in Eq. 8). Under the
 * causal mask of Eq. 6 the row at position p attends to keys 0..p only: its
 * softmax runs over those p + 1 keys, and visual tokens after p get nothing
 * from it. With one row at P_r - 1 per request this is oracle_scores.
 * q: [G][M_total][Hq][Dh] (the queries of those rows, M_total = cu_rows[R]),
 * k: [G][T_total][Hkv][Dh]. w_out: [N_total] normalised scores (Eq. 8);
 * s_out (nullable): [N_total] the sums s_i before normalisation.
 * Returns 1 for malformed arguments (a row outside [0, P_r)), 3 if a request's
 * rows see no visual token (Eq. 8 undefined).
 */
int oracle_rows_scores(int R, int G, int Hq, int Hkv, int Dh, int qk_dtype,
                       double scale, const int32_t *cu_seqlens,
                       const int32_t *vis_start, const int32_t *cu_vis,
                       const int32_t *cu_rows, const int32_t *row_pos,
                       const void *q, const void *k, double *w_out,
                       double *s_out, int nthreads) {
  if (R < 0 || G < 1 || Hq < 1 || Hkv < 1 || Dh < 1 || Hq % Hkv != 0)
    return 1;
  const int g = Hq / Hkv;
  const int64_t T_total = cu_seqlens[R];
  const int64_t M_total = cu_rows[R];
  if (scale <= 0.0) scale = 1.0 / sqrt((double)Dh);
  for (int r = 0; r < R; ++r)
    for (int64_t m = cu_rows[r]; m < cu_rows[r + 1]; ++m)
      if (row_pos[m] < 0 || row_pos[m] >= cu_seqlens[r + 1] - cu_seqlens[r]) return 1;
  orc_set_threads(nthreads);
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int r = 0; r < R; ++r) {
    const int64_t tok0 = cu_seqlens[r];
    const int64_t P = (int64_t)cu_seqlens[r + 1] - tok0;
    const int64_t v0 = vis_start[r];
    const int64_t N = (int64_t)cu_vis[r + 1] - cu_vis[r];
    double *logit = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    double *s = (double *)calloc((size_t)(N > 0 ? N : 1), sizeof(double));
    /* one layer's keys of one KV head, and one query row, widened to fp64 */
    double *kx = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1) * (size_t)Dh);
    double *qx = (double *)malloc(sizeof(double) * (size_t)Dh);
    if (!logit || !s || !kx || !qx) {
      bad |= 2;
      free(logit);
      free(s);
      free(kx);
      free(qx);
      continue;
    }
    for (int l = 0; l < G; ++l) {
      for (int h = 0; h < Hq; ++h) {
        const int kv = h / g;
        if (h % g == 0)
          for (int64_t j = 0; j < P; ++j)
            for (int d = 0; d < Dh; ++d)
              kx[j * Dh + d] = orc_widen(k, (((int64_t)l * T_total + tok0 + j) * Hkv + kv) * Dh + d, qk_dtype);
        for (int64_t m = cu_rows[r]; m < cu_rows[r + 1]; ++m) {
          const int64_t p = row_pos[m];
          const int64_t qoff = (((int64_t)l * M_total + m) * Hq + h) * Dh;
          for (int d = 0; d < Dh; ++d) qx[d] = orc_widen(q, qoff + d, qk_dtype);
          /* the row sees keys 0..p (causal mask, Eq. 6) */
          for (int64_t j = 0; j <= p; ++j) {
            double acc = 0.0;
            for (int d = 0; d < Dh; ++d) acc += qx[d] * kx[j * Dh + d];
            logit[j] = scale * acc;
          }
          double mx = -INFINITY;
          for (int64_t j = 0; j <= p; ++j)
            if (logit[j] > mx) mx = logit[j];
          double Z = 0.0;
          for (int64_t j = 0; j <= p; ++j) Z += exp(logit[j] - mx);
          /* visual columns the row can see, summed over rows, layers, heads */
          for (int64_t i = 0; i < N && v0 + i <= p; ++i) s[i] += exp(logit[v0 + i] - mx) / Z;
        }
      }
    }
    double tot = 0.0;
    for (int64_t i = 0; i < N; ++i) tot += s[i];
    if (!(tot > 0.0)) bad |= 1;
    for (int64_t i = 0; i < N; ++i) {
      w_out[cu_vis[r] + i] = tot > 0.0 ? s[i] / tot : 0.0;
      if (s_out) s_out[cu_vis[r] + i] = s[i];
    }
    free(logit);
    free(s);
    free(kx);
    free(qx);
  }
  return (bad & 2) ? 2 : (bad & 1) ? 3 : 0;
}

/*
 * Sec. 3.3, Eq. 6: the causal self-attention of the guidance model's prefill,
 * whose attention tensors LAST reads (Sec. 3.3 reads row p* of A from the
 * same prefill pass). For every request, layer, query head h and position p:
 *   a_j = softmax_j(sigma q_p . k_j) over j = 0..p (causal mask),
 *   out_p = sum_j a_j v_j.
 * q: [G][T_total][Hq][Dh] (every position), k and v: [G][T_total][Hkv][Dh];
 * out: [G][T_total][Hq][Dh] in fp64. Query head h reads KV head h / (Hq/Hkv).
 */
int oracle_prefill(int R, int G, int Hq, int Hkv, int Dh, int qk_dtype,
                   double scale, const int32_t *cu_seqlens, const void *q,
                   const void *k, const void *v, double *out, int nthreads) {
  if (R < 0 || G < 1 || Hq < 1 || Hkv < 1 || Dh < 1 || Hq % Hkv != 0)
    return 1;
  const int g = Hq / Hkv;
  const int64_t T_total = cu_seqlens[R];
  if (scale <= 0.0) scale = 1.0 / sqrt((double)Dh);
  orc_set_threads(nthreads);
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
  for (int r = 0; r < R; ++r) {
    const int64_t tok0 = cu_seqlens[r];
    const int64_t P = (int64_t)cu_seqlens[r + 1] - tok0;
    double *logit = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1));
    double *kx = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1) * (size_t)Dh);
    double *vx = (double *)malloc(sizeof(double) * (size_t)(P > 0 ? P : 1) * (size_t)Dh);
    double *qx = (double *)malloc(sizeof(double) * (size_t)Dh);
    if (!logit || !kx || !vx || !qx) {
      bad = 1;
      free(logit);
      free(kx);
      free(vx);
      free(qx);
      continue;
    }
    for (int l = 0; l < G; ++l) {
      for (int h = 0; h < Hq; ++h) {
        const int kv = h / g;
        if (h % g == 0)
          for (int64_t j = 0; j < P; ++j)
            for (int d = 0; d < Dh; ++d) {
              const int64_t off = (((int64_t)l * T_total + tok0 + j) * Hkv + kv) * Dh + d;
              kx[j * Dh + d] = orc_widen(k, off, qk_dtype);
              vx[j * Dh + d] = orc_widen(v, off, qk_dtype);
            }
        for (int64_t p = 0; p < P; ++p) {
          const int64_t qoff = (((int64_t)l * T_total + tok0 + p) * Hq + h) * Dh;
          for (int d = 0; d < Dh; ++d) qx[d] = orc_widen(q, qoff + d, qk_dtype);
          /* row p sees keys 0..seen (causal mask: seen = p) */
          const int64_t seen = p;
          double rmax = -INFINITY;
          for (int64_t j = 0; j <= seen; ++j) {
            double acc = 0.0;
            for (int d = 0; d < Dh; ++d) acc += qx[d] * kx[j * Dh + d];
            logit[j] = scale * acc;
            if (logit[j] > rmax) rmax = logit[j];
          }
          double rsum = 0.0;
          for (int64_t j = 0; j <= seen; ++j) rsum += exp(logit[j] - rmax);
          double *o = out + qoff;
          for (int d = 0; d < Dh; ++d) o[d] = 0.0;
          for (int64_t j = 0; j <= seen; ++j) {
            const double a = exp(logit[j] - rmax) / rsum;
            for (int d = 0; d < Dh; ++d) o[d] += a * vx[j * Dh + d];
          }
        }
      }
    }
    free(logit);
    free(kx);
    free(vx);
    free(qx);
  }
  return bad ? 2 : 0;
}

/*
 * Sec. 3.4 (after Eq. 12), Sec. 3.2: the cloud applies its token-wise connector to the
 * transmitted rows, H_S = phi_c(X_S). Reading (the paper gives no formula;
 * this is the token-wise connector structure of the InternVL models it uses):
 *   xhat = (x - mean(x)) / sqrt(var(x) + eps) * gamma + beta     (LayerNorm)
 *   h    = W1 xhat + b1,   g = GELU(h) = h/2 (1 + erf(h / sqrt 2)),
 *   y    = W2 g + b2
 * for every row x of X_S. x: [K][Dv] (bf16 bits or fp32), W1: [Dh][Dv],
 * W2: [Do][Dh] (same storage type, one output feature per row); gamma, beta
 * [Dv], b1 [Dh], b2 [Do] fp32. y_out [K][Do]; xhat_out [K][Dv] and h_out
 * [K][Dh] (nullable) return the intermediate values. All in fp64.
 */
int oracle_connector(int64_t K, int Dv, int Dh, int Do, int dtype, double eps,
                     const void *x, const float *gamma, const float *beta,
                     const void *w1, const float *b1, const void *w2,
                     const float *b2, double *y_out, double *xhat_out,
                     double *h_out, int nthreads) {
  if (K < 0 || Dv < 1 || Dh < 1 || Do < 1) return 1;
  orc_set_threads(nthreads);
  int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
  for (int64_t t = 0; t < K; ++t) {
    double *xh = (double *)malloc(sizeof(double) * (size_t)Dv);
    double *g = (double *)malloc(sizeof(double) * (size_t)Dh);
    if (!xh || !g) {
      bad = 1;
      free(xh);
      free(g);
      continue;
    }
    double mean = 0.0;
    for (int d = 0; d < Dv; ++d) mean += orc_widen(x, t * Dv + d, dtype);
    mean /= Dv;
    double var = 0.0;
    for (int d = 0; d < Dv; ++d) {
      const double c = orc_widen(x, t * Dv + d, dtype) - mean;
      var += c * c;
    }
    var /= Dv;
    const double rstd = 1.0 / sqrt(var + eps);
    for (int d = 0; d < Dv; ++d)
      xh[d] = (orc_widen(x, t * Dv + d, dtype) - mean) * rstd * gamma[d] + beta[d];
    for (int j = 0; j < Dh; ++j) {
      double acc = b1[j];
      for (int d = 0; d < Dv; ++d) acc += orc_widen(w1, (int64_t)j * Dv + d, dtype) * xh[d];
      if (h_out) h_out[t * Dh + j] = acc;
      g[j] = 0.5 * acc * (1.0 + erf(acc / sqrt(2.0)));
    }
    for (int o = 0; o < Do; ++o) {
      double acc = b2[o];
      for (int j = 0; j < Dh; ++j) acc += orc_widen(w2, (int64_t)o * Dh + j, dtype) * g[j];
      y_out[t * Do + o] = acc;
    }
    if (xhat_out)
      for (int d = 0; d < Dv; ++d) xhat_out[t * Dv + d] = xh[d];
    free(xh);
    free(g);
  }
  return bad ? 2 : 0;
}

/*
 * Sec. 4.3, Table 4: the attention sources compared there, for a text query
 * of M = qe - qb tokens q_1 .. q_M at positions qb .. qe - 1 (q_M is the last
 * query token p*). Writes the positions of the source's rows to pos and
 * returns how many: 0 Last -> q_M; 1 First -> q_1; 2 Middle -> q_ceil(M/2);
 * 3 All Mean -> q_1 .. q_M. Returns -1 for an empty query or an unknown source.
 */
int oracle_source_rows(int src, int32_t qb, int32_t qe, int32_t *pos) {
  const int32_t M = qe - qb;
  if (M < 1 || qb < 0) return -1;
  switch (src) {
    case 0: pos[0] = qb + M - 1; return 1;
    case 1: pos[0] = qb; return 1;
    case 2: pos[0] = qb + (M + 1) / 2 - 1; return 1;
    case 3:
      for (int32_t m = 0; m < M; ++m) pos[m] = qb + m;
      return M;
    default: return -1;
  }
}

/*
 * One request's features widened to fp64, plus squared norms (Sec. 3.4).
 * The cosine of Eq. 10 is evaluated as x_i.x_j / sqrt(|x_i|^2 |x_j|^2),
 * which equals xbar_i.xbar_j and gives exactly 1 for bitwise-identical rows;
 * a zero-norm row has cosine 0 with everything (its unit vector is taken as 0).
 */
typedef struct {
  double *x;  /* [N][Dv] */
  double *nn; /* [N] squared norms */
  int Dv;
} orc_feats;

static int orc_load_feats(orc_feats *f, const void *feats, int64_t row0,
                          int64_t N, int Dv, int f_dtype) {
  const size_t n = (size_t)(N > 0 ? N : 1);
  f->Dv = Dv;
  f->x = (double *)malloc(sizeof(double) * n * (size_t)Dv);
  f->nn = (double *)malloc(sizeof(double) * n);
  if (!f->x || !f->nn) {
    free(f->x);
    free(f->nn);
    return 1;
  }
  for (int64_t i = 0; i < N; ++i) {
    double *xi = f->x + i * Dv;
    double ss = 0.0;
    for (int d = 0; d < Dv; ++d) {
      xi[d] = orc_widen(feats, (row0 + i) * Dv + d, f_dtype);
      ss += xi[d] * xi[d];
    }
    f->nn[i] = ss;
  }
  return 0;
}

static void orc_free_feats(orc_feats *f) {
  free(f->x);
  free(f->nn);
}

/* Coverage term of Eq. 10 for one pair, clamped at zero. */
static double orc_cover(const orc_feats *f, int64_t i, int64_t j) {
  if (f->nn[i] <= 0.0 || f->nn[j] <= 0.0) return 1.0;
  const double *xi = f->x + i * f->Dv, *xj = f->x + j * f->Dv;
  double dot = 0.0;
  for (int d = 0; d < f->Dv; ++d) dot += xi[d] * xj[d];
  const double t = 1.0 - dot / sqrt(f->nn[i] * f->nn[j]);
  return t > 0.0 ? t : 0.0;
}

/*
 * Eq. 8 makes the relevance a probability, finite and >= 0; on such inputs the
 * two helpers below are the identity. Relevance from elsewhere is read as
 * follows: a value that is not > 0 (negative, NaN) counts as 0, and an
 * objective w * delta that is NaN (+inf relevance on a covered token, delta = 0)
 * counts as 0.
 */
static double orc_rel(float w) { return (double)w > 0.0 ? (double)w : 0.0; }
static double orc_obj(double v) { return v == v ? v : 0.0; }

/* Lowest index attaining the maximum of o over unselected i. */
static int64_t orc_argmax(const double *o, const unsigned char *sel, int64_t N) {
  int64_t best = -1;
  for (int64_t i = 0; i < N; ++i) {
    if (sel[i]) continue;
    if (best < 0 || o[i] > o[best]) best = i;
  }
  return best;
}

static int orc_cmp_i32(const void *a, const void *b) {
  const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* Top-k ordering: larger score first, then lower index (Table 5 ablation). */
static const float *orc_sort_keys;
static int orc_cmp_topk(const void *a, const void *b) {
  const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  const double wx = orc_rel(orc_sort_keys[x]), wy = orc_rel(orc_sort_keys[y]);
  if (wx > wy) return -1;
  if (wx < wy) return 1;
  return (x > y) - (x < y);
}

/*
 * Eq. 9-12 (mode 0, importance-weighted greedy k-center) or the Table 5
 * Top-k ablation (mode 1). w: [N_total] fp32 relevance scores; feats:
 * [N_total][Dv]; K_r = cu_keep[r+1]-cu_keep[r], 1 <= K_r <= N_r.
 * Outputs (request-local indices): kept [K_total] ascending, order [K_total]
 * pick sequence, gains [K_total] objective value at each pick (w at t = 1).
 */
int oracle_select(int R, int Dv, int f_dtype, int mode, const float *w,
                  const void *feats, const int32_t *cu_vis,
                  const int32_t *cu_keep, int32_t *kept, int32_t *order,
                  double *gains, int nthreads) {
  orc_set_threads(nthreads);
  for (int r = 0; r < R; ++r) {
    const int64_t row0 = cu_vis[r];
    const int64_t N = (int64_t)cu_vis[r + 1] - row0;
    const int64_t K = (int64_t)cu_keep[r + 1] - cu_keep[r];
    const int64_t out0 = cu_keep[r];
    if (K < 1 || K > N) return 1;
    if (mode == 1) {
      int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
      if (!idx) return 2;
      for (int64_t i = 0; i < N; ++i) idx[i] = (int32_t)i;
      orc_sort_keys = w + row0;
      qsort(idx, (size_t)N, sizeof(int32_t), orc_cmp_topk);
      for (int64_t t = 0; t < K; ++t) {
        order[out0 + t] = idx[t];
        gains[out0 + t] = orc_rel(w[row0 + idx[t]]);
        kept[out0 + t] = idx[t];
      }
      qsort(kept + out0, (size_t)K, sizeof(int32_t), orc_cmp_i32);
      free(idx);
      continue;
    }
    orc_feats xf;
    if (orc_load_feats(&xf, feats, row0, N, Dv, f_dtype)) return 2;
    double *delta = (double *)malloc(sizeof(double) * (size_t)N);
    double *o = (double *)malloc(sizeof(double) * (size_t)N);
    unsigned char *sel = (unsigned char *)calloc((size_t)N, 1);
    if (!delta || !o || !sel) {
      orc_free_feats(&xf); free(delta); free(o); free(sel);
      return 2;
    }
    /* Eq. 9: start from the most relevant token */
    for (int64_t i = 0; i < N; ++i) o[i] = orc_rel(w[row0 + i]);
    int64_t j = orc_argmax(o, sel, N);
    if (j < 0) {
      orc_free_feats(&xf); free(delta); free(o); free(sel);
      return 1;
    }
    sel[j] = 1;
    order[out0] = (int32_t)j;
    gains[out0] = o[j];
    for (int64_t i = 0; i < N; ++i) delta[i] = INFINITY;
    for (int64_t t = 1; t < K; ++t) {
      /* Eq. 10, incremental: fold in the distance to the newest pick */
#pragma omp parallel for schedule(static)
      for (int64_t i = 0; i < N; ++i) {
        const double c = orc_cover(&xf, i, j);
        if (c < delta[i]) delta[i] = c;
        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);
      }
      /* Eq. 11 */
      j = orc_argmax(o, sel, N);
      if (j < 0) break;
      sel[j] = 1;
      order[out0 + t] = (int32_t)j;
      gains[out0 + t] = o[j];
    }
    /* Eq. 12: original order */
    int64_t c = 0;
    for (int64_t i = 0; i < N; ++i)
      if (sel[i]) kept[out0 + c++] = (int32_t)i;
    orc_free_feats(&xf); free(delta); free(o); free(sel);
  }
  return 0;
}

/*
 * Teacher-forced replay of a candidate pick sequence `picks` (request-local,
 * [K_total]) under the greedy rule of Eq. 9-11. At step t the oracle takes
 * the candidate's own prefix as the selected set, computes every objective
 * o_i in fp64 and its maximum o*, then classifies the candidate's pick g_t:
 *   0 exact   -- g_t is the lowest index attaining o*;
 *   1 excused -- o* - o_{g_t} <= rel_tol * o* (a near-tie);
 *   2 failed  -- anything else, including an out-of-range or repeated index.
 * margin[t] receives (o* - o_{g_t}) / o* (0 when o* == 0), and objective[t]
 * (nullable) the oracle's own objective o_{g_t} of the candidate's pick. After
 * a failed index that cannot be replayed (out of range / repeated) the
 * remaining steps of that request are marked failed.
 */
int oracle_replay(int R, int Dv, int f_dtype, const float *w,
                  const void *feats, const int32_t *cu_vis,
                  const int32_t *cu_keep, const int32_t *picks,
                  double rel_tol, int32_t *status, double *margin,
                  double *objective, int nthreads) {
  orc_set_threads(nthreads);
  for (int r = 0; r < R; ++r) {
    const int64_t row0 = cu_vis[r];
    const int64_t N = (int64_t)cu_vis[r + 1] - row0;
    const int64_t K = (int64_t)cu_keep[r + 1] - cu_keep[r];
    const int64_t out0 = cu_keep[r];
    orc_feats xf;
    if (orc_load_feats(&xf, feats, row0, N, Dv, f_dtype)) return 2;
    double *delta = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    double *o = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
    unsigned char *sel = (unsigned char *)calloc((size_t)(N > 0 ? N : 1), 1);
    if (!delta || !o || !sel) {
      orc_free_feats(&xf); free(delta); free(o); free(sel);
      return 2;
    }
    for (int64_t i = 0; i < N; ++i) {
      delta[i] = INFINITY;
      o[i] = orc_rel(w[row0 + i]);
    }
    int broken = 0;
    for (int64_t t = 0; t < K; ++t) {
      if (broken) {
        status[out0 + t] = 2;
        margin[out0 + t] = INFINITY;
        if (objective) objective[out0 + t] = NAN;
        continue;
      }
      const int64_t best = orc_argmax(o, sel, N);
      const int64_t gp = picks[out0 + t];
      if (gp < 0 || gp >= N || sel[gp]) {
        status[out0 + t] = 2;
        margin[out0 + t] = INFINITY;
        if (objective) objective[out0 + t] = NAN;
        broken = 1;
        continue;
      }
      if (objective) objective[out0 + t] = o[gp];
      const double ostar = o[best];
      const double gap = ostar - o[gp];
      margin[out0 + t] = ostar > 0.0 ? gap / ostar : 0.0;
      if (gp == best)
        status[out0 + t] = 0;
      else if (gap <= rel_tol * ostar)
        status[out0 + t] = 1;
      else
        status[out0 + t] = 2;
      sel[gp] = 1;
#pragma omp parallel for schedule(static)
      for (int64_t i = 0; i < N; ++i) {
        const double c = orc_cover(&xf, i, gp);
        if (c < delta[i]) delta[i] = c;
        o[i] = orc_obj(orc_rel(w[row0 + i]) * delta[i]);
      }
    }
    orc_free_feats(&xf); free(delta); free(o); free(sel);
  }
  return 0;
}

/* Eq. 12: byte copy of the kept rows, request by request. */
int oracle_gather(int R, int64_t row_bytes, const void *feats,
                  const int32_t *cu_vis, const int32_t *kept,
                  const int32_t *cu_keep, void *out) {
  const unsigned char *src = (const unsigned char *)feats;
  unsigned char *dst = (unsigned char *)out;
  for (int r = 0; r < R; ++r) {
    for (int64_t t = cu_keep[r]; t < cu_keep[r + 1]; ++t) {
      const int64_t row = (int64_t)cu_vis[r] + kept[t];
      memcpy(dst + t * row_bytes, src + row * row_bytes, (size_t)row_bytes);
    }
  }
  return 0;
}
