/*
 * CPU oracle, part 2: the paper's position-level selector and message rule.
 * TEST INFRASTRUCTURE ONLY (test suite, smoke check, benchmark CPU baseline).
 * Plain, slow, single-threaded, fp64 unless a function says otherwise.
 * Shares no code with the HIP library.
 *
 * Appendix C.1 ("General scoring rule"):
 *   a[l,h,r,t]  attention from query token r in query head h of layer l to
 *               sender position t (softmax over the T sender positions,
 *               scale 1/sqrt(D)), as in oracle.c.
 *   Pool_w      local maximum over the w positions centred on t, clipped at
 *               the sequence ends (w = 7 in the paper).
 *   Q_t         mean-query-attention equation: Pool_w of the layer sum of the
 *               per-layer mean over query tokens and query heads.
 *   b[s,r,t]    mean over the query heads of KV-head group s (one group per
 *               layer and KV head) of a[l,h,r,t].
 *   C_{p,t}     CacheBack-correction equation: the ratio of
 *                 sum_s mean_r Pool_w(b[s,r,.])^p        (pool, power, mean)
 *               to
 *                 sum_s Pool_w(mean_r b[s,r,.])^p        (mean, pool, power)
 *               raised to 1/(p-1); 1 when both sums are zero.  At p = inf
 *               (Appendix D.2) the ratio of the largest pooled per-token
 *               value to the largest pooled mean.
 *   S_t         general-score equation (Appendix D.2): Q_t * C_{p,t}^alpha;
 *               CacheBack is p = alpha = 2, mean query attention alpha = 0.
 *
 * Appendix C.2 ("Budgets and position selection"): the fan-out budget
 * ceil(T/r), the chain budgets, and the span rule.  Appendix C.3 and section
 * 3.1.2 ("State Representation"): each selected position is sent as one
 * continuous row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static double widen2(const void* base, int dtype, size_t i) {
  if (dtype == 0) return (double)((const float*)base)[i];
  uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* out[t] = max of x over [t - (w-1)/2, t + (w-1)/2] clipped to [0, T). */
static void pool_max(const double* x, int64_t T, int w, double* out) {
  const int64_t half = (w - 1) / 2;
  for (int64_t t = 0; t < T; ++t) {
    int64_t lo = t - half < 0 ? 0 : t - half;
    int64_t hi = t + half > T - 1 ? T - 1 : t + half;
    double m = x[lo];
    for (int64_t j = lo + 1; j <= hi; ++j)
      if (x[j] > m) m = x[j];
    out[t] = m;
  }
}

/* a[r][t] for one (layer, query head) of one sender: softmax over t of
 * scale * q[l][h][r] . k[s][l][g][t]. */
static void attention_rows(const void* q, const void* k, int dtype, int L, int Hq, int Hkv,
                           int D, int m, int64_t T, double scale, int s, int l, int h, int g,
                           double* a /* [m][T] */) {
  (void)L;
  size_t kbase = ((((size_t)s * L + l) * Hkv + g) * (size_t)T) * D;
  for (int r = 0; r < m; ++r) {
    size_t qbase = (((size_t)l * Hq + h) * m + r) * D;
    double* row = a + (size_t)r * T;
    for (int64_t t = 0; t < T; ++t) {
      double dot = 0.0;
      for (int d = 0; d < D; ++d)
        dot += widen2(q, dtype, qbase + d) * widen2(k, dtype, kbase + (size_t)t * D + d);
      row[t] = scale * dot;
    }
    double mx = row[0];
    for (int64_t t = 1; t < T; ++t)
      if (row[t] > mx) mx = row[t];
    double z = 0.0;
    for (int64_t t = 0; t < T; ++t) z += exp(row[t] - mx);
    for (int64_t t = 0; t < T; ++t) row[t] = exp(row[t] - mx) / z;
  }
}

int cbo_position_score(const void* q, const void* k, int dtype, int S, int L, int Hq, int Hkv,
                       int D, int m, int64_t T, double scale, int pool_width, double p,
                       double alpha, double* score, double* qscore, double* corr) {
  if (!q || !k || !score) return -1;
  if (S < 1 || L < 1 || Hq < 1 || Hkv < 1 || D < 1 || m < 1 || T < 1) return -2;
  if (Hq % Hkv != 0 || pool_width < 1 || pool_width % 2 == 0) return -2;
  if (dtype != 0 && dtype != 1) return -3;
  if (!(p > 1.0) || !(alpha >= 0.0)) return -2;
  if (scale == 0.0) scale = 1.0 / sqrt((double)D);
  const int G = Hq / Hkv;
  const int p_inf = isinf(p);
  double* a = (double*)malloc(sizeof(double) * (size_t)m * T);
  double* b = (double*)malloc(sizeof(double) * (size_t)m * T);
  double* mean_b = (double*)malloc(sizeof(double) * (size_t)T);
  double* pooled = (double*)malloc(sizeof(double) * (size_t)T);
  double* q_pre = (double*)malloc(sizeof(double) * (size_t)T);
  double* num = (double*)malloc(sizeof(double) * (size_t)T);
  double* den = (double*)malloc(sizeof(double) * (size_t)T);
  double* qpool = (double*)malloc(sizeof(double) * (size_t)T);
  if (!a || !b || !mean_b || !pooled || !q_pre || !num || !den || !qpool) {
    free(a); free(b); free(mean_b); free(pooled); free(q_pre); free(num); free(den); free(qpool);
    return -7;
  }

  for (int s = 0; s < S; ++s) {
    for (int64_t t = 0; t < T; ++t) q_pre[t] = num[t] = den[t] = 0.0;
    for (int l = 0; l < L; ++l)
      for (int g = 0; g < Hkv; ++g) {
        /* b[r][t]: mean over the G query heads of KV-head group (l, g). */
        for (size_t i = 0; i < (size_t)m * T; ++i) b[i] = 0.0;
        for (int h = g * G; h < (g + 1) * G; ++h) {
          attention_rows(q, k, dtype, L, Hq, Hkv, D, m, T, scale, s, l, h, g, a);
          for (int r = 0; r < m; ++r)
            for (int64_t t = 0; t < T; ++t) {
              b[(size_t)r * T + t] += a[(size_t)r * T + t] / G;
              /* mean over query tokens and all Hq heads of layer l */
              q_pre[t] += a[(size_t)r * T + t] / ((double)m * Hq);
            }
        }
        /* numerator: pool over positions, raise to p, then mean over r */
        for (int r = 0; r < m; ++r) {
          pool_max(b + (size_t)r * T, T, pool_width, pooled);
          for (int64_t t = 0; t < T; ++t) {
            if (p_inf) {
              if (pooled[t] > num[t]) num[t] = pooled[t];
            } else {
              num[t] += pow(pooled[t], p) / m;
            }
          }
        }
        /* denominator: mean over r, then pool, then raise to p */
        for (int64_t t = 0; t < T; ++t) {
          double acc = 0.0;
          for (int r = 0; r < m; ++r) acc += b[(size_t)r * T + t];
          mean_b[t] = acc / m;
        }
        pool_max(mean_b, T, pool_width, pooled);
        for (int64_t t = 0; t < T; ++t) {
          if (p_inf) {
            if (pooled[t] > den[t]) den[t] = pooled[t];
          } else {
            den[t] += pow(pooled[t], p);
          }
        }
      }
    pool_max(q_pre, T, pool_width, qpool);
    for (int64_t t = 0; t < T; ++t) {
      double c;
      if (num[t] == 0.0 && den[t] == 0.0) {
        c = 1.0;
      } else if (p_inf) {
        c = num[t] / den[t];
      } else {
        c = pow(num[t] / den[t], 1.0 / (p - 1.0));
      }
      size_t o = (size_t)s * T + t;
      score[o] = qpool[t] * pow(c, alpha);
      if (qscore) qscore[o] = qpool[t];
      if (corr) corr[o] = c;
    }
  }
  free(a); free(b); free(mean_b); free(pooled); free(q_pre); free(num); free(den); free(qpool);
  return 0;
}

/* ---- budgets (Appendix C.2) --------------------------------------------- */

/* Fan-out budget equation: B = ceil(T / r) for an integer ratio r >= 1. */
int64_t cbo_budget_fanout(int64_t T, int64_t r) {
  if (T < 1 || r < 1) return -2;
  return (T + r - 1) / r;
}

/* Chain budgets: relative = T_old + ceil(T_new / r); fixed =
 * min(B_max, T_old + T_new). */
int64_t cbo_budget_chain(int64_t T_old, int64_t T_new, int64_t r, int relative, int64_t B_max) {
  if (T_old < 0 || T_new < 1 || r < 1) return -2;
  if (relative) return T_old + (T_new + r - 1) / r;
  if (B_max < 1) return -2;
  return B_max < T_old + T_new ? B_max : T_old + T_new;
}

/* ---- span selection (Appendix C.2) -------------------------------------- */

typedef struct {
  double key;
  int64_t span;
} span_entry;

/* Higher mean first; equal means favour the earlier span. */
static int by_mean_then_span(const void* pa, const void* pb) {
  const span_entry* a = (const span_entry*)pa;
  const span_entry* b = (const span_entry*)pb;
  if (a->key > b->key) return -1;
  if (a->key < b->key) return 1;
  return (a->span < b->span) ? -1 : (a->span > b->span);
}

/*
 * One sender's selection from scores s[0..T) (fp32, or fp64 for the _f64
 * entry point; both are widened to fp64 exactly):
 *   1. The first position and the last n_latent positions (the current
 *      latent steps) are kept; they count toward the budget.
 *   2. Position 0's score is replaced by the maximum score.
 *   3. Spans of `width` positions start at 0 (the last may be shorter); each
 *      is ranked by its mean score, equal means favouring the earlier span.
 *      A span's mean is the fp64 sum of its fp32 scores in position order
 *      divided by its length.
 *   4. Spans are visited in rank order and their unselected positions added
 *      while they fit.  The first span whose unselected positions would
 *      exceed what is left contributes only the unselected positions
 *      closest to its highest-scoring position (ties to the lower position),
 *      taken in the order p*, p*+1, p*-1, p*+2, p*-2, ... inside the span,
 *      until the budget is full.
 *   5. The selected positions are written in source order.
 * Requires n_forced <= budget, where n_forced = |{0} U [T-n_latent, T)|;
 * a budget above T keeps every position.  Writes min(budget, T) entries and
 * returns that count, or a negative status.
 */
static int64_t select_spans(const void* score, int is_f32, int64_t T, int64_t budget,
                            int64_t n_latent, int width, int32_t* out) {
  if (!score || !out) return -1;
  if (T < 1 || T > 2147483647LL || budget < 1 || n_latent < 0 || width < 1) return -2;
  if (budget > T) budget = T;
  if (n_latent > T) n_latent = T;
  unsigned char* sel = (unsigned char*)calloc((size_t)T, 1);
  double* s = (double*)malloc(sizeof(double) * (size_t)T);
  const int64_t nspan = (T + width - 1) / width;
  span_entry* spans = (span_entry*)malloc(sizeof(span_entry) * (size_t)nspan);
  if (!sel || !s || !spans) {
    free(sel); free(s); free(spans);
    return -7;
  }
  int64_t taken = 0;
  sel[0] = 1;
  taken = 1;
  for (int64_t t = T - n_latent; t < T; ++t)
    if (!sel[t]) {
      sel[t] = 1;
      ++taken;
    }
  if (taken > budget) {
    free(sel); free(s); free(spans);
    return -2;
  }
  for (int64_t t = 0; t < T; ++t)
    s[t] = is_f32 ? (double)((const float*)score)[t] : ((const double*)score)[t];
  double mx = s[0];
  for (int64_t t = 1; t < T; ++t)
    if (s[t] > mx) mx = s[t];
  s[0] = mx;
  for (int64_t j = 0; j < nspan; ++j) {
    int64_t lo = j * width, hi = lo + width < T ? lo + width : T;
    double sum = 0.0;
    for (int64_t t = lo; t < hi; ++t) sum += s[t];
    spans[j].key = sum / (double)(hi - lo);
    spans[j].span = j;
  }
  qsort(spans, (size_t)nspan, sizeof(span_entry), by_mean_then_span);
  for (int64_t i = 0; i < nspan && taken < budget; ++i) {
    int64_t lo = spans[i].span * width;
    int64_t hi = lo + width < T ? lo + width : T;
    int64_t fresh = 0;
    for (int64_t t = lo; t < hi; ++t) fresh += !sel[t];
    if (fresh <= budget - taken) {
      for (int64_t t = lo; t < hi; ++t)
        if (!sel[t]) {
          sel[t] = 1;
          ++taken;
        }
      continue;
    }
    /* the span does not fit: an interval around its top position */
    int64_t top = lo;
    for (int64_t t = lo + 1; t < hi; ++t)
      if (s[t] > s[top]) top = t;
    for (int64_t d = 0; taken < budget && d < width; ++d) {
      int64_t right = top + d, left = top - d;
      if (right < hi && !sel[right]) {
        sel[right] = 1;
        ++taken;
      }
      if (d > 0 && taken < budget && left >= lo && !sel[left]) {
        sel[left] = 1;
        ++taken;
      }
    }
  }
  int64_t n = 0;
  for (int64_t t = 0; t < T; ++t)
    if (sel[t]) out[n++] = (int32_t)t;
  free(sel); free(s); free(spans);
  return n;
}

int64_t cbo_select_spans(const float* score, int64_t T, int64_t budget, int64_t n_latent,
                         int width, int32_t* out) {
  return select_spans(score, 1, T, budget, n_latent, width, out);
}

int64_t cbo_select_spans_f64(const double* score, int64_t T, int64_t budget, int64_t n_latent,
                             int width, int32_t* out) {
  return select_spans(score, 0, T, budget, n_latent, width, out);
}

/* ---- continuous rows (Appendix C.3) ------------------------------------- */

/* out[s*count + j] = rows[s][idx[s*count + j]] (row_bytes bytes each). */
int cbo_gather_rows(const void* rows, int S, int64_t T, int64_t row_bytes, const int32_t* idx,
                    int64_t count, void* out) {
  if (!rows || !idx || !out) return -1;
  if (S < 1 || T < 1 || row_bytes < 1 || count < 0) return -2;
  for (int s = 0; s < S; ++s)
    for (int64_t j = 0; j < count; ++j) {
      int64_t t = idx[(size_t)s * count + j];
      if (t < 0 || t >= T) return -2;
      memcpy((char*)out + ((size_t)s * count + j) * row_bytes,
             (const char*)rows + ((size_t)s * T + t) * row_bytes, (size_t)row_bytes);
    }
  return 0;
}
