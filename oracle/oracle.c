/*
 * CPU oracle for receiver-conditioned KV selection.  TEST INFRASTRUCTURE
 * ONLY: the test suite, the smoke check and the benchmark's CPU-baseline leg
 * are its only users.  Plain, slow, single-threaded, fp64.  Shares no code
 * with the HIP library.
 *
 * What it computes, for every unit (sender s, layer l, KV head g):
 *
 *   1. Attention from each receiver-query token r, in each query head h that
 *      reads KV head g, to each sender position t (paper, Appendix C.1,
 *      "Adapting SnapKV": the receiver query is appended after the sender's
 *      prefill and only the query tokens are run against the existing cache;
 *      a_{l,h,r,t} is the attention weight).  The softmax runs over the T
 *      sender positions with scale 1/sqrt(D).
 *   2. Importance I[s,l,g,t] = sum over the grouped heads h and query rows r
 *      of a_{l,h,r,t}.  This is the inner double sum of the mean-query-
 *      attention equation (Appendix C.1) restricted to one KV-head group,
 *      before the 1/(m|H_l|) factor, the layer sum and the 7-wide pooling.
 *   3. keep = ceil(ratio * T), the per-sender budget of the fan-out budget
 *      equation (Appendix C.2) with ratio = 1/r.
 *   4. The keep positions of highest importance, ties going to the earlier
 *      position, returned in source order (Appendix C.2: equal scores favour
 *      the earlier span; selected positions are returned in source order).
 *   5. The K and V rows at those positions, copied into a compact cache.
 */
#include "oracle.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

static double widen(const void* base, int dtype, size_t i) {
  if (dtype == 0) return (double)((const float*)base)[i];
  uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Budget: ceil(ratio*T), clamped to [1, T].  A product that lands within
 * four units in the last place of an integer is taken as that integer, so
 * that rounding in ratio*T (0.07*100 evaluates to 7.000000000000001) does not
 * add a position; a genuine fractional part larger than that still rounds up.
 * Returns -4 for a ratio outside (0, 1] or NaN, -2 for T < 1. */
int64_t cbo_keep_count(int64_t T, double keep_ratio) {
  if (!(keep_ratio > 0.0 && keep_ratio <= 1.0)) return -4;
  if (T < 1) return -2;
  double x = keep_ratio * (double)T;
  double nearest = floor(x + 0.5);
  double tol = 4.0 * DBL_EPSILON * (x > 1.0 ? x : 1.0);
  double c = (fabs(x - nearest) <= tol) ? nearest : ceil(x);
  int64_t keep = (int64_t)c;
  if (keep < 1) keep = 1;
  if (keep > T) keep = T;
  return keep;
}

int cbo_score(const void* q, const void* k, int dtype, int S, int L, int Hq,
              int Hkv, int D, int m, int64_t T, double scale,
              double* importance, double* row_lse) {
  if (!q || !k || !importance) return -1;
  if (S < 1 || L < 1 || Hq < 1 || Hkv < 1 || D < 1 || m < 1 || T < 1) return -2;
  if (Hq % Hkv != 0) return -2;
  if (dtype != 0 && dtype != 1) return -3;
  if (scale == 0.0) scale = 1.0 / sqrt((double)D);
  const int G = Hq / Hkv;
  double* logit = (double*)malloc(sizeof(double) * (size_t)T);
  if (!logit) return -7;

  for (int s = 0; s < S; ++s)
    for (int l = 0; l < L; ++l)
      for (int g = 0; g < Hkv; ++g) {
        size_t unit = ((size_t)s * L + l) * Hkv + g;
        double* imp = importance + unit * (size_t)T;
        size_t kbase = unit * (size_t)T * D;
        for (int64_t t = 0; t < T; ++t) imp[t] = 0.0;
        /* query head h reads KV head h / G (contiguous grouping) */
        for (int h = g * G; h < (g + 1) * G; ++h)
          for (int r = 0; r < m; ++r) {
            size_t qbase = (((size_t)l * Hq + h) * m + r) * D;
            for (int64_t t = 0; t < T; ++t) {
              double dot = 0.0;
              for (int d = 0; d < D; ++d)
                dot += widen(q, dtype, qbase + d) *
                       widen(k, dtype, kbase + (size_t)t * D + d);
              logit[t] = scale * dot;
            }
            double mx = logit[0];
            for (int64_t t = 1; t < T; ++t)
              if (logit[t] > mx) mx = logit[t];
            double z = 0.0;
            for (int64_t t = 0; t < T; ++t) z += exp(logit[t] - mx);
            for (int64_t t = 0; t < T; ++t) imp[t] += exp(logit[t] - mx) / z;
            if (row_lse)
              row_lse[(((size_t)s * L + l) * Hq + h) * m + r] = mx + log(z);
          }
      }
  free(logit);
  return 0;
}

/* ---- selection: a comparison sort with an explicit total order ---------- */

typedef struct {
  double key;
  int is_nan;
  int64_t index;
} entry;

/* Higher key first; NaN ranks below every number; equal keys (including
 * -0 == +0) go to the lower index. */
static int by_score_then_index(const void* pa, const void* pb) {
  const entry* a = (const entry*)pa;
  const entry* b = (const entry*)pb;
  if (a->is_nan != b->is_nan) return a->is_nan ? 1 : -1;
  if (!a->is_nan) {
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
  }
  return (a->index < b->index) ? -1 : (a->index > b->index);
}

static int ascending_i32(const void* pa, const void* pb) {
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  return (a > b) - (a < b);
}

static int select_rows(const void* imp, int is_f32, int64_t units, int64_t T,
                       int64_t keep, int32_t* idx) {
  if (!imp || !idx) return -1;
  if (units < 1 || T < 1 || keep < 1 || keep > T || T > 2147483647LL) return -2;
  entry* e = (entry*)malloc(sizeof(entry) * (size_t)T);
  if (!e) return -7;
  for (int64_t u = 0; u < units; ++u) {
    for (int64_t t = 0; t < T; ++t) {
      double v = is_f32 ? (double)((const float*)imp)[u * T + t]
                        : ((const double*)imp)[u * T + t];
      e[t].key = v;
      e[t].is_nan = isnan(v) ? 1 : 0;
      e[t].index = t;
    }
    qsort(e, (size_t)T, sizeof(entry), by_score_then_index);
    int32_t* out = idx + u * keep;
    for (int64_t j = 0; j < keep; ++j) out[j] = (int32_t)e[j].index;
    qsort(out, (size_t)keep, sizeof(int32_t), ascending_i32);
  }
  free(e);
  return 0;
}

int cbo_select(const double* importance, int64_t units, int64_t T,
               int64_t keep, int32_t* idx) {
  return select_rows(importance, 0, units, T, keep, idx);
}

int cbo_select_f32(const float* importance, int64_t units, int64_t T,
                   int64_t keep, int32_t* idx) {
  return select_rows(importance, 1, units, T, keep, idx);
}

/* ---- compaction: byte copies of the selected rows ----------------------- */

int cbo_compact(const void* k, const void* v, const int32_t* idx, int dtype,
                int S, int L, int Hkv, int D, int64_t T, int64_t keep,
                void* k_out, void* v_out) {
  if (!k || !v || !idx || !k_out || !v_out) return -1;
  if (S < 1 || L < 1 || Hkv < 1 || D < 1 || T < 1 || keep < 1 || keep > T)
    return -2;
  if (dtype != 0 && dtype != 1) return -3;
  const size_t row = (size_t)D * (dtype == 0 ? 4 : 2);
  for (int s = 0; s < S; ++s)
    for (int l = 0; l < L; ++l)
      for (int g = 0; g < Hkv; ++g) {
        size_t unit = ((size_t)s * L + l) * Hkv + g;
        for (int64_t j = 0; j < keep; ++j) {
          int64_t t = idx[unit * keep + j];
          if (t < 0 || t >= T) return -2;
          size_t src = (unit * (size_t)T + (size_t)t) * row;
          size_t dst = ((((size_t)l * Hkv + g) * S + s) * (size_t)keep + j) * row;
          memcpy((char*)k_out + dst, (const char*)k + src, row);
          memcpy((char*)v_out + dst, (const char*)v + src, row);
        }
      }
  return 0;
}
