/*
 * CPU oracle for receiver-conditioned KV selection (CacheBack's scoring layer).
 *
 * TEST INFRASTRUCTURE ONLY.  This library defines what the GPU path must
 * compute and exists to check it.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * Everything is plain, single-threaded C in double precision.  Inputs are
 * widened exactly (bf16 and fp32 are subsets of fp64).
 *
 * Layouts (row-major, contiguous):
 *   q          [L][Hq][m][D]           receiver query projections, per layer
 *   k, v       [S][L][Hkv][T][D]       sender caches, S senders
 *   importance [S][L][Hkv][T]          fp64
 *   row_lse    [S][L][Hq][m]           fp64, natural log (optional)
 *   idx        [S][L][Hkv][keep]       int32, strictly ascending per unit
 *   k_out,v_out[L][Hkv][S*keep][D]     senders concatenated in order
 * dtype: 0 = fp32, 1 = bf16 (raw 16-bit patterns).
 *
 * message.c adds the paper's position-level score, its budgets, its span
 * rule and the continuous-row gather (Appendix C):
 *   score, qscore, corr [S][T]          fp64, one row per sender
 *   selected positions  [count]         int32, ascending
 *   rows                [S][T][row_bytes], out [S][count][row_bytes]
 */
#ifndef CB_ORACLE_H
#define CB_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

int64_t cbo_keep_count(int64_t T, double keep_ratio);
int cbo_score(const void* q, const void* k, int dtype, int S, int L, int Hq,
              int Hkv, int D, int m, int64_t T, double scale,
              double* importance, double* row_lse);
int cbo_select(const double* importance, int64_t units, int64_t T,
               int64_t keep, int32_t* idx);
int cbo_select_f32(const float* importance, int64_t units, int64_t T,
                   int64_t keep, int32_t* idx);
int cbo_compact(const void* k, const void* v, const int32_t* idx, int dtype,
                int S, int L, int Hkv, int D, int64_t T, int64_t keep,
                void* k_out, void* v_out);

int cbo_position_score(const void* q, const void* k, int dtype, int S, int L, int Hq,
                       int Hkv, int D, int m, int64_t T, double scale, int pool_width,
                       double p, double alpha, double* score, double* qscore, double* corr);
int64_t cbo_budget_fanout(int64_t T, int64_t r);
int64_t cbo_budget_chain(int64_t T_old, int64_t T_new, int64_t r, int relative,
                         int64_t B_max);
int64_t cbo_select_spans(const float* score, int64_t T, int64_t budget,
                         int64_t n_latent, int width, int32_t* out);
int64_t cbo_select_spans_f64(const double* score, int64_t T, int64_t budget,
                             int64_t n_latent, int width, int32_t* out);
int cbo_gather_rows(const void* rows, int S, int64_t T, int64_t row_bytes,
                    const int32_t* idx, int64_t count, void* out);

#ifdef __cplusplus
}
#endif
#endif
