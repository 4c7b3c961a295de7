// C ABI of the receiver-conditioned KV selection path: argument validation,
// workspace carve-up and launches.  Declared in include/cacheback.h.
//
// cb_score enqueues one small kernel that clears the call's synchronisation
// words and one persistent kernel that runs both score passes of every unit
// from a device work queue (score.hip); more than 512 query rows per unit add
// a row-group sum.  cb_pipeline follows it with the select and gather
// kernels.  Everything runs on the caller's stream.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "../../include/cacheback.h"
#include "kernels.h"
#include "position.h"

// Workspace of cb_pipeline_noalloc: one copy per device, held until the
// process ends.  Host code never passes this name to a kernel or a copy: it
// is a host-side stand-in; the device address comes from hipGetSymbolAddress.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

int scratch_on_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return CB_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return CB_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CB_OK;
}

// Polls of a dependency wait before the kernel gives up on it (about a
// second; a wait normally ends within microseconds).  cb_set_wait_limit
// changes it for the calls that follow (tests of the timeout path).
constexpr uint32_t kSpinLimit = 1u << 21;
std::atomic<uint32_t> g_wait_limit{kSpinLimit};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_layout(const cb_layout* lay) {
  if (!lay) return CB_ERR_NULL;
  if (lay->dtype != CB_F32 && lay->dtype != CB_BF16) return CB_ERR_DTYPE;
  if (lay->layers < 1 || lay->q_heads < 1 || lay->kv_heads < 1 || lay->q_len < 1 ||
      lay->senders < 1 || lay->seq_len < 1)
    return CB_ERR_SHAPE;
  if (lay->q_heads % lay->kv_heads != 0) return CB_ERR_SHAPE;
  if (lay->head_dim != 64 && lay->head_dim != 128) return CB_ERR_SHAPE;
  if (lay->seq_len > cb::kMaxSeqLen) return CB_ERR_SHAPE;
  if (!(lay->scale >= 0.f) || !isfinite(lay->scale)) return CB_ERR_SHAPE;
  const int64_t units = (int64_t)lay->senders * lay->layers * lay->kv_heads;
  if (units > (1 << 30)) return CB_ERR_SHAPE;
  if ((int64_t)(lay->q_heads / lay->kv_heads) * lay->q_len > cb::kMaxRows) return CB_ERR_SHAPE;
  return CB_OK;
}

bool plan_for(const cb_layout* lay, cb::ScorePlan* p, bool position = false) {
  return cb::make_score_plan(lay->layers, lay->q_heads, lay->kv_heads, lay->head_dim,
                             lay->q_len, lay->senders, lay->seq_len, lay->dtype, lay->scale,
                             position, p);
}

int prepare_score(const void* q, const void* k, const cb_layout* lay, float* importance,
                  float* row_lse, void* ws, size_t ws_bytes, cb::ScorePlan* p,
                  cb::PersistArgs* a, bool position = false) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  if (!q || !k || !importance) return CB_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(importance) ||
      (row_lse && !aligned16(row_lse)))
    return CB_ERR_ALIGN;
  if (!plan_for(lay, p, position)) return CB_ERR_SHAPE;
  if (!ws || ws_bytes < p->total_bytes) return CB_ERR_WORKSPACE;
  if (!aligned16(ws)) return CB_ERR_ALIGN;
  unsigned char* w = static_cast<unsigned char*>(ws);
  *a = cb::PersistArgs{};
  a->q = q;
  a->k = k;
  a->importance = importance;
  a->row_lse = row_lse;
  a->partial = reinterpret_cast<float2*>(w + p->off_partial);
  a->imp_partial = reinterpret_cast<float*>(w + p->off_imp_partial);
  a->numer_partial = reinterpret_cast<float*>(w + p->off_numer_partial);
  a->sync = reinterpret_cast<uint32_t*>(w + p->off_sync);
  a->T = p->T;
  a->L = p->L;
  a->Hq = p->Hq;
  a->Hkv = p->Hkv;
  a->G = p->G;
  a->m = p->m;
  a->R = p->R;
  a->S = p->S;
  a->Gp = p->Gp;
  a->gshift = p->Gp == 8 ? 3 : 2;
  a->Rp = p->Rp;
  a->chunks = p->chunks;
  a->row_groups = p->row_groups;
  a->units = p->units;
  a->c2 = p->c2;
  a->spin_limit = g_wait_limit.load(std::memory_order_relaxed);
  return CB_OK;
}

// Workspace of cb_position_score: the score kernel's, then the per-unit
// numerator terms, then (when the caller passes no importance buffer) the
// importance, then the fp64 per-position layer sums and corrections.
struct PositionWs {
  cb::ScorePlan plan;
  size_t off_numer, off_importance, off_qpre, off_corr, total;
};

bool position_ws(const cb_layout* lay, PositionWs* pw) {
  if (check_layout(lay) != CB_OK || !plan_for(lay, &pw->plan, true)) return false;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t ut = (size_t)pw->plan.units * (size_t)pw->plan.T;
  const size_t st = (size_t)pw->plan.S * (size_t)pw->plan.T;
  size_t off = al(pw->plan.total_bytes);
  pw->off_numer = off; off = al(off + ut * sizeof(float));
  pw->off_importance = off; off = al(off + ut * sizeof(float));
  pw->off_qpre = off; off = al(off + st * sizeof(double));
  pw->off_corr = off; off = al(off + st * sizeof(double));
  pw->total = off;
  return true;
}

int64_t forced_count(int64_t T, int64_t n_latent) { return n_latent + 1 < T ? n_latent + 1 : T; }

// Workspace of cb_select_ws: an error word (and three spare words), the
// arrival counters of every unit, then the digit counts and part totals.
constexpr size_t kSelWsHeaderWords = 4;
size_t select_ws_data_offset(int64_t units) {
  const size_t b = (kSelWsHeaderWords + (size_t)units * cb::kSplitCounterWords) * sizeof(uint32_t);
  return (b + 255) & ~(size_t)255;
}

}  // namespace

extern "C" {

size_t cb_score_workspace_bytes(const cb_layout* lay) {
  if (check_layout(lay) != CB_OK) return 0;
  cb::ScorePlan p;
  if (!plan_for(lay, &p)) return 0;
  return p.total_bytes;
}

int cb_score(const void* q, const void* k, const cb_layout* lay, float* importance,
             float* row_lse, void* ws, size_t ws_bytes, void* stream) {
  cb::ScorePlan p;
  cb::PersistArgs a;
  const int st = prepare_score(q, k, lay, importance, row_lse, ws, ws_bytes, &p, &a);
  if (st != CB_OK) return st;
  return cb::launch_persistent(p, a, static_cast<hipStream_t>(stream)) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
}

int64_t cb_keep_count(int64_t T, double keep_ratio) {
  if (isnan(keep_ratio) || keep_ratio <= 0.0 || keep_ratio > 1.0) return CB_ERR_RATIO;
  if (T < 1) return CB_ERR_SHAPE;
  // ceil(x - tol): a product within four units in the last place of an
  // integer n gives n (rounding in ratio*T), otherwise ceil(x).
  const double x = keep_ratio * (double)T;
  const double tol = 4.0 * 2.220446049250313e-16 * fmax(1.0, x);
  int64_t keep = (int64_t)ceil(x - tol);
  if (keep < 1) keep = 1;
  if (keep > T) keep = T;
  return keep;
}

int cb_select(const float* importance, int64_t units, int64_t T, double keep_ratio,
              int32_t* idx, int64_t* k_out, void* stream) {
  if (!importance || !idx) return CB_ERR_NULL;
  if (units < 1 || T < 1 || T > cb::kMaxSeqLen || units > (1 << 30)) return CB_ERR_SHAPE;
  const int64_t keep = cb_keep_count(T, keep_ratio);
  if (keep < 0) return (int)keep;
  if (!aligned16(importance) || !aligned16(idx)) return CB_ERR_ALIGN;
  if (k_out) *k_out = keep;
  if (cb::launch_select(importance, units, T, keep, idx, nullptr,
                        static_cast<hipStream_t>(stream)) != hipSuccess)
    return CB_ERR_HIP;
  return CB_OK;
}

size_t cb_select_workspace_bytes(int64_t units, int64_t T) {
  if (units < 1 || T < 1 || T > cb::kMaxSeqLen || units > (1 << 30)) return 0;
  cb::SelectSplit sp;
  if (!cb::select_split_plan(units, T, &sp)) return 0;
  return select_ws_data_offset(units) + (size_t)units * sp.data_words_per_unit * sizeof(uint32_t);
}

int cb_select_ws(const float* importance, int64_t units, int64_t T, double keep_ratio,
                 int32_t* idx, int64_t* k_out, void* ws, size_t ws_bytes, void* stream) {
  if (!importance || !idx) return CB_ERR_NULL;
  if (units < 1 || T < 1 || T > cb::kMaxSeqLen || units > (1 << 30)) return CB_ERR_SHAPE;
  const int64_t keep = cb_keep_count(T, keep_ratio);
  if (keep < 0) return (int)keep;
  if (!aligned16(importance) || !aligned16(idx)) return CB_ERR_ALIGN;
  cb::SelectSplit sp;
  const bool split = cb::select_split_plan(units, T, &sp);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (split && ws) {
    if (ws_bytes < cb_select_workspace_bytes(units, T)) return CB_ERR_WORKSPACE;
    if (!aligned16(ws)) return CB_ERR_ALIGN;
  }
  if (k_out) *k_out = keep;
  if (split && ws) {
    // error word and arrival counters start at zero
    uint32_t* w = static_cast<uint32_t*>(ws);
    if (cb::launch_clear_words(w, (int64_t)(select_ws_data_offset(units) / sizeof(uint32_t)), s) !=
        hipSuccess)
      return CB_ERR_HIP;
    if (cb::select_split_fits(sp, units)) {
      uint32_t* data = reinterpret_cast<uint32_t*>(static_cast<unsigned char*>(ws) +
                                                   select_ws_data_offset(units));
      return cb::launch_select_split(importance, units, T, keep, idx, sp, w + kSelWsHeaderWords,
                                     data, w, g_wait_limit.load(std::memory_order_relaxed),
                                     s) == hipSuccess
                 ? CB_OK
                 : CB_ERR_HIP;
    }
  }
  return cb::launch_select(importance, units, T, keep, idx, nullptr, s) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
}

int cb_select_status(int64_t units, int64_t T, const void* ws, size_t ws_bytes, void* stream) {
  if (units < 1 || T < 1 || T > cb::kMaxSeqLen || units > (1 << 30)) return CB_ERR_SHAPE;
  const size_t need = cb_select_workspace_bytes(units, T);
  if (need == 0) return CB_OK;   // no split: no wait that could give up
  if (!ws || ws_bytes < need) return CB_ERR_WORKSPACE;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return CB_ERR_HIP;
  uint32_t word = 0;
  if (hipMemcpy(&word, ws, sizeof word, hipMemcpyDeviceToHost) != hipSuccess) return CB_ERR_HIP;
  return word != 0u ? CB_ERR_TIMEOUT : CB_OK;
}

int cb_compact(const void* k, const void* v, const int32_t* idx, const cb_layout* lay,
               int64_t keep, void* k_out, void* v_out, void* stream) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  if (!k || !v || !idx || !k_out || !v_out) return CB_ERR_NULL;
  if (keep < 1 || keep > lay->seq_len) return CB_ERR_SHAPE;
  if (!aligned16(k) || !aligned16(v) || !aligned16(idx) || !aligned16(k_out) ||
      !aligned16(v_out))
    return CB_ERR_ALIGN;
  const int row_bytes = lay->head_dim * (lay->dtype == CB_BF16 ? 2 : 4);
  const int64_t units = (int64_t)lay->senders * lay->layers * lay->kv_heads;
  if (cb::launch_compact(k, v, idx, lay->senders, lay->layers, lay->kv_heads, lay->seq_len,
                         row_bytes, keep, 0, units, k_out, v_out,
                         static_cast<hipStream_t>(stream)) != hipSuccess)
    return CB_ERR_HIP;
  return CB_OK;
}

int cb_pipeline(const void* q, const void* k, const void* v, const cb_layout* lay,
                double keep_ratio, float* importance, float* row_lse, int32_t* idx,
                void* k_out, void* v_out, void* ws, size_t ws_bytes, int64_t* keep_out,
                void* stream) {
  cb::ScorePlan p;
  cb::PersistArgs a;
  const int st = prepare_score(q, k, lay, importance, row_lse, ws, ws_bytes, &p, &a);
  if (st != CB_OK) return st;
  if (!v || !idx || !k_out || !v_out) return CB_ERR_NULL;
  const int64_t keep = cb_keep_count(lay->seq_len, keep_ratio);
  if (keep < 0) return (int)keep;
  if (!aligned16(v) || !aligned16(idx) || !aligned16(k_out) || !aligned16(v_out))
    return CB_ERR_ALIGN;
  if (keep_out) *keep_out = keep;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (cb::launch_persistent(p, a, s) != hipSuccess) return CB_ERR_HIP;
  hipError_t e;
  if (cb::select_split_fits(p.sel, p.units)) {
    uint32_t* data = reinterpret_cast<uint32_t*>(static_cast<unsigned char*>(ws) + p.off_sel_data);
    e = cb::launch_select_split(importance, p.units, p.T, keep, idx, p.sel,
                                a.sync + p.off_sel_counters, data, a.sync + cb::kSyncError,
                                a.spin_limit, s);
  } else {
    e = cb::launch_select(importance, p.units, p.T, keep, idx, a.sync + cb::kSyncError, s);
  }
  if (e != hipSuccess) return CB_ERR_HIP;
  return cb::launch_compact(k, v, idx, lay->senders, lay->layers, lay->kv_heads, p.T,
                            p.D * (p.dtype == CB_BF16 ? 2 : 4), keep, 0, p.units, k_out, v_out,
                            s) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
}

int cb_pipeline_noalloc(const void* q, const void* k, const void* v, const cb_layout* lay,
                        double keep_ratio, float* importance, float* row_lse, int32_t* idx,
                        void* k_out, void* v_out, int64_t* keep_out, void* stream) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  const size_t need = cb_score_workspace_bytes(lay);
  if (need == 0) return CB_ERR_SHAPE;
  if (need > kNoAllocScratchBytes) return CB_ERR_WORKSPACE;
  void* ws = nullptr;
  const int st2 = scratch_on_current_device(&ws);
  if (st2 != CB_OK) return st2;
  return cb_pipeline(q, k, v, lay, keep_ratio, importance, row_lse, idx, k_out, v_out, ws,
                     kNoAllocScratchBytes, keep_out, stream);
}

int cb_score_status(const cb_layout* lay, const void* ws, size_t ws_bytes, void* stream) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  cb::ScorePlan p;
  if (!plan_for(lay, &p)) return CB_ERR_SHAPE;
  if (!ws || ws_bytes < p.total_bytes) return CB_ERR_WORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipStreamSynchronize(s) != hipSuccess) return CB_ERR_HIP;
  uint32_t word = 0;
  const unsigned char* w = static_cast<const unsigned char*>(ws);
  if (hipMemcpy(&word, w + p.off_sync + cb::kSyncError * sizeof(uint32_t), sizeof word,
                hipMemcpyDeviceToHost) != hipSuccess)
    return CB_ERR_HIP;
  return word != 0u ? CB_ERR_TIMEOUT : CB_OK;
}

int cb_position_status(const cb_layout* lay, const void* ws, size_t ws_bytes, void* stream) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  PositionWs pw;
  if (!position_ws(lay, &pw)) return CB_ERR_SHAPE;
  if (!ws || ws_bytes < pw.total) return CB_ERR_WORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipStreamSynchronize(s) != hipSuccess) return CB_ERR_HIP;
  uint32_t word = 0;
  const unsigned char* w = static_cast<const unsigned char*>(ws);
  if (hipMemcpy(&word, w + pw.plan.off_sync + cb::kSyncError * sizeof(uint32_t), sizeof word,
                hipMemcpyDeviceToHost) != hipSuccess)
    return CB_ERR_HIP;
  return word != 0u ? CB_ERR_TIMEOUT : CB_OK;
}

uint32_t cb_set_wait_limit(uint32_t polls) {
  return g_wait_limit.exchange(polls, std::memory_order_relaxed);
}

size_t cb_position_workspace_bytes(const cb_layout* lay) {
  PositionWs pw;
  return position_ws(lay, &pw) ? pw.total : 0;
}

int cb_position_score(const void* q, const void* k, const cb_layout* lay, double p, double alpha,
                      float* score, float* qscore, float* corr, float* importance, void* ws,
                      size_t ws_bytes, void* stream) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  if (!score || !ws) return !score ? CB_ERR_NULL : CB_ERR_WORKSPACE;
  if (!(p > 1.0) || (!isinf(p) && p > 8.0) || !(alpha >= 0.0) || !isfinite(alpha))
    return CB_ERR_SHAPE;
  PositionWs pw;
  if (!position_ws(lay, &pw)) return CB_ERR_SHAPE;
  if (ws_bytes < pw.total) return CB_ERR_WORKSPACE;
  if (!aligned16(ws) || !aligned16(score) || (qscore && !aligned16(qscore)) ||
      (corr && !aligned16(corr)))
    return CB_ERR_ALIGN;
  unsigned char* w = static_cast<unsigned char*>(ws);
  float* imp = importance ? importance : reinterpret_cast<float*>(w + pw.off_importance);
  cb::ScorePlan plan;
  cb::PersistArgs a;
  const int st2 = prepare_score(q, k, lay, imp, nullptr, ws, ws_bytes, &plan, &a, true);
  if (st2 != CB_OK) return st2;
  const int G = plan.G, m = plan.m;
  a.numer = reinterpret_cast<float*>(w + pw.off_numer);
  double num_scale;
  if (isinf(p)) {
    a.pow_mode = cb::kPowMax;
    num_scale = 1.0 / G;   // the terms are G * Pool(b)
  } else if (p == 2.0) {
    a.pow_mode = cb::kPowSquare;
    a.sq_scale = 0x1p40f;   // (P * 2^40)^2 stays normal for P >= 2^-103
    num_scale = 0x1p-80 / ((double)G * G * m);
  } else {
    a.pow_mode = cb::kPowGeneral;
    // terms P^p * 2^kappa with P <= 8: sums of up to 2^8 of them stay below
    // 2^127
    const double kappa = floor(118.0 - 3.0 * p);
    a.pow_p = (float)p;
    a.pow_kappa = (float)kappa;
    num_scale = exp2(-kappa) / (pow((double)G, p) * m);
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (cb::launch_persistent(plan, a, s) != hipSuccess) return CB_ERR_HIP;
  cb::PositionFinish f;
  f.importance = imp;
  f.numer = a.numer;
  f.qpre = reinterpret_cast<double*>(w + pw.off_qpre);
  f.corr64 = reinterpret_cast<double*>(w + pw.off_corr);
  f.score = score;
  f.qscore = qscore;
  f.corr = corr;
  f.T = plan.T;
  f.S = plan.S;
  f.LH = plan.L * plan.Hkv;
  f.m = m;
  f.G = G;
  f.Hq = plan.Hq;
  f.pow_mode = a.pow_mode;
  f.p = p;
  f.alpha = alpha;
  f.num_scale = num_scale;
  return cb::launch_position_finish(f, s) == hipSuccess ? CB_OK : CB_ERR_HIP;
}

int64_t cb_budget_fanout(int64_t T, int64_t r) {
  if (T < 1 || r < 1) return CB_ERR_SHAPE;
  return (T + r - 1) / r;
}

int64_t cb_budget_chain(int64_t T_old, int64_t T_new, int64_t r, int relative, int64_t B_max) {
  if (T_old < 0 || T_new < 1 || r < 1) return CB_ERR_SHAPE;
  if (relative) return T_old + (T_new + r - 1) / r;
  if (B_max < 1) return CB_ERR_SHAPE;
  return B_max < T_old + T_new ? B_max : T_old + T_new;
}

size_t cb_spans_workspace_bytes(int64_t senders, int64_t T, int32_t width) {
  if (senders < 1 || T < 1 || T > cb::kMaxSeqLen || width < 1 || width > 64) return 0;
  return (((size_t)senders * (size_t)((T + width - 1) / width) * sizeof(uint64_t)) + 255) &
         ~(size_t)255;
}

int cb_select_spans(const float* score, int64_t senders, int64_t T, int64_t budget,
                    int64_t n_latent, int32_t width, int32_t* idx, int64_t* count_out, void* ws,
                    size_t ws_bytes, void* stream) {
  if (!score || !idx) return CB_ERR_NULL;
  if (senders < 1 || senders > (1 << 30) || T < 1 || T > cb::kMaxSeqLen || budget < 1 ||
      n_latent < 0 || width < 1 || width > 64)
    return CB_ERR_SHAPE;
  const int64_t nf = forced_count(T, n_latent);
  if (budget < nf) return CB_ERR_SHAPE;
  const size_t need = cb_spans_workspace_bytes(senders, T, width);
  if (!ws || ws_bytes < need) return CB_ERR_WORKSPACE;
  if (!aligned16(score) || !aligned16(idx) || !aligned16(ws)) return CB_ERR_ALIGN;
  const int64_t out_count = budget < T ? budget : T;
  if (count_out) *count_out = out_count;
  return cb::launch_spans(score, senders, T, width, n_latent, out_count - nf, out_count,
                          static_cast<uint64_t*>(ws), idx,
                          static_cast<hipStream_t>(stream)) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
}

int cb_gather_rows(const void* rows, int64_t senders, int64_t T, int64_t row_bytes,
                   const int32_t* idx, int64_t count, void* out, void* stream) {
  if (!rows || !idx || !out) return CB_ERR_NULL;
  if (senders < 1 || T < 1 || T > cb::kMaxSeqLen || count < 1 || row_bytes < 4 ||
      row_bytes % 4 != 0)
    return CB_ERR_SHAPE;
  const uintptr_t am = row_bytes % 16 == 0 ? 15u : 3u;
  if ((reinterpret_cast<uintptr_t>(rows) & am) || (reinterpret_cast<uintptr_t>(out) & am) ||
      (reinterpret_cast<uintptr_t>(idx) & 3u))
    return CB_ERR_ALIGN;
  return cb::launch_gather_rows(rows, senders, T, row_bytes, idx, count, out,
                                static_cast<hipStream_t>(stream)) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
}

const char* cb_status_string(int status) {
  switch (status) {
    case CB_OK: return "ok";
    case CB_ERR_NULL: return "a required pointer is NULL";
    case CB_ERR_SHAPE: return "invalid shape or layout";
    case CB_ERR_DTYPE: return "unsupported dtype";
    case CB_ERR_RATIO: return "keep_ratio must be in (0, 1]";
    case CB_ERR_WORKSPACE: return "workspace missing or too small";
    case CB_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case CB_ERR_HIP: return "HIP launch error";
    case CB_ERR_TIMEOUT: return "a dependency wait in the score kernel timed out";
    default: return "unknown status";
  }
}

}  // extern "C"
