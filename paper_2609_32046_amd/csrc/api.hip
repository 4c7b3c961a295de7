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

#include "../../include/cacheback.h"
#include "kernels.h"

namespace {

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

bool plan_for(const cb_layout* lay, cb::ScorePlan* p) {
  return cb::make_score_plan(lay->layers, lay->q_heads, lay->kv_heads, lay->head_dim,
                             lay->q_len, lay->senders, lay->seq_len, lay->dtype, lay->scale, p);
}

int prepare_score(const void* q, const void* k, const cb_layout* lay, float* importance,
                  float* row_lse, void* ws, size_t ws_bytes, cb::ScorePlan* p,
                  cb::PersistArgs* a) {
  const int st = check_layout(lay);
  if (st != CB_OK) return st;
  if (!q || !k || !importance) return CB_ERR_NULL;
  if (!aligned16(q) || !aligned16(k) || !aligned16(importance) ||
      (row_lse && !aligned16(row_lse)))
    return CB_ERR_ALIGN;
  if (!plan_for(lay, p)) return CB_ERR_SHAPE;
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
  a->sync = reinterpret_cast<uint32_t*>(w + p->off_sync);
  a->T = p->T;
  a->L = p->L;
  a->Hq = p->Hq;
  a->Hkv = p->Hkv;
  a->G = p->G;
  a->m = p->m;
  a->R = p->R;
  a->S = p->S;
  a->chunks = p->chunks;
  a->row_groups = p->row_groups;
  a->units = p->units;
  a->c2 = p->c2;
  a->spin_limit = g_wait_limit.load(std::memory_order_relaxed);
  return CB_OK;
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
  if (cb::launch_select(importance, p.units, p.T, keep, idx, a.sync + cb::kSyncError, s) !=
      hipSuccess)
    return CB_ERR_HIP;
  return cb::launch_compact(k, v, idx, lay->senders, lay->layers, lay->kv_heads, p.T,
                            p.D * (p.dtype == CB_BF16 ? 2 : 4), keep, 0, p.units, k_out, v_out,
                            s) == hipSuccess
             ? CB_OK
             : CB_ERR_HIP;
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

uint32_t cb_set_wait_limit(uint32_t polls) {
  return g_wait_limit.exchange(polls, std::memory_order_relaxed);
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
