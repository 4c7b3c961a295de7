// Host side of the persistent score kernel: the work list, the plan and
// workspace carve-up of one call, and the dispatch to the per-dtype launch
// instantiations (score_impl.h, score_*.hip).
#include <math.h>

#include <algorithm>

#include "kernels.h"

namespace cb {

void make_work_list(int units, int nstages, const int* per_unit, int resident, WorkList* wl) {
  *wl = WorkList{};
  wl->nstages = nstages;
  wl->units = units;
  for (int s = 0; s < nstages; ++s) {
    wl->per_unit[s] = per_unit[s];
  }
  // P2 trails P1 by enough steps that about 1.5 x the resident workgroups'
  // worth of P1 items is taken in between (one P1 item time, so that the
  // statistics are normally complete when a P2 item is taken), but never by
  // more than the number of units (so no step is empty).
  wl->lag[0] = 0;
  for (int s = 1; s < nstages; ++s) {
    int64_t gap = (3LL * resident + 2LL * wl->per_unit[s - 1] - 1) / (2LL * wl->per_unit[s - 1]);
    if (gap < 1) gap = 1;
    if (gap > units) gap = units;
    wl->lag[s] = wl->lag[s - 1] + (int)gap;
  }
  // Segment boundaries: where some stage starts or ends.
  int b[2 * kMaxStages];
  int nb = 0;
  for (int s = 0; s < nstages; ++s) {
    b[nb++] = wl->lag[s];
    b[nb++] = wl->lag[s] + units;
  }
  std::sort(b, b + nb);
  nb = (int)(std::unique(b, b + nb) - b);
  int64_t item = 0;
  wl->nseg = 0;
  for (int i = 0; i + 1 < nb; ++i) {
    int size = 0;
    for (int s = 0; s < nstages; ++s)
      if (wl->lag[s] <= b[i] && b[i] < wl->lag[s] + units) size += wl->per_unit[s];
    if (size == 0) continue;
    wl->seg_step[wl->nseg] = b[i];
    wl->seg_size[wl->nseg] = size;
    wl->seg_item[wl->nseg] = item;
    ++wl->nseg;
    item += (int64_t)size * (b[i + 1] - b[i]);
  }
  wl->items = item;
}

bool make_score_plan(int L, int Hq, int Hkv, int D, int m, int S, int64_t T, int dtype,
                     float scale, bool position, ScorePlan* p) {
  if (L < 1 || Hq < 1 || Hkv < 1 || m < 1 || S < 1 || T < 1) return false;
  if (Hq % Hkv != 0 || (D != 64 && D != 128) || T > kMaxSeqLen) return false;
  if (!(scale >= 0.f) || !isfinite(scale)) return false;
  const int G = Hq / Hkv;
  if ((int64_t)G * m > kMaxRows) return false;
  p->T = T;
  p->L = L; p->Hq = Hq; p->Hkv = Hkv; p->G = G; p->m = m; p->R = G * m; p->D = D;
  p->dtype = dtype;
  p->S = S;
  p->units = S * L * Hkv;
  p->position = position;
  if (position) {
    if (G > 8) return false;
    p->Gp = G <= 4 ? 4 : 8;
    if ((int64_t)p->Gp * m > kMaxRows) return false;
    p->Rp = p->Gp * m;
  } else {
    p->Gp = G;
    p->Rp = p->R;
  }
  p->chunks = (int)((T + kMinChunkTokens - 1) / kMinChunkTokens);
  // Waves of 64 rows in a power-of-two workgroup, except that a unit of 257
  // to 320 rows (five query heads per KV head at m = 64) takes four waves of
  // 80 rows (five MFMA row blocks): as five waves of an eight-wave workgroup
  // it would leave three waves idle and, at two waves per SIMD, one SIMD
  // with twice the rows of the others.
  if (!position && p->Rp > 4 * kRowsPerWave && p->Rp <= 4 * 80) {
    p->rb = 5;
    p->row_groups = 1;
    p->waves = 4;
  } else {
    p->rb = 4;
    p->row_groups = (p->Rp + kRowsPerGroup - 1) / kRowsPerGroup;
    const int rows0 = p->Rp < kRowsPerGroup ? p->Rp : kRowsPerGroup;
    const int need = (rows0 + kRowsPerWave - 1) / kRowsPerWave;
    p->waves = need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : 8;
  }
  const float sc = scale > 0.f ? scale : (float)(1.0 / sqrt((double)D));
  p->c2 = (float)((double)sc * 1.4426950408889634);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  p->off_partial = off; off = al(off + (size_t)p->units * p->chunks * p->Rp * sizeof(float2));
  p->off_imp_partial = off;
  if (p->row_groups > 1) off = al(off + (size_t)p->row_groups * p->units * (size_t)T * sizeof(float));
  p->off_numer_partial = off;
  if (position && p->row_groups > 1)
    off = al(off + (size_t)p->row_groups * p->units * (size_t)T * sizeof(float));
  // cb_pipeline's selection of the same units: its arrival counters follow
  // the score kernel's synchronisation words (cleared by the same launch),
  // its digit counts come last.
  p->sel = SelectSplit{1, 0, 0, 0};
  if (!position) select_split_plan(p->units, T, &p->sel);
  p->off_sync = off;
  p->off_sel_counters = kSyncHeader + (size_t)p->units * p->row_groups + (size_t)p->units;
  p->sync_words = p->off_sel_counters +
                  (p->sel.parts > 1 ? (size_t)p->units * kSplitCounterWords : 0);
  off = al(off + p->sync_words * sizeof(uint32_t));
  p->off_sel_data = off;
  if (p->sel.parts > 1)
    off = al(off + (size_t)p->units * p->sel.data_words_per_unit * sizeof(uint32_t));
  p->total_bytes = off;
  return true;
}

hipError_t launch_persistent(const ScorePlan& p, PersistArgs& a, hipStream_t s) {
  if (p.position) {
    if (p.dtype == 1)
      return p.D == 128 ? launch_position_d<2, 128>(p, a, s) : launch_position_d<2, 64>(p, a, s);
    return p.D == 128 ? launch_position_d<4, 128>(p, a, s) : launch_position_d<4, 64>(p, a, s);
  }
  if (p.dtype == 1)
    return p.D == 128 ? launch_score_d<2, 128>(p, a, s) : launch_score_d<2, 64>(p, a, s);
  return p.D == 128 ? launch_score_d<4, 128>(p, a, s) : launch_score_d<4, 64>(p, a, s);
}

}  // namespace cb
